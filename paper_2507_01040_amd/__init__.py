"""Python binding of libcliffconv.so, the MI355X (gfx950) Clifford
convolution library.

The entry points carry the names of the C ABI in include/cliffconv.h and only
marshal arguments; every step of the computation runs in the library's HIP
kernels.  torch is used for device memory and the current stream only.  The
library is built in-tree by ``paper_2507_01040_amd.build`` (or
``__graft_entry__.build()``); importing this module does not build it, and
every call raises if it is missing.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcliffconv.so")

CLIFF_OK, CLIFF_EINVAL, CLIFF_ESHAPE, CLIFF_EALIGN = 0, 1, 2, 3
CLIFF_EOVERLAP, CLIFF_EUNSUPPORTED, CLIFF_EDEVICE, CLIFF_ESCRATCH = 4, 5, 6, 7
STATUS_NAMES = {0: "CLIFF_OK", 1: "CLIFF_EINVAL", 2: "CLIFF_ESHAPE",
                3: "CLIFF_EALIGN", 4: "CLIFF_EOVERLAP",
                5: "CLIFF_EUNSUPPORTED", 6: "CLIFF_EDEVICE", 7: "CLIFF_ESCRATCH"}
NOALLOC_SCRATCH_FLOATS = 16 * 1024 * 1024  # CLIFF_NOALLOC_SCRATCH_FLOATS
AGG_LINEAR, AGG_SUM, AGG_MEAN = 0, 1, 2
ALGO_AUTO, ALGO_DIRECT, ALGO_MFMA = 0, 1, 2
ALGO_MFMA_WIDE, ALGO_MFMA_MEDIUM, ALGO_MFMA_NARROW, ALGO_MFMA_TINY = 3, 4, 5, 6
ALGO_MFMA_STREAM = 7  # linear layers only
BLOCK_AUTO, BLOCK_TWO_LAUNCH, BLOCK_FUSED = 0, 1, 2

EXPORTED = ("clifford_conv_nd", "clifford_conv_nd_algo", "clifford_linear",
            "multivector_act", "cliffconv_cayley_table", "cliffconv_status_string",
            "cliffconv_mfma_peak_probe", "clifford_block2_nd", "clifford_block2_nd_path",
            "clifford_block2_nd_noalloc")


class CliffActDesc(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("K", ctypes.c_int32),
                ("blade_idx", ctypes.c_int32 * 8),
                ("weight", ctypes.c_void_p), ("bias", ctypes.c_void_p)]


class CliffError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s: %s (%s)" % (where, STATUS_NAMES.get(status, status),
                                          status_string(status)))


_lib = None


def load(path: str = LIB_PATH):
    """Loads the HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    # torch first: the library then binds to the HIP runtime torch loaded (the
    # same soname), so that streams, memory and launch errors are shared.  The
    # other order loads a second copy of the runtime next to torch's, whose
    # launches fail or race with torch's streams.
    import torch  # noqa: F401
    if not os.path.exists(path):
        raise RuntimeError(
            "libcliffconv.so is not built (%s); run __graft_entry__.build()" % path)
    lib = ctypes.CDLL(path)
    i64, vp, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    conv_args = [i32, vp, i64, i64, i64, i64, i64, vp, vp, vp, vp,
                 ctypes.POINTER(CliffActDesc), vp]
    lib.clifford_conv_nd.argtypes = conv_args
    lib.clifford_conv_nd_algo.argtypes = conv_args + [i32]
    lib.clifford_linear.argtypes = [i32, vp, i64, i64, i64, vp, vp, vp, vp,
                                    ctypes.POINTER(CliffActDesc), vp]
    lib.multivector_act.argtypes = [i32, i64, i64, i64,
                                    ctypes.POINTER(CliffActDesc), vp, vp, vp]
    lib.cliffconv_cayley_table.argtypes = [i32, vp, vp, vp]
    lib.cliffconv_mfma_peak_probe.argtypes = [i64, ctypes.c_int32, vp, vp]
    block_args = [i32, vp, i64, i64, i64, i64, i64, i64, vp, vp, vp,
                  ctypes.POINTER(CliffActDesc), vp, vp, ctypes.POINTER(CliffActDesc), vp, vp, vp]
    lib.clifford_block2_nd.argtypes = block_args
    lib.clifford_block2_nd_path.argtypes = block_args + [i32]
    # the block without the workspace argument
    lib.clifford_block2_nd_noalloc.argtypes = block_args[:15] + block_args[16:]
    lib.cliffconv_status_string.argtypes = [i32]
    lib.cliffconv_status_string.restype = ctypes.c_char_p
    for name in ("clifford_conv_nd", "clifford_conv_nd_algo", "clifford_linear",
                 "multivector_act", "cliffconv_cayley_table", "cliffconv_mfma_peak_probe",
                 "clifford_block2_nd", "clifford_block2_nd_path", "clifford_block2_nd_noalloc"):
        getattr(lib, name).restype = i32
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().cliffconv_status_string(status).decode()


def _g_array(g: Sequence[int]):
    arr = (ctypes.c_int8 * max(len(g), 1))(*[int(v) for v in g])
    return arr


def make_act_desc(mode: int, blades: Sequence[int], weight_ptr: int = 0,
                  bias_ptr: int = 0) -> CliffActDesc:
    d = CliffActDesc()
    d.mode = int(mode)
    d.K = len(blades)
    for t, b in enumerate(blades[:8]):
        d.blade_idx[t] = int(b)
    d.weight = weight_ptr or None
    d.bias = bias_ptr or None
    return d


# ---------------------------------------------------------------------------
# Raw C-ABI calls (pointers are ints, as from torch.Tensor.data_ptr()).
# ---------------------------------------------------------------------------

def clifford_conv_nd(k: int, g: Sequence[int], B: int, C_in: int, C_out: int,
                     d_image: int, d_filter: int, input_ptr: int,
                     filters_ptr: int, bias_ptr: int, output_ptr: int,
                     act: Optional[CliffActDesc] = None, stream: int = 0) -> int:
    """Returns the cliff_status of the C call."""
    return load().clifford_conv_nd(
        k, _g_array(g), B, C_in, C_out, d_image, d_filter, input_ptr or None,
        filters_ptr or None, bias_ptr or None, output_ptr or None,
        ctypes.byref(act) if act is not None else None, stream or None)


def clifford_conv_nd_algo(k: int, g: Sequence[int], B: int, C_in: int,
                          C_out: int, d_image: int, d_filter: int,
                          input_ptr: int, filters_ptr: int, bias_ptr: int,
                          output_ptr: int, act: Optional[CliffActDesc] = None,
                          stream: int = 0, algo: int = ALGO_AUTO) -> int:
    return load().clifford_conv_nd_algo(
        k, _g_array(g), B, C_in, C_out, d_image, d_filter, input_ptr or None,
        filters_ptr or None, bias_ptr or None, output_ptr or None,
        ctypes.byref(act) if act is not None else None, stream or None, algo)


def clifford_linear(k: int, g: Sequence[int], B: int, C_in: int, C_out: int,
                    input_ptr: int, weight_ptr: int, bias_ptr: int, output_ptr: int,
                    act: Optional[CliffActDesc] = None, stream: int = 0) -> int:
    return load().clifford_linear(
        k, _g_array(g), B, C_in, C_out, input_ptr or None, weight_ptr or None,
        bias_ptr or None, output_ptr or None,
        ctypes.byref(act) if act is not None else None, stream or None)


def multivector_act(nb: int, B: int, C: int, P: int, act: CliffActDesc,
                    input_ptr: int, output_ptr: int, stream: int = 0) -> int:
    return load().multivector_act(nb, B, C, P, ctypes.byref(act),
                                  input_ptr or None, output_ptr or None,
                                  stream or None)


def clifford_block2_nd_path(k: int, g: Sequence[int], B: int, C_in: int, C_mid: int,
                            C_out: int, d_image: int, d_filter: int, input_ptr: int,
                            filters1_ptr: int, bias1_ptr: int, act1: Optional[CliffActDesc],
                            filters2_ptr: int, bias2_ptr: int, act2: Optional[CliffActDesc],
                            workspace_ptr: int, output_ptr: int, stream: int = 0,
                            path: int = 0) -> int:
    return load().clifford_block2_nd_path(
        k, _g_array(g), B, C_in, C_mid, C_out, d_image, d_filter, input_ptr or None,
        filters1_ptr or None, bias1_ptr or None,
        ctypes.byref(act1) if act1 is not None else None, filters2_ptr or None,
        bias2_ptr or None, ctypes.byref(act2) if act2 is not None else None,
        workspace_ptr or None, output_ptr or None, stream or None, path)


def clifford_block2_nd_noalloc(k: int, g: Sequence[int], B: int, C_in: int, C_mid: int,
                               C_out: int, d_image: int, d_filter: int, input_ptr: int,
                               filters1_ptr: int, bias1_ptr: int, act1: Optional[CliffActDesc],
                               filters2_ptr: int, bias2_ptr: int, act2: Optional[CliffActDesc],
                               output_ptr: int, stream: int = 0) -> int:
    """The block without a workspace: the intermediate lives in the library's
    fixed scratch array (callers that cannot allocate).  Returns the
    cliff_status."""
    return load().clifford_block2_nd_noalloc(
        k, _g_array(g), B, C_in, C_mid, C_out, d_image, d_filter, input_ptr or None,
        filters1_ptr or None, bias1_ptr or None,
        ctypes.byref(act1) if act1 is not None else None, filters2_ptr or None,
        bias2_ptr or None, ctypes.byref(act2) if act2 is not None else None,
        output_ptr or None, stream or None)


def cliffconv_cayley_table(k: int, g: Sequence[int]):
    """(src, sign) as nested lists [N_B][N_B]; raises on bad arguments."""
    nb = 1 << k
    src = (ctypes.c_int8 * (nb * nb))()
    sign = (ctypes.c_int8 * (nb * nb))()
    st = load().cliffconv_cayley_table(k, _g_array(g), src, sign)
    if st != CLIFF_OK:
        raise CliffError(st, "cliffconv_cayley_table")
    return ([[src[i * nb + j] for j in range(nb)] for i in range(nb)],
            [[sign[i * nb + j] for j in range(nb)] for i in range(nb)])


# ---------------------------------------------------------------------------
# torch-tensor conveniences (device memory and stream plumbing only).
# ---------------------------------------------------------------------------

def _check_dev(t, name, device=None):
    """t must be a contiguous float32 GPU tensor (on ``device`` if given)."""
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError("%s must be a GPU tensor" % name)
    if t.dtype != torch.float32 or not t.is_contiguous():
        raise ValueError("%s must be contiguous float32" % name)
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, not on %s with the input" % (name, t.device, device))


def _check_shape(t, shape, name):
    """t's full shape must be ``shape`` (checked before any device check, so
    that a wrong shape is reported as such)."""
    got = tuple(getattr(t, "shape", ()))
    if got != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, got, tuple(shape)))


def _check_act_arg(act, C: int, nb: int, name: str):
    """act is None or (mode, blades, weight [C, K] or None, bias [C] or None):
    blades distinct in [0, N_B); Linear needs both tensors."""
    if act is None:
        return
    mode, blades, aw, ab = act
    K = len(blades)
    if not 1 <= K <= nb or len(set(int(b) for b in blades)) != K or \
            any(not 0 <= int(b) < nb for b in blades):
        raise ValueError("%s: blades %s must be 1..%d distinct indices in [0, %d)"
                         % (name, tuple(blades), nb, nb))
    if mode == AGG_LINEAR:
        if aw is None or ab is None:
            raise ValueError("%s: the Linear gate needs a weight and a bias" % name)
        _check_shape(aw, (C, K), name + " weight")
        _check_shape(ab, (C,), name + " bias")
    elif mode not in (AGG_SUM, AGG_MEAN):
        raise ValueError("%s: unknown aggregation mode %r" % (name, mode))


def _check_act_dev(act, device, name):
    if act is not None and act[0] == AGG_LINEAR:
        _check_dev(act[2], name + " weight", device)
        _check_dev(act[3], name + " bias", device)


def _conv_dims(x, filters, k: int, name: str = "filters"):
    """(B, C_in, C_out, d_image, d_filter) of x [B, C_in, d^k, N_B] and
    filters [C_in, C_out, d_f^k, N_B], with every dimension checked."""
    nb = 1 << k
    xs, fs = tuple(getattr(x, "shape", ())), tuple(getattr(filters, "shape", ()))
    if len(xs) != k + 3 or xs[-1] != nb or len(set(xs[2:-1])) != 1:
        raise ValueError("x has shape %s, expected [B, C_in] + [d_image] * %d + [%d]"
                         % (xs, k, nb))
    B, C_in, d_image = xs[0], xs[1], xs[2]
    if len(fs) != k + 3 or fs[0] != C_in or fs[-1] != nb or len(set(fs[2:-1])) != 1:
        raise ValueError("%s has shape %s, expected [%d, C_out] + [d_filter] * %d + [%d]"
                         % (name, fs, C_in, k, nb))
    C_out, d_filter = fs[1], fs[2]
    if d_filter > d_image:
        raise ValueError("d_filter %d exceeds d_image %d" % (d_filter, d_image))
    return B, C_in, C_out, d_image, d_filter


def _stream_ptr(stream) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def from_paper_protocol(filters, bias=None):
    """Filters (N_B, C_in, C_out, d_f^k) and bias (N_B, C_out) in the paper's
    input/output protocol ("Optimization Performed", convolutional layers:
    blade axis first) to the library's blade-last layouts [C_in, C_out,
    d_f^k, N_B] and [C_out, N_B], as contiguous copies (numpy arrays or torch
    tensors, on the device they are on).  A caller-side layout conversion,
    done once per set of weights; no step of the layer runs here."""
    def last(a):
        if a is None:
            return None
        if hasattr(a, "movedim"):
            return a.movedim(0, -1).contiguous()
        import numpy as np
        return np.ascontiguousarray(np.moveaxis(a, 0, -1))
    return last(filters), last(bias)


def _conv_checked(x, filters, bias, g: Sequence[int], act, out):
    """conv_nd's checks; returns the call's sizes, the output tensor and the
    activation descriptor."""
    import torch
    k = len(g)
    nb = 1 << k
    B, C_in, C_out, d_image, d_filter = _conv_dims(x, filters, k)
    d_out = d_image - d_filter + 1
    shape = (B, C_out) + (d_out,) * k + (nb,)
    if bias is not None:
        _check_shape(bias, (C_out, nb), "bias")
    _check_act_arg(act, C_out, nb, "act")
    if out is not None:
        _check_shape(out, shape, "out")
    _check_dev(x, "x")
    _check_dev(filters, "filters", x.device)
    if bias is not None:
        _check_dev(bias, "bias", x.device)
    _check_act_dev(act, x.device, "act")
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=x.device)
    _check_dev(out, "out", x.device)
    return (k, B, C_in, C_out, d_image, d_filter), out, _act_desc(act)


def conv_nd(x, filters, bias, g: Sequence[int], act: Optional[Tuple] = None,
            out=None, stream=None, algo: int = ALGO_AUTO):
    """Clifford convolution of GPU tensors x [B,C_in,d^k,N_B] and filters
    [C_in,C_out,d_f^k,N_B] with bias [C_out,N_B] (or None); ``act`` is None or
    (mode, blades, weight [C_out,K] or None, bias [C_out] or None).  Returns
    the output tensor [B,C_out,d_out^k,N_B] (allocated with torch unless
    ``out`` is given).  Every tensor's shape, dtype, layout and device is
    checked before the library is called: the C ABI takes raw pointers and
    cannot check the buffers behind them."""
    (k, B, C_in, C_out, d_image, d_filter), out, desc = _conv_checked(x, filters, bias, g,
                                                                       act, out)
    st = clifford_conv_nd_algo(k, g, B, C_in, C_out, d_image, d_filter,
                               x.data_ptr(), filters.data_ptr(),
                               bias.data_ptr() if bias is not None else 0,
                               out.data_ptr(), desc, _stream_ptr(stream), algo)
    if st != CLIFF_OK:
        raise CliffError(st, "clifford_conv_nd")
    return out


class Plan:
    """One library call with its tensors checked and its arguments marshalled
    once, for callers that repeat the same call on the same buffers (loops of
    fixed shape, benchmarks): ``plan()`` enqueues it on the stream it was made
    for, ``plan(stream)`` on another torch stream (or raw stream handle); a
    status other than CLIFF_OK raises CliffError.  The library checks its
    arguments on every call as usual.  The plan holds references to its
    tensors and descriptors; ``plan.out`` is the output tensor."""

    def __init__(self, fn, args, stream_index: int, name: str, out, keep):
        self._fn = fn
        self._args = list(args)
        self._si = stream_index
        self._stream = self._args[stream_index]
        self._name = name
        self.out = out
        self._keep = keep

    def __call__(self, stream=None):
        if stream is None:
            self._args[self._si] = self._stream
        else:
            handle = int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)
            self._args[self._si] = handle or None
        st = self._fn(*self._args)
        if st != CLIFF_OK:
            raise CliffError(st, self._name)
        return self.out


def conv_plan(x, filters, bias, g: Sequence[int], act: Optional[Tuple] = None,
              out=None, stream=None, algo: int = ALGO_AUTO) -> Plan:
    """conv_nd as a Plan: the checks of conv_nd once, then each call only the
    C ABI call (``out`` is allocated here unless given)."""
    (k, B, C_in, C_out, d_image, d_filter), out, desc = _conv_checked(x, filters, bias, g,
                                                                       act, out)
    garr = _g_array(g)
    args = (k, garr, B, C_in, C_out, d_image, d_filter, x.data_ptr(), filters.data_ptr(),
            bias.data_ptr() if bias is not None else None, out.data_ptr(),
            ctypes.byref(desc) if desc is not None else None, _stream_ptr(stream) or None, algo)
    return Plan(load().clifford_conv_nd_algo, args, 12, "clifford_conv_nd", out,
                (x, filters, bias, act, garr, desc))


def linear(x, weight, bias, g: Sequence[int], act: Optional[Tuple] = None,
           out=None, stream=None):
    """Clifford linear layer of GPU tensors x [B, C_in, N_B], weight
    [C_in, C_out, N_B], bias [C_out, N_B] or None; ``act`` as for conv_nd.
    Shapes and devices are checked as in conv_nd."""
    import torch
    k = len(g)
    nb = 1 << k
    xs, ws = tuple(getattr(x, "shape", ())), tuple(getattr(weight, "shape", ()))
    if len(xs) != 3 or xs[-1] != nb:
        raise ValueError("x has shape %s, expected [B, C_in, %d]" % (xs, nb))
    B, C_in = xs[0], xs[1]
    if len(ws) != 3 or ws[0] != C_in or ws[-1] != nb:
        raise ValueError("weight has shape %s, expected [%d, C_out, %d]" % (ws, C_in, nb))
    C_out = ws[1]
    if bias is not None:
        _check_shape(bias, (C_out, nb), "bias")
    _check_act_arg(act, C_out, nb, "act")
    if out is not None:
        _check_shape(out, (B, C_out, nb), "out")
    _check_dev(x, "x")
    _check_dev(weight, "weight", x.device)
    if bias is not None:
        _check_dev(bias, "bias", x.device)
    _check_act_dev(act, x.device, "act")
    if out is None:
        out = torch.empty((B, C_out, nb), dtype=torch.float32, device=x.device)
    _check_dev(out, "out", x.device)
    desc = _act_desc(act)
    st = clifford_linear(k, g, B, C_in, C_out, x.data_ptr(), weight.data_ptr(),
                         bias.data_ptr() if bias is not None else 0, out.data_ptr(),
                         desc, _stream_ptr(stream))
    if st != CLIFF_OK:
        raise CliffError(st, "clifford_linear")
    return out


def act_nd(x, mode: int, blades: Sequence[int], weight=None, bias=None,
           out=None, stream=None):
    """Multivector activation of a GPU tensor [B, C, (positions...), N_B];
    weight [C, K] and bias [C] for the Linear gate.  ``out`` may be x (in
    place).  Shapes and devices are checked before the library is called."""
    import torch
    xs = tuple(getattr(x, "shape", ()))
    if len(xs) < 3 or xs[-1] not in (2, 4, 8):
        raise ValueError("x has shape %s, expected [B, C, (positions...), N_B] with "
                         "N_B in (2, 4, 8)" % (xs,))
    B, C, nb = xs[0], xs[1], xs[-1]
    P = 1
    for s in xs[2:-1]:
        P *= s
    _check_act_arg((mode, blades, weight, bias), C, nb, "activation")
    if out is not None:
        _check_shape(out, xs, "out")
    _check_dev(x, "x")
    _check_act_dev((mode, blades, weight, bias), x.device, "activation")
    if out is None:
        out = torch.empty_like(x)
    _check_dev(out, "out", x.device)
    desc = _act_desc((mode, blades, weight, bias))
    st = multivector_act(nb, B, C, P, desc, x.data_ptr(), out.data_ptr(),
                         _stream_ptr(stream))
    if st != CLIFF_OK:
        raise CliffError(st, "multivector_act")
    return out


def _act_desc(act):
    if act is None:
        return None
    mode, blades, aw, ab = act
    return make_act_desc(mode, blades, aw.data_ptr() if aw is not None else 0,
                         ab.data_ptr() if ab is not None else 0)


def _block2_checked(x, layer1, layer2, g: Sequence[int], out, workspace):
    """block2's checks; returns the call's sizes, the workspace and output
    tensors and both activation descriptors."""
    import torch
    k = len(g)
    nb = 1 << k
    (f1, b1, a1), (f2, b2, a2) = layer1, layer2
    B, C_in, C_mid, d_image, d_filter = _conv_dims(x, f1, k, "filters1")
    d_mid = d_image - d_filter + 1
    fs2 = tuple(getattr(f2, "shape", ()))
    if len(fs2) != k + 3 or fs2[0] != C_mid or fs2[2:] != (d_filter,) * k + (nb,):
        raise ValueError("filters2 has shape %s, expected [%d, C_out] + [%d] * %d + [%d]"
                         % (fs2, C_mid, d_filter, k, nb))
    C_out = fs2[1]
    if d_mid < d_filter:
        raise ValueError("d_image %d is too small for two layers of d_filter %d"
                         % (d_image, d_filter))
    d_out = d_mid - d_filter + 1
    if b1 is not None:
        _check_shape(b1, (C_mid, nb), "bias1")
    if b2 is not None:
        _check_shape(b2, (C_out, nb), "bias2")
    _check_act_arg(a1, C_mid, nb, "act1")
    _check_act_arg(a2, C_out, nb, "act2")
    ws_shape = (B, C_mid) + (d_mid,) * k + (nb,)
    out_shape = (B, C_out) + (d_out,) * k + (nb,)
    if workspace is not None and getattr(workspace, "numel", lambda: -1)() != \
            B * C_mid * d_mid ** k * nb:
        raise ValueError("workspace holds %s floats, expected %d (B * C_mid * d_mid^k * N_B)"
                         % (getattr(workspace, "numel", lambda: None)(),
                            B * C_mid * d_mid ** k * nb))
    if out is not None:
        _check_shape(out, out_shape, "out")
    _check_dev(x, "x")
    for t, n in ((f1, "filters1"), (f2, "filters2"), (b1, "bias1"), (b2, "bias2")):
        if t is not None:
            _check_dev(t, n, x.device)
    _check_act_dev(a1, x.device, "act1")
    _check_act_dev(a2, x.device, "act2")
    if workspace is None:
        workspace = torch.empty(ws_shape, dtype=torch.float32, device=x.device)
    if out is None:
        out = torch.empty(out_shape, dtype=torch.float32, device=x.device)
    _check_dev(workspace, "workspace", x.device)
    _check_dev(out, "out", x.device)
    return ((k, B, C_in, C_mid, C_out, d_image, d_filter), workspace, out, _act_desc(a1),
            _act_desc(a2))


def block2(x, layer1, layer2, g: Sequence[int], out=None, workspace=None, stream=None,
           path: int = 0):
    """Two-layer block through clifford_block2_nd: ``layer1``/``layer2`` are
    (filters, bias or None, act or None) as in block_forward.  The workspace
    (B * C_mid * d_mid^k * N_B floats) and the output are allocated with
    torch unless given.  Shapes and devices are checked before the library
    is called."""
    (f1, b1, _), (f2, b2, _) = layer1, layer2
    (k, B, C_in, C_mid, C_out, d_image, d_filter), workspace, out, d1, d2 = _block2_checked(
        x, layer1, layer2, g, out, workspace)
    st = clifford_block2_nd_path(k, g, B, C_in, C_mid, C_out, d_image, d_filter,
                                 x.data_ptr(), f1.data_ptr(),
                                 b1.data_ptr() if b1 is not None else 0, d1,
                                 f2.data_ptr(), b2.data_ptr() if b2 is not None else 0,
                                 d2, workspace.data_ptr(), out.data_ptr(),
                                 _stream_ptr(stream), path)
    if st != CLIFF_OK:
        raise CliffError(st, "clifford_block2_nd")
    return out


def block2_plan(x, layer1, layer2, g: Sequence[int], out=None, workspace=None, stream=None,
                path: int = 0) -> Plan:
    """block2 as a Plan: the checks once, then each call only the C ABI call."""
    (f1, b1, a1), (f2, b2, a2) = layer1, layer2
    (k, B, C_in, C_mid, C_out, d_image, d_filter), workspace, out, d1, d2 = _block2_checked(
        x, layer1, layer2, g, out, workspace)
    garr = _g_array(g)
    args = (k, garr, B, C_in, C_mid, C_out, d_image, d_filter, x.data_ptr(), f1.data_ptr(),
            b1.data_ptr() if b1 is not None else None,
            ctypes.byref(d1) if d1 is not None else None, f2.data_ptr(),
            b2.data_ptr() if b2 is not None else None,
            ctypes.byref(d2) if d2 is not None else None, workspace.data_ptr(), out.data_ptr(),
            _stream_ptr(stream) or None, path)
    return Plan(load().clifford_block2_nd_path, args, 17, "clifford_block2_nd", out,
                (x, layer1, layer2, workspace, garr, d1, d2))


def block_forward(x, layers, g: Sequence[int], outs=None, stream=None):
    """Block composition: conv (+ fused bias and activation) for each layer
    in turn, the intermediate kept in HBM in the blade-last layout.
    ``layers`` is a sequence of (filters, bias, act) with act None or
    (mode, blades, weight or None, bias or None); ``outs`` optionally gives
    preallocated outputs per layer."""
    y = x
    for li, (f, b, a) in enumerate(layers):
        y = conv_nd(y, f, b, g, act=a, out=None if outs is None else outs[li],
                    stream=stream)
    return y
