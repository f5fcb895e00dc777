"""CPU oracle for the Clifford convolution and multivector activation.

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg use it; the GPU library never does.  It
shares no code with the GPU path.

The arithmetic lives in ``cliff_oracle.c`` (plain C, fp64, following the
definitions of the paper's "Background" section and Algorithms 1, 2 and 3).  This
module compiles it with gcc into ``liboracle.so`` next to it and marshals numpy
arrays in and out; it adds no arithmetic of its own (inputs are only widened
to float64 and cropped by slicing).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cliff_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

CFLAGS = ["-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
          "-shared", "-pthread"]


def build(force: bool = True) -> str:
    """Compile cliff_oracle.c with gcc into liboracle.so."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or (
                os.path.getmtime(_LIB) < os.path.getmtime(_SRC)):
            build()
        lib = ctypes.CDLL(_LIB)
        i64, p = ctypes.c_int64, ctypes.c_void_p
        lib.oracle_cayley.argtypes = [ctypes.c_int, p, p, p]
        lib.oracle_mv_mul.argtypes = [ctypes.c_int, p, p, p, p]
        lib.oracle_conv_nd.argtypes = [ctypes.c_int, p, i64, i64, i64, i64,
                                       i64, p, p, p, p, ctypes.c_int]
        lib.oracle_conv_points.argtypes = [ctypes.c_int, p, i64, i64, i64, i64,
                                           i64, p, p, p, i64, p, p, p, p]
        lib.oracle_act.argtypes = [ctypes.c_int, i64, i64, i64, ctypes.c_int,
                                   ctypes.c_int, p, p, p, p, p]
        lib.oracle_linear.argtypes = [ctypes.c_int, p, i64, i64, i64, p, p, p, p]
        for f in (lib.oracle_cayley, lib.oracle_mv_mul, lib.oracle_conv_nd,
                  lib.oracle_conv_points, lib.oracle_act, lib.oracle_linear):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _g(g: Sequence[int]) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(g, dtype=np.int32))


def default_threads() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def cayley(k: int, g: Sequence[int]):
    """(blade[a, b], sign[a, b]) with e_a e_b = sign * e_blade (grade-lex
    blade order, 0-based)."""
    nb = 1 << k
    blade = np.zeros((nb, nb), np.int32)
    sign = np.zeros((nb, nb), np.float64)
    gg = _g(g)
    if _load().oracle_cayley(k, _ptr(gg), _ptr(blade), _ptr(sign)) != nb:
        raise ValueError("bad k")
    return blade, sign


def mv_mul(k: int, g: Sequence[int], x, y) -> np.ndarray:
    """Geometric product x * y of two multivectors."""
    nb = 1 << k
    xx, yy = _f64(x).reshape(nb), _f64(y).reshape(nb)
    z = np.zeros(nb, np.float64)
    gg = _g(g)
    if _load().oracle_mv_mul(k, _ptr(gg), _ptr(xx), _ptr(yy), _ptr(z)):
        raise ValueError("bad k")
    return z


def _conv_dims(x, f, k):
    B, C_in = x.shape[0], x.shape[1]
    d_image = x.shape[2]
    C_out, d_filter = f.shape[1], f.shape[2]
    nb = 1 << k
    assert x.shape == (B, C_in) + (d_image,) * k + (nb,), x.shape
    assert f.shape == (C_in, C_out) + (d_filter,) * k + (nb,), f.shape
    return B, C_in, C_out, d_image, d_filter


def conv_nd(x, f, bias, g: Sequence[int], nthreads: Optional[int] = None
            ) -> np.ndarray:
    """Algorithm 1 in fp64.  x [B,C_in,d^k,N_B], f [C_in,C_out,d_f^k,N_B],
    bias [C_out,N_B] or None (zero).  Returns [B,C_out,d_out^k,N_B] float64."""
    k = len(g)
    x, f = _f64(x), _f64(f)
    b = None if bias is None else _f64(bias)
    B, C_in, C_out, d_image, d_filter = _conv_dims(x, f, k)
    d_out = d_image - d_filter + 1
    out = np.empty((B, C_out) + (d_out,) * k + (1 << k,), np.float64)
    gg = _g(g)
    rc = _load().oracle_conv_nd(k, _ptr(gg), B, C_in, C_out, d_image,
                                d_filter, _ptr(x), _ptr(f), _ptr(b),
                                _ptr(out), nthreads or default_threads())
    if rc:
        raise ValueError("oracle_conv_nd rejected the arguments")
    return out


def conv_points(x, f, bias, g: Sequence[int], bs, cos, ps) -> np.ndarray:
    """Selected outputs of Algorithm 1: row s is output[bs[s], cos[s], p]
    with p the flat row-major output position ps[s].  Returns [n, N_B]."""
    k = len(g)
    x, f = _f64(x), _f64(f)
    b = None if bias is None else _f64(bias)
    B, C_in, C_out, d_image, d_filter = _conv_dims(x, f, k)
    bs = np.ascontiguousarray(bs, np.int64)
    cos = np.ascontiguousarray(cos, np.int64)
    ps = np.ascontiguousarray(ps, np.int64)
    n = bs.shape[0]
    out = np.empty((n, 1 << k), np.float64)
    gg = _g(g)
    rc = _load().oracle_conv_points(k, _ptr(gg), B, C_in, C_out, d_image,
                                    d_filter, _ptr(x), _ptr(f), _ptr(b), n,
                                    _ptr(bs), _ptr(cos), _ptr(ps), _ptr(out))
    if rc:
        raise ValueError("oracle_conv_points rejected the arguments")
    return out


def linear(x, w, bias, g: Sequence[int]) -> np.ndarray:
    """Algorithm 2 in fp64: x [B, C_in, N_B], w [C_in, C_out, N_B], bias
    [C_out, N_B] or None.  Returns [B, C_out, N_B] float64."""
    k = len(g)
    x, w = _f64(x), _f64(w)
    b = None if bias is None else _f64(bias)
    B, C_in, nb = x.shape
    C_out = w.shape[1]
    assert nb == 1 << k and w.shape == (C_in, C_out, nb), (x.shape, w.shape)
    out = np.empty((B, C_out, nb), np.float64)
    gg = _g(g)
    if _load().oracle_linear(k, _ptr(gg), B, C_in, C_out, _ptr(x), _ptr(w), _ptr(b),
                             _ptr(out)):
        raise ValueError("oracle_linear rejected the arguments")
    return out


def act(x, mode: int, blades: Sequence[int], weight=None, bias=None
        ) -> np.ndarray:
    """Algorithm 3 in fp64 on x [B, C, (positions...), N_B]; positions share
    the channel's weight [C, K] and bias [C] (Linear mode only)."""
    x = _f64(x)
    B, C, nb = x.shape[0], x.shape[1], x.shape[-1]
    P = int(np.prod(x.shape[2:-1])) if x.ndim > 3 else 1
    idx = np.ascontiguousarray(blades, np.int32)
    K = idx.shape[0]
    w = None if weight is None else _f64(weight).reshape(C, K)
    b = None if bias is None else _f64(bias).reshape(C)
    if mode == 0 and (w is None or b is None):
        raise ValueError("Linear mode needs weight and bias")
    out = np.empty_like(x)
    rc = _load().oracle_act(nb, B, C, P, mode, K, _ptr(idx), _ptr(w), _ptr(b),
                            _ptr(x), _ptr(out))
    if rc:
        raise ValueError("oracle_act rejected the arguments")
    return out


def block(x, layers, g: Sequence[int], nthreads: Optional[int] = None
          ) -> np.ndarray:
    """conv -> act -> conv -> act ... in fp64 end to end.  ``layers`` is a
    sequence of (filters, bias, act) with act None or (mode, blades, weight,
    bias)."""
    y = _f64(x)
    for f, b, a in layers:
        y = conv_nd(y, f, b, g, nthreads)
        if a is not None:
            mode, blades, aw, ab = a
            y = act(y, mode, blades, aw, ab)
    return y
