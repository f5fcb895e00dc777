"""Host-side tests of the C ABI (no kernel is ever launched here).

* libcliffconv.so loads and exports every entry point the headers in
  include/ declare;
* the library's signature-driven table (closed form on bitmasks) equals the
  oracle's word-rewriting table for all 39 signatures with k <= 3;
* every argument error is reported before any device work.

The error cases pass fake, never-dereferenced device addresses, so each case
carries a defect the library must reject; the module is skipped where a GPU
is visible (the GPU suite checks the same errors with real buffers).
"""
import ctypes
import glob
import itertools
import os
import re

import pytest

import oracle
import paper_2507_01040_amd as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


def _lib_or_skip():
    if not os.path.exists(P.LIB_PATH):
        pytest.skip("libcliffconv.so not built")
    return P.load()


def _declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M))
    return names


def test_header_declares_the_entry_points():
    decl = _declared_functions()
    assert set(P.EXPORTED) <= decl, decl


def test_library_exports_every_declared_symbol():
    lib = _lib_or_skip()
    for name in _declared_functions():
        assert hasattr(lib, name), name


def test_status_strings():
    _lib_or_skip()
    for s in range(8):
        assert P.status_string(s) and "unknown" not in P.status_string(s)
    assert "unknown" in P.status_string(99)


@pytest.mark.parametrize("g", [g for k in (1, 2, 3)
                               for g in itertools.product((-1, 0, 1), repeat=k)],
                         ids=str)
def test_library_table_equals_oracle_table(g):
    _lib_or_skip()
    k = len(g)
    nb = 1 << k
    src, sign = P.cliffconv_cayley_table(k, g)
    blade, osign = oracle.cayley(k, g)
    for i in range(nb):
        for j in range(nb):
            a = src[i][j]
            # e_a e_j = sign * e_i
            assert blade[a][j] == i, (g, i, j)
            assert osign[a][j] == sign[i][j], (g, i, j)


FAKE = 0x7F0000000000  # 16-byte aligned, never dereferenced


def _conv(**kw):
    args = dict(k=2, g=(1, 1), B=2, C_in=3, C_out=4, d_image=8, d_filter=3,
                input_ptr=FAKE, filters_ptr=FAKE + (1 << 24),
                bias_ptr=FAKE + (2 << 24), output_ptr=FAKE + (3 << 24),
                act=None, stream=0)
    args.update(kw)
    return P.clifford_conv_nd(**args)


@pytest.fixture(scope="module", autouse=False)
def no_gpu():
    import torch
    if torch.cuda.is_available():
        pytest.skip("host-only error tests; the GPU suite covers these with real buffers")
    _lib_or_skip()


CONV_ERRORS = [
    (dict(input_ptr=0), P.CLIFF_EINVAL),
    (dict(filters_ptr=0), P.CLIFF_EINVAL),
    (dict(output_ptr=0), P.CLIFF_EINVAL),
    (dict(k=0, g=()), P.CLIFF_EINVAL),
    (dict(k=4, g=(1, 1, 1, 1)), P.CLIFF_EINVAL),
    (dict(g=(2, 1)), P.CLIFF_EINVAL),
    (dict(g=(0, 0)), P.CLIFF_EINVAL),
    (dict(B=-1), P.CLIFF_ESHAPE),
    (dict(C_in=0), P.CLIFF_ESHAPE),
    (dict(C_out=0), P.CLIFF_ESHAPE),
    (dict(d_filter=0), P.CLIFF_ESHAPE),
    (dict(d_image=2), P.CLIFF_ESHAPE),
    (dict(B=1 << 30, C_in=1 << 10), P.CLIFF_ESHAPE),
    (dict(input_ptr=FAKE + 4), P.CLIFF_EALIGN),
    (dict(output_ptr=FAKE + (3 << 24) + 8), P.CLIFF_EALIGN),
    (dict(bias_ptr=FAKE + (2 << 24) + 4), P.CLIFF_EALIGN),
    (dict(output_ptr=FAKE + 256), P.CLIFF_EOVERLAP),
    (dict(output_ptr=FAKE + (1 << 24) - 1024), P.CLIFF_EOVERLAP),
    (dict(bias_ptr=FAKE + (3 << 24) + 64), P.CLIFF_EOVERLAP),
]


@pytest.mark.parametrize("kw,expect", CONV_ERRORS, ids=lambda v: str(v))
def test_conv_argument_errors(no_gpu, kw, expect):
    assert _conv(**kw) == expect


ACT_ERRORS = [
    (dict(mode=3), P.CLIFF_EINVAL),
    (dict(blades=()), P.CLIFF_EINVAL),
    (dict(blades=(0, 1, 2, 3, 0)), P.CLIFF_EINVAL),
    (dict(blades=(4,)), P.CLIFF_EINVAL),
    (dict(blades=(1, 1)), P.CLIFF_EINVAL),
    (dict(blades=(-1,)), P.CLIFF_EINVAL),
    (dict(weight=0), P.CLIFF_EINVAL),
    (dict(bias=0), P.CLIFF_EINVAL),
    (dict(weight=FAKE + (4 << 24) + 2), P.CLIFF_EALIGN),
]


def _act_desc(mode=P.AGG_LINEAR, blades=(0, 1, 2, 3), weight=FAKE + (4 << 24),
              bias=FAKE + (5 << 24)):
    return P.make_act_desc(mode, blades, weight, bias)


@pytest.mark.parametrize("kw,expect", ACT_ERRORS, ids=lambda v: str(v))
def test_fused_act_errors(no_gpu, kw, expect):
    assert _conv(act=_act_desc(**kw)) == expect


def test_fused_act_weight_overlapping_output(no_gpu):
    d = _act_desc(weight=FAKE + (3 << 24) + 16)
    assert _conv(act=d) == P.CLIFF_EOVERLAP


@pytest.mark.parametrize("kw,expect", ACT_ERRORS, ids=lambda v: str(v))
def test_standalone_act_errors(no_gpu, kw, expect):
    d = _act_desc(**kw)
    assert P.multivector_act(4, 2, 3, 5, d, FAKE, FAKE + (1 << 24)) == expect


def test_standalone_act_shape_and_pointer_errors(no_gpu):
    d = _act_desc()
    assert P.multivector_act(3, 2, 3, 5, d, FAKE, FAKE + (1 << 24)) == P.CLIFF_EINVAL
    assert P.multivector_act(4, 2, 0, 5, d, FAKE, FAKE + (1 << 24)) == P.CLIFF_ESHAPE
    assert P.multivector_act(4, 2, 3, 0, d, FAKE, FAKE + (1 << 24)) == P.CLIFF_ESHAPE
    assert P.multivector_act(4, -1, 3, 5, d, FAKE, FAKE + (1 << 24)) == P.CLIFF_ESHAPE
    assert P.multivector_act(4, 2, 3, 5, d, 0, FAKE) == P.CLIFF_EINVAL
    assert P.multivector_act(4, 2, 3, 5, d, FAKE + 8, FAKE + (1 << 24)) == P.CLIFF_EALIGN
    # partial overlap of input and output
    assert P.multivector_act(4, 2, 3, 5, d, FAKE, FAKE + 32) == P.CLIFF_EOVERLAP
    lib = P.load()
    assert lib.multivector_act(4, 2, 3, 5, None, FAKE, FAKE + (1 << 24), None) == P.CLIFF_EINVAL


def test_forced_tile_refuses_unstageable_k1(no_gpu):
    # the 1-D medium tile (64 channels) with 4-byte filter loads (odd C_out)
    # cannot stage 64 x 17 filter taps per channel pair: refused before any
    # launch
    st = P.clifford_conv_nd_algo(1, (-1,), 2, 3, 65, 60, 17, FAKE, FAKE + (1 << 24),
                                 FAKE + (2 << 24), FAKE + (3 << 24), None, 0,
                                 P.ALGO_MFMA_MEDIUM)
    assert st == P.CLIFF_EUNSUPPORTED


def test_mfma_probe_argument_errors(no_gpu):
    lib = P.load()
    assert lib.cliffconv_mfma_peak_probe(4, 8, None, None) == P.CLIFF_EINVAL
    assert lib.cliffconv_mfma_peak_probe(0, 8, FAKE, None) == P.CLIFF_ESHAPE
    assert lib.cliffconv_mfma_peak_probe(4, 0, FAKE, None) == P.CLIFF_ESHAPE
    assert lib.cliffconv_mfma_peak_probe(1 << 31, 8, FAKE, None) == P.CLIFF_ESHAPE


def _block(**kw):
    args = dict(k=2, g=(1, 1), B=2, C_in=3, C_mid=4, C_out=5, d_image=9, d_filter=3,
                input_ptr=FAKE, filters1_ptr=FAKE + (1 << 24), bias1_ptr=FAKE + (2 << 24),
                act1=None, filters2_ptr=FAKE + (3 << 24), bias2_ptr=FAKE + (4 << 24),
                act2=None, workspace_ptr=FAKE + (5 << 24), output_ptr=FAKE + (6 << 24),
                stream=0, path=P.BLOCK_AUTO)
    args.update(kw)
    return P.clifford_block2_nd_path(**args)


BLOCK_ERRORS = [
    (dict(workspace_ptr=0), P.CLIFF_EINVAL),
    (dict(filters2_ptr=0), P.CLIFF_EINVAL),
    (dict(path=3), P.CLIFF_EINVAL),
    (dict(g=(0, 0)), P.CLIFF_EINVAL),
    (dict(C_mid=0), P.CLIFF_ESHAPE),
    (dict(d_image=4), P.CLIFF_ESHAPE),          # d_out would be 0
    (dict(workspace_ptr=FAKE + (5 << 24) + 4), P.CLIFF_EALIGN),
    (dict(bias2_ptr=FAKE + (4 << 24) + 8), P.CLIFF_EALIGN),
    (dict(workspace_ptr=FAKE + (6 << 24) + 64), P.CLIFF_EOVERLAP),   # workspace over output
    (dict(workspace_ptr=FAKE + (3 << 24) + 16), P.CLIFF_EOVERLAP),   # workspace over filters2
    (dict(output_ptr=FAKE + 32), P.CLIFF_EOVERLAP),                  # output over input
]


@pytest.mark.parametrize("kw,expect", BLOCK_ERRORS, ids=lambda v: str(v))
def test_block_argument_errors(no_gpu, kw, expect):
    assert _block(**kw) == expect


def test_block_zero_batch_is_noop(no_gpu):
    assert _block(B=0) == P.CLIFF_OK


def test_bad_algo(no_gpu):
    st = P.clifford_conv_nd_algo(2, (1, 1), 2, 3, 4, 8, 3, FAKE, FAKE + (1 << 24),
                                 FAKE + (2 << 24), FAKE + (3 << 24), None, 0, 8)
    assert st == P.CLIFF_EINVAL


def test_table_rejects_bad_arguments():
    _lib_or_skip()
    with pytest.raises(P.CliffError):
        P.cliffconv_cayley_table(4, (1, 1, 1, 1))
    with pytest.raises(P.CliffError):
        P.cliffconv_cayley_table(2, (1, 3))


def test_missing_library_fails_loudly(tmp_path):
    import importlib
    saved = P._lib
    try:
        P._lib = None
        with pytest.raises(RuntimeError, match="not built"):
            P.load(str(tmp_path / "nope.so"))
    finally:
        P._lib = saved


def test_stream_algo_refuses_convolution(no_gpu):
    # the streamed kernel is for linear layers only: refused before any launch
    st = P.clifford_conv_nd_algo(2, (1, 1), 2, 32, 32, 8, 3, FAKE, FAKE + (1 << 24),
                                 FAKE + (2 << 24), FAKE + (3 << 24), None, 0,
                                 P.ALGO_MFMA_STREAM)
    assert st == P.CLIFF_EUNSUPPORTED


def test_one_hip_runtime_per_process():
    # The binding loads torch before the library, so the library binds to the
    # HIP runtime torch brought (both carry the soname libamdhip64.so.7): one
    # runtime in the process.  Loaded the other way round, the dynamic linker
    # maps a second copy of the runtime (torch asks for it by file name), and
    # launches on torch's streams and memory fail or race.
    import subprocess
    import sys
    code = ("import sys; sys.path.insert(0, %r)\n"
            "import paper_2507_01040_amd as P\n"
            "P.load()\n"
            "import torch\n"
            "maps = open('/proc/self/maps').read().splitlines()\n"
            "print(len({l.split()[-1] for l in maps if 'libamdhip64' in l}))\n") % ROOT
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    assert r.stdout.strip().splitlines()[-1] == "1", r.stdout
