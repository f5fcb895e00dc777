"""Every launch the library would make, checked on the CPU before any GPU
sees it.

A CPU build of the library (its own host sources, AddressSanitizer and
UndefinedBehaviorSanitizer on) runs the C ABI entry points with a launch
observer installed (tests/hostcheck/): argument checks, sign table and kernel
choice run as on the GPU, and each launch plan goes to a checker that walks
the kernel's own address arithmetic over every workgroup and lane.  For the
matrix-core convolution (k = 2, 3) that is every direct global->LDS load in
bounds, every LDS word a fragment reads written by the stage with the input
or filter element the product needs, every output stored once in bounds
(tests/hostcheck/check_conv_mfma.cpp); the same for the 1-D matrix-core
convolution (check_conv1d.cpp), the fused small block
(check_block_small.cpp), the streamed linear layer (check_linear.cpp) and the
standalone activation (check_act.cpp) and the direct (vector-ALU) kernel
(check_direct.cpp).

Cases: the GPU parity shapes with every tile shape forced, the benchmark's
workloads at full size, the random sweeps' draws (convolutions and blocks),
the block entry point's cases, and wide images.  Each must come back "ok"
with the status the GPU tests expect (CLIFF_OK, or CLIFF_EUNSUPPORTED for a
forced tile that refuses a shape).
"""
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

import paper_2507_01040_amd as P  # noqa: E402
import workloads as W  # noqa: E402
from hostcheck import build as HC  # noqa: E402

ALGOS = [P.ALGO_AUTO, P.ALGO_MFMA, P.ALGO_DIRECT, P.ALGO_MFMA_WIDE, P.ALGO_MFMA_MEDIUM,
         P.ALGO_MFMA_NARROW, P.ALGO_MFMA_TINY]
ALGO_NAMES = dict(zip(ALGOS, ["auto", "mfma", "direct", "wide", "medium", "narrow", "tiny"]))


def act_field(act):
    if act is None:
        return "-1 0"
    mode, blades = act[0], act[1]
    return "%d %d %s" % (mode, len(blades), " ".join(str(b) for b in blades))


def conv_line(k, g, B, C_in, C_out, d, df, algo, act=None):
    return "conv %d %s %d %d %d %d %d %d %s" % (k, " ".join(str(v) for v in g), B, C_in, C_out,
                                               d, df, algo, act_field(act))


def block_line(k, g, B, C_in, C_mid, C_out, d, df, path, act1=None, act2=None):
    return "block %d %s %d %d %d %d %d %d %d %s %s" % (
        k, " ".join(str(v) for v in g), B, C_in, C_mid, C_out, d, df, path, act_field(act1),
        act_field(act2))


def _run_cases(cases, allow_unsupported):
    """cases: (label, line); every result must be ok with CLIFF_OK (or, where
    allowed, CLIFF_EUNSUPPORTED: a forced tile refusing the shape)."""
    out = HC.run([line for _, line in cases])
    assert len(out) == len(cases), out[-5:]
    bad = []
    for (label, line), res in zip(cases, out):
        f = res.split()
        ok_status = {P.CLIFF_OK} | ({P.CLIFF_EUNSUPPORTED} if allow_unsupported(line) else set())
        if f[0] != "ok" or int(f[1]) not in ok_status:
            bad.append("%s: %s" % (label, res[:600]))
    assert not bad, "\n".join(bad[:20])
    return out


def _is_forced_tile(line):
    f = line.split()
    if f[0] != "conv":
        return False
    k = int(f[1])
    algo = int(f[2 + k + 5])
    return algo >= P.ALGO_MFMA_WIDE


def test_parity_shapes_every_tile():
    import test_parity_gpu as T
    cases = []
    for g, shapes in (((1, 1), T.SHAPES2), ((1, 1, 1), T.SHAPES3), ((-1,), T.SHAPES1)):
        k = len(g)
        for (B, C_in, C_out, d, df) in shapes:
            for algo in ALGOS:
                for act in (None, (P.AGG_LINEAR, tuple(range(1 << k)))):
                    cases.append(("%s %s %s act=%s" % (g, (B, C_in, C_out, d, df), ALGO_NAMES[algo],
                                                       act is not None),
                                  conv_line(k, g, B, C_in, C_out, d, df, algo, act)))
    _run_cases(cases, _is_forced_tile)


def test_benchmark_workloads_full_size():
    cases = []
    for name, w in W.WORKLOADS.items():
        for li, (s, act) in enumerate(zip(w.layers, w.acts)):
            a = None if act is None else (act.mode, act.blades)
            for algo in (P.ALGO_AUTO, P.ALGO_MFMA):
                cases.append(("%s layer %d algo %s" % (name, li, ALGO_NAMES[algo]),
                              conv_line(s.k, s.g, s.B, s.C_in, s.C_out, s.d_image, s.d_filter,
                                        algo, a)))
        if len(w.layers) == 2:
            s0, s1 = w.layers
            a0 = None if w.acts[0] is None else (w.acts[0].mode, w.acts[0].blades)
            a1 = None if w.acts[1] is None else (w.acts[1].mode, w.acts[1].blades)
            cases.append(("%s block" % name,
                          block_line(s0.k, s0.g, s0.B, s0.C_in, s0.C_out, s1.C_out, s0.d_image,
                                     s0.d_filter, P.BLOCK_AUTO, a0, a1)))
    _run_cases(cases, lambda line: False)


def test_random_sweep_draws():
    import test_random_sweep_gpu as R
    cases = []
    for (k, g, B, C_in, C_out, d, df, algo, act, seed) in R.CASES:
        cases.append((str((k, g, B, C_in, C_out, d, df, algo, act)),
                      conv_line(k, g, B, C_in, C_out, d, df, algo, act)))
    _run_cases(cases, _is_forced_tile)


def test_block_entry_cases():
    import test_block_gpu as TB
    import test_random_block_gpu as RB
    cases = []
    for c in TB.CASES:
        g, B, C_in, C_mid, C_out, d, df, (a1, a2) = c
        for path in (P.BLOCK_AUTO, P.BLOCK_TWO_LAUNCH, P.BLOCK_FUSED):
            cases.append((str(c) + " path %d" % path,
                          block_line(len(g), g, B, C_in, C_mid, C_out, d, df, path, a1, a2)))
    for c in RB.BLOCKS:
        g, B, C_in, C_mid, C_out, d, df, (a1, a2) = c[:8]
        for path in (P.BLOCK_TWO_LAUNCH, P.BLOCK_FUSED):
            cases.append((str(c) + " path %d" % path,
                          block_line(len(g), g, B, C_in, C_mid, C_out, d, df, path, a1, a2)))
    _run_cases(cases, lambda line: int(line.split()[8 + int(line.split()[1])]) == P.BLOCK_FUSED)


def test_medium_images_every_tile():
    # images around the sizes where the wide tiles switch between whole-row
    # and row-aligned blocks, and the 96-position tile
    cases = []
    for d, C, B in ((96, 64, 8), (130, 64, 2), (258, 64, 1), (300, 32, 1), (520, 16, 1),
                    (1030, 8, 1)):
        for df in (3, 5):
            for algo in (P.ALGO_AUTO, P.ALGO_MFMA_WIDE, P.ALGO_MFMA_NARROW):
                cases.append(("2D d %d C %d df %d algo %s" % (d, C, df, ALGO_NAMES[algo]),
                              conv_line(2, (1, 1), B, C, C, d, df, algo)))
    for d, C in ((24, 32), (42, 32), (34, 64), (20, 16)):
        for algo in (P.ALGO_AUTO, P.ALGO_MFMA_WIDE, P.ALGO_MFMA_MEDIUM):
            cases.append(("3D d %d C %d algo %s" % (d, C, ALGO_NAMES[algo]),
                          conv_line(3, (1, 1, 1), 2, C, C, d, 3, algo)))
    _run_cases(cases, _is_forced_tile)


def test_wide_images_row_aligned():
    # 2D images of 2048 and more positions per row: row-aligned blocks only
    # (whole-row slabs do not fit), 32-bit offsets from the block's rows
    cases = []
    for d, C, B in ((2050, 16, 1), (2049, 8, 1), (4098, 4, 1), (3000, 2, 1)):
        for algo in (P.ALGO_AUTO, P.ALGO_MFMA_WIDE, P.ALGO_MFMA_NARROW):
            cases.append(("2D d %d C %d algo %s" % (d, C, ALGO_NAMES[algo]),
                          conv_line(2, (1, 1), B, C, C, d, 3, algo)))
    out = _run_cases(cases, lambda line: False)
    for (label, _), res in zip(cases, out):
        assert res.split()[4] == "1", (label, res)  # one matrix-core launch, no fallback


def test_conv1d_176_position_tile():
    # The paper's 1-D filter length (17) on layers whose blocks fill the last
    # round of CUs better at 176 positions than at 128: the quantisation
    # model takes the 176-position form of the wide tile (template NW = 11),
    # and the checker walks it, with 16-byte (d_image even) and 4-byte (odd)
    # input loads.  At B = 8192 the 128-position form fills every round; odd
    # C_out (4-byte filter loads) keeps it too.
    cases, want = [], []
    for B, C_in, C_out, d, nw in ((4096, 64, 64, 60, 11), (1024, 64, 64, 60, 11),
                                  (1000, 64, 62, 60, 11), (2048, 128, 128, 60, 11),
                                  (1001, 64, 64, 61, 11), (8192, 64, 64, 60, 4),
                                  (1000, 64, 63, 60, 4)):
        for algo in (P.ALGO_AUTO, P.ALGO_MFMA_WIDE):
            cases.append(("1-D B %d C %d->%d d %d algo %s" % (B, C_in, C_out, d, ALGO_NAMES[algo]),
                          conv_line(1, (-1,), B, C_in, C_out, d, 17, algo)))
            want.append(nw)
    out = _run_cases(cases, lambda line: False)
    for (label, _), res, nw in zip(cases, out, want):
        f = res.split()
        assert f[4] == "2", (label, res)  # one 1-D matrix-core launch
        assert int(f[5].split(".")[4]) == nw, (label, res)


def test_wide_112_position_tiles():
    # The 112-position forms of the 2D 64-channel and 3D 32-channel wide tiles
    # (template NW = 7): the quantisation model takes them where their blocks
    # fill the last round of CUs best, keeps 128 (the headline's row-aligned
    # blocks, the 2D block's first layer, 3D d 34) or 96 (3D d 32, 2D d 96)
    # elsewhere, and the checker walks each choice.
    cases, want = [], []
    for k, g, B, C_in, C_out, d, nw in ((2, (1, 1), 8, 4, 64, 84, 7), (2, (1, 1), 16, 64, 64, 44, 7),
                                        (2, (1, 1), 4, 64, 64, 148, 7), (2, (-1, 0), 8, 4, 64, 102, 7),
                                        (2, (1, 1), 8, 64, 64, 128, 8), (2, (1, -1), 8, 64, 64, 130, 8),
                                        (2, (1, 1), 8, 4, 64, 96, 6), (3, (1, 1, 1), 8, 4, 32, 24, 7),
                                        (3, (1, -1, 1), 8, 32, 32, 36, 7), (3, (1, 1, 1), 8, 32, 32, 42, 7),
                                        (3, (1, 1, 1), 8, 32, 32, 32, 6), (3, (1, 1, 1), 8, 32, 32, 34, 8)):
        cases.append(("%dD B %d C %d->%d d %d" % (k, B, C_in, C_out, d),
                      conv_line(k, g, B, C_in, C_out, d, 3, P.ALGO_AUTO)))
        want.append(nw)
    out = _run_cases(cases, lambda line: False)
    for (label, _), res, nw in zip(cases, out, want):
        f = res.split()
        assert f[4] == "1", (label, res)  # one matrix-core convolution launch
        assert int(f[5].split(".")[7]) == nw, (label, res)


def test_wide_16_channel_tile():
    # The 2D wide tile's 16-channel form (one wave of channels by four of
    # positions, 512 positions per block), taken for C_out <= 16: the parity
    # cases, forced and automatic, and wide images with row-aligned blocks
    import test_parity_gpu as T
    cases = []
    for g, (B, C_in, C_out, d, df) in T.WIDE16_CASES:
        for algo in (P.ALGO_MFMA_WIDE, P.ALGO_AUTO):
            cases.append(("%s %s algo %s" % (g, (B, C_in, C_out, d, df), ALGO_NAMES[algo]),
                          conv_line(2, g, B, C_in, C_out, d, df, algo)))
    for B, C, d in ((2, 16, 2050), (1, 12, 4098), (128, 16, 130)):
        cases.append(("2D B %d C %d d %d auto" % (B, C, d),
                      conv_line(2, (1, 1), B, C, C, d, 3, P.ALGO_AUTO)))
    out = _run_cases(cases, lambda line: False)
    for (label, _), res in zip(cases, out):
        f = res.split()
        assert f[4] == "1", (label, res)  # one matrix-core launch
        if "wide" in label or "2D B" in label or "514" in label:
            # forced, or a problem large enough that the automatic choice
            # takes it; the small ones may go to a narrower tile
            assert f[5].split(".")[4:9] == ["1", "4", "4", "8", "10"], (label, res)


def test_small_channel_tile_widths():
    # the automatic choice among the 16- and 8-channel tiles' widths (512,
    # 384 or 256 positions; template WCO.WPOS.MW.NW) on the GPU parity cases
    import test_parity_gpu as T
    cases = [("%s %s" % (g, shape), conv_line(2, g, *shape, P.ALGO_AUTO))
             for g, shape in T.SMALL_CHANNEL_WIDTH_CASES]
    out = _run_cases(cases, lambda line: False)
    for (label, _), res, want in zip(cases, out, T.SMALL_CHANNEL_WIDTH_TILES):
        f = res.split()
        assert f[4] == "1", (label, res)
        assert ".".join(f[5].split(".")[4:8]) == want, (label, res, want)


def test_3d_8_channel_tile():
    # the 3D 8-channel tile (template WCO.WPOS.MW.NW 1.4.4.4), forced and
    # automatic, on the GPU parity cases and larger layers
    import test_parity_gpu as T
    cases = []
    for g, shape in T.W3_8_CASES + [((1, 1, 1), (8, 8, 8, 34, 3)), ((1, 0, 1), (2, 8, 8, 66, 3))]:
        for algo in (P.ALGO_MFMA_WIDE, P.ALGO_AUTO):
            cases.append(("%s %s %s" % (g, shape, ALGO_NAMES[algo]),
                          conv_line(3, g, *shape, algo)))
    out = _run_cases(cases, lambda line: False)
    for (label, _), res in zip(cases, out):
        f = res.split()
        assert f[4] == "1", (label, res)
        if "wide" in label or ", 34, 3)" in label or ", 66, 3)" in label:
            # forced, or large enough that the automatic choice takes it (the
            # small layers go to the tiny tile)
            assert ".".join(f[5].split(".")[4:8]) == "1.4.4.4", (label, res)


def test_5x5_7x7_unrolled():
    # 2D 5x5 and 7x7 filters: every matrix-core launch is the unrolled
    # instantiation (template DF = 5, 7), on the GPU parity cases with every
    # tile forced and on larger layers
    import test_parity_gpu as T
    cases = []
    shapes = T.DF5_CASES + [((1, 1), (8, 64, 64, 128, 5)), ((1, 1), (1, 64, 64, 2052, 5)),
                            ((1, 1), (32, 8, 8, 130, 5)), ((1, 1), (8, 64, 64, 70, 7)),
                            ((1, 1), (2, 64, 64, 262, 7)), ((1, 1), (32, 8, 8, 134, 7))]
    dfs = []
    for g, shape in shapes:
        for algo in (P.ALGO_AUTO, P.ALGO_MFMA_WIDE, P.ALGO_MFMA_MEDIUM, P.ALGO_MFMA_NARROW,
                     P.ALGO_MFMA_TINY):
            cases.append(("%s %s %s" % (g, shape, ALGO_NAMES[algo]),
                          conv_line(2, g, *shape, algo)))
            dfs.append(shape[4])
    out = _run_cases(cases, _is_forced_tile)
    for (label, _), res, df in zip(cases, out, dfs):
        f = res.split()
        if int(f[1]) == P.CLIFF_OK:
            assert f[4] == "1" and f[5].startswith("2.4.%d." % df), (label, res)


def test_narrow_10_slots():
    # the narrow tile's 10-slot form (template WCO.WPOS.MW.NW.SLOTS
    # 1.4.2.4.10), taken where a large filter's stage needs more than 8 slots
    import test_parity_gpu as T
    cases = []
    for g, shape in T.NARROW10_CASES + [((1, 1), (8, 64, 64, 130, 7)), ((1, 1), (2, 64, 64, 262, 7))]:
        for algo in (P.ALGO_AUTO, P.ALGO_MFMA_NARROW):
            cases.append(("%s %s %s" % (g, shape, ALGO_NAMES[algo]),
                          conv_line(2, g, *shape, algo)))
    out = _run_cases(cases, lambda line: False)
    for (label, _), res in zip(cases, out):
        f = res.split()
        assert f[4] == "1", (label, res)
        assert ".".join(f[5].split(".")[4:9]) == "1.4.2.4.10", (label, res)


def test_wide_64_position_tile():
    # the 64-position form of the 2D 64-channel wide tile (template
    # WCO.WPOS.MW.NW 4.1.4.4), which the automatic choice takes for small
    # single-image layers
    import test_parity_gpu as T
    cases = [("%s %s" % (g, shape), conv_line(2, g, *shape, P.ALGO_AUTO))
             for g, shape in T.WIDE64_CASES + [((1, 1), (1, 64, 64, 128, 3))]]
    out = _run_cases(cases, lambda line: False)
    for (label, _), res in zip(cases, out):
        f = res.split()
        assert f[4] == "1", (label, res)
        assert ".".join(f[5].split(".")[4:8]) == "4.1.4.4", (label, res)


def test_reciprocal_division():
    # the per-lane divisions of the convolution kernels' staging and fragment
    # offsets go through a reciprocal formed once per workgroup (fdiv in
    # conv_mfma_geom.hpp); the checker compares it with integer division
    out = HC.run(["fastdiv"])
    assert out == ["ok 0 0 0 - -"], out


def act_line(nb, B, C, Pn, act):
    return "act %d %d %d %d %s" % (nb, B, C, Pn, act_field(act))


def test_standalone_activation():
    # the GPU parity shapes (every N_B and mode, P = 1), positions around the
    # 512 per workgroup, the benchmark's activation shapes and the > 2^31
    # element in-place case (the checker walks every workgroup of grids up to
    # 2^15 and counts each output multivector; larger grids are sampled)
    cases = []
    for nb in (2, 4, 8):
        for mode in (P.AGG_LINEAR, P.AGG_SUM, P.AGG_MEAN):
            K = max(1, nb - 1)
            for (B, C, Pn) in ((3, 7, 11), (5, 9, 1), (2, 3, 513), (1, 2, 1024)):
                cases.append(("nb %d mode %d B %d C %d P %d" % (nb, mode, B, C, Pn),
                              act_line(nb, B, C, Pn, (mode, tuple(range(K))))))
    cases.append(("bench linear", act_line(4, 8, 64, 16384, (P.AGG_LINEAR, (0, 1, 2, 3)))))
    cases.append(("bench mean", act_line(8, 8, 64, 39304, (P.AGG_MEAN, tuple(range(8))))))
    cases.append(("> 2^31 elements", act_line(4, 520, 64, 126 * 126,
                                              (P.AGG_LINEAR, (0, 1, 2, 3)))))
    out = _run_cases(cases, lambda line: False)
    for (label, _), res in zip(cases, out):
        assert res.split()[4] == "6", (label, res)  # one activation launch


def test_streamed_linear_layers():
    # the streamed linear kernel (d_image = d_filter = 1, forced or chosen):
    # the GPU tests' widths, rectangular layers and batch sizes (one tile and
    # a ragged last tile), many tiles per wave, the random draws and the
    # benchmark's layers (sampled tiles past 2^15; every wave's A reads)
    import test_linear_stream_gpu as LS
    import test_random_linear_gpu as RL
    cases = []
    S = P.ALGO_MFMA_STREAM

    def add(label, g, B, C_in, C_out, algo, act=None):
        cases.append((label, conv_line(len(g), g, B, C_in, C_out, 1, 1, algo, act)))
    for g, C in LS.WIDTHS:
        nb = 1 << len(g)
        for B in (1, 17, 1000):
            add("width %s C %d B %d" % (g, C, B), g, B, C, C, S)
        add("width %s C %d many tiles" % (g, C), g, (1 << 20) // (C * nb // 32) + 13, C, C, S)
        add("width %s C %d linear gate" % (g, C), g, 5000, C, C, S,
            (P.AGG_LINEAR, tuple(range(nb))))
    for g, C_in, C_out in LS.RECT:
        for B in (37, 1000):
            add("rect %s %d->%d B %d" % (g, C_in, C_out, B), g, B, C_in, C_out, S)
    for (g, C_in, C_out, B, has_bias, act, seed) in RL.draw_layers():
        add("random %s %d->%d B %d" % (g, C_in, C_out, B), g, B, C_in, C_out, P.ALGO_AUTO,
            None if act is None else act)
    for k, B in ((2, 1 << 20), (3, 1 << 19), (1, 1 << 21)):
        g = (1,) * k
        add("benchmark k %d" % k, g, B, 32, 32, P.ALGO_AUTO)
    out = _run_cases(cases, lambda line: False)
    for (label, line), res in zip(cases, out):
        if int(line.split()[2 + int(line.split()[1]) + 5]) == S:
            assert res.split()[4] == "4", (label, res)  # one streamed-linear launch
