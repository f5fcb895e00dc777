"""Times every MFMA tile shape, forced through clifford_conv_nd_algo, beside
the library's automatic choice, on a list of convolutions (one JSON line per
problem): the measurement behind the tile-choice model of the 2D/3D
convolution kernel.

    python -m paper_2507_01040_amd.tile_sweep            # the built-in list
    python -m paper_2507_01040_amd.tile_sweep 2,8,64,64,128,3 3,8,32,32,32,3

A problem is k,B,C_in,C_out,d_image,d_filter (signature (1,)*k, random
inputs).  Each shape is timed with HIP events on the launch stream, median of
18 launches taken in 3 interleaved rounds after 3 warm-ups per round.
"""
import json
import sys

import numpy as np

PROBLEMS = [(2, 8, 48, 48, 96, 3), (2, 32, 64, 64, 32, 3), (2, 8, 16, 16, 128, 3),
            (2, 4, 64, 64, 100, 3), (2, 8, 64, 64, 70, 3), (2, 2, 64, 64, 128, 3),
            (3, 8, 32, 32, 16, 3), (3, 2, 64, 64, 24, 3), (2, 8, 96, 96, 64, 3),
            (2, 16, 32, 32, 64, 3), (3, 4, 16, 16, 24, 3), (2, 8, 64, 64, 40, 3),
            (2, 8, 64, 64, 128, 3), (3, 8, 32, 32, 32, 3), (2, 8, 64, 64, 130, 3),
            (3, 8, 64, 64, 36, 3), (3, 8, 64, 64, 34, 3), (2, 8, 64, 64, 32, 3),
            (2, 8, 64, 64, 66, 3), (3, 8, 32, 32, 18, 3), (3, 4, 64, 64, 18, 3),
            (2, 2, 32, 32, 66, 3), (3, 8, 32, 32, 24, 3), (3, 4, 32, 32, 40, 3)]


def sweep(problems, peak_tflops=157.3):
    import torch
    import paper_2507_01040_amd as P
    algos = {"auto": P.ALGO_AUTO, "wide": P.ALGO_MFMA_WIDE, "medium": P.ALGO_MFMA_MEDIUM,
             "narrow": P.ALGO_MFMA_NARROW, "tiny": P.ALGO_MFMA_TINY}
    for k, B, Ci, Co, d, df in problems:
        g = (1,) * k
        nb = 1 << k
        x = torch.randn((B, Ci) + (d,) * k + (nb,), device="cuda:0")
        w = torch.rand((Ci, Co) + (df,) * k + (nb,), device="cuda:0") / Ci
        do = d - df + 1
        out = torch.empty((B, Co) + (do,) * k + (nb,), device="cuda:0")
        st = int(torch.cuda.current_stream().cuda_stream)
        calls = {n: (lambda a=a: P.clifford_conv_nd_algo(k, g, B, Ci, Co, d, df, x.data_ptr(),
                                                          w.data_ptr(), 0, out.data_ptr(),
                                                          None, st, a))
                 for n, a in algos.items()}
        ok = [n for n in calls if calls[n]() == P.CLIFF_OK]
        torch.cuda.synchronize()
        times = {n: [] for n in ok}
        for _ in range(3):
            for n in ok:
                for _ in range(3):
                    calls[n]()
                ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                      for _ in range(6)]
                for e0, e1 in ev:
                    e0.record()
                    calls[n]()
                    e1.record()
                torch.cuda.synchronize()
                times[n] += [e0.elapsed_time(e1) for e0, e1 in ev]
        flops = 2.0 * B * Co * Ci * nb * nb * df ** k * do ** k
        frac = {n: round(flops / float(np.median(v)) / 1e9 / peak_tflops, 3)
                for n, v in times.items()}
        best = max((v, n) for n, v in frac.items() if n != "auto")
        print(json.dumps({"problem": [k, B, Ci, Co, d, df], "frac_of_peak": frac,
                          "best_forced": best[1],
                          "auto_vs_best": round(frac["auto"] / best[0], 3)}), flush=True)


if __name__ == "__main__":
    probs = [tuple(int(v) for v in a.split(",")) for a in sys.argv[1:]] or PROBLEMS
    sweep(probs)
