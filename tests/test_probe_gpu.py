"""The MFMA throughput probe really multiplies: its per-thread output equals
the closed form of its register-only MFMA chains (A = 1e-3 x thread index,
B = 1e-3 x workgroup index, K = 4, 16 chains, `iters` steps)."""
import numpy as np
import pytest
import torch

import paper_2507_01040_amd as P

pytestmark = pytest.mark.gpu


def test_probe_closed_form():
    n_wg, iters = 6, 5
    out = torch.full((n_wg * 256,), float("nan"), device="cuda:0")
    lib = P.load()
    assert lib.cliffconv_mfma_peak_probe(n_wg, iters, out.data_ptr(), None) == P.CLIFF_OK
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    exp = np.zeros(n_wg * 256)
    for wg in range(n_wg):
        for t in range(256):
            wave, lane = divmod(t, 64)
            base = 64 * wave
            s = 0.0
            for r in range(4):
                i = 4 * (lane // 16) + r          # D row held by this lane
                # D[i][j] = sum_k A[i][k] B[k][j], A[i][k] from thread base + i + 16 k
                s += sum(1e-3 * (base + i + 16 * k) for k in range(4)) * 1e-3 * wg
            exp[wg * 256 + t] = 16 * iters * s
    np.testing.assert_allclose(got, exp, rtol=1e-5, atol=1e-9)
