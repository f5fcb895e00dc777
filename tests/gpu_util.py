"""Helpers of the GPU parity tests: device copies, HIP-path calls through the
C ABI with NaN-prefilled outputs, and the parity measure.

Parity measure: normwise relative error max_i |y_i - r_i| / max_i |r_i|
against the fp64 oracle, gated at 1e-4 (fp32 arithmetic; the derivation of
the bound is in the test module docstrings).  Beside it every parity check
reports, without gating on it, the element-wise relative error
max_i |y_i - r_i| / |r_i| over the outputs with |r_i| >= 1e-3 max |r|, so that
an error confined to small outputs (a saturated gate, one bad tile of
near-zero values) shows in the message even when the normwise figure hides it.
"""
import numpy as np
import torch

import paper_2507_01040_amd as P

TOL = 1e-4


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def normwise(y: np.ndarray, r: np.ndarray) -> float:
    y = np.asarray(y, np.float64)
    r = np.asarray(r, np.float64)
    assert y.shape == r.shape, (y.shape, r.shape)
    assert np.all(np.isfinite(y)), "non-finite values in GPU output"
    den = max(float(np.max(np.abs(r))), 1e-30)
    return float(np.max(np.abs(y - r))) / den


ELEM_FLOOR = 1e-3


def elementwise(y: np.ndarray, r: np.ndarray, floor: float = ELEM_FLOOR) -> float:
    """max |y - r| / |r| over the outputs with |r| >= floor * max |r|."""
    y = np.asarray(y, np.float64)
    r = np.asarray(r, np.float64)
    assert y.shape == r.shape, (y.shape, r.shape)
    ar = np.abs(r)
    sel = ar >= floor * max(float(np.max(ar)) if ar.size else 0.0, 1e-30)
    if not np.any(sel):
        return 0.0
    return float(np.max(np.abs(y[sel] - r[sel]) / ar[sel]))


def parity_errors(y, r):
    """(normwise, element-wise) relative errors of y against the oracle r."""
    return normwise(y, r), elementwise(y, r)


def assert_parity(y, r, tol=TOL, what=""):
    e, el = parity_errors(y, r)
    assert e <= tol, "%s normwise error %.3e > %.1e (element-wise %.3e over |r| >= %.0e max|r|)" % (
        what, e, tol, el, ELEM_FLOOR)
    return e


def assert_parity_report(y, r, tol=TOL, what=""):
    """assert_parity, returning (normwise, element-wise) and printing both."""
    e, el = parity_errors(y, r)
    assert e <= tol, "%s normwise error %.3e > %.1e (element-wise %.3e over |r| >= %.0e max|r|)" % (
        what, e, tol, el, ELEM_FLOOR)
    print("%s: normwise %.3e (gate %.0e), element-wise %.3e over |r| >= %.0e max|r|, %d outputs"
          % (what, e, tol, el, ELEM_FLOOR, np.asarray(r).size), flush=True)
    return e, el


def gpu_conv(g, x, f, b, act=None, algo=P.ALGO_AUTO, expect=P.CLIFF_OK,
             xt=None, ft=None, bt=None):
    """Runs the HIP convolution on numpy inputs; returns the output as
    numpy (or None when the call returned `expect` != OK)."""
    k = len(g)
    xt = dev(x) if xt is None else xt
    ft = dev(f) if ft is None else ft
    bt = (dev(b) if b is not None else None) if bt is None else bt
    B, C_in, d_image = x.shape[0], x.shape[1], x.shape[2]
    C_out, d_filter = f.shape[1], f.shape[2]
    d_out = d_image - d_filter + 1
    out = torch.full((B, C_out) + (d_out,) * k + (1 << k,), float("nan"),
                     dtype=torch.float32, device="cuda:0")
    desc = None
    keep = []
    if act is not None:
        mode, blades, aw, ab = act
        awt = dev(aw) if aw is not None else None
        abt = dev(ab) if ab is not None else None
        keep += [awt, abt]
        desc = P.make_act_desc(mode, blades, awt.data_ptr() if awt is not None else 0,
                               abt.data_ptr() if abt is not None else 0)
    st = P.clifford_conv_nd_algo(
        k, g, B, C_in, C_out, d_image, d_filter, xt.data_ptr(), ft.data_ptr(),
        bt.data_ptr() if bt is not None else 0, out.data_ptr(), desc,
        int(torch.cuda.current_stream().cuda_stream), algo)
    torch.cuda.synchronize()
    assert st == expect, (P.STATUS_NAMES.get(st, st), P.STATUS_NAMES.get(expect))
    if st != P.CLIFF_OK:
        return None
    return out.cpu().numpy()


def gpu_act(x, mode, blades, aw=None, ab=None, inplace=False):
    B, C, nb = x.shape[0], x.shape[1], x.shape[-1]
    Pn = int(np.prod(x.shape[2:-1])) if x.ndim > 3 else 1
    xt = dev(x)
    out = xt if inplace else torch.full_like(xt, float("nan"))
    awt = dev(aw) if aw is not None else None
    abt = dev(ab) if ab is not None else None
    desc = P.make_act_desc(mode, blades, awt.data_ptr() if awt is not None else 0,
                           abt.data_ptr() if abt is not None else 0)
    st = P.multivector_act(nb, B, C, Pn, desc, xt.data_ptr(), out.data_ptr(),
                           int(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert st == P.CLIFF_OK, P.STATUS_NAMES.get(st, st)
    return out.cpu().numpy()
