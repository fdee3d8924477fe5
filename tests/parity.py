"""Comparison rules for GPU-vs-oracle parity.

State: max relative error = max |g - o| / max |o| over all cells and channels;
bound 1e-3 for fp32 storage, 1e-2 for fp16 storage.
Readout: agreement >= 0.9999 (fp32) / 0.999 (fp16) as a rate over the
compared cells: on N cells at most ceil((1 - rate) N) disagreements (one on a
case of fewer than 10^4 cells, where the rate allows no whole cell), and every
disagreeing cell must be a near tie of the oracle's last two channels (margin
within the state bound), since there the argmax is not determined by the
method to better than rounding.
Input channels, masks and indices: bit-exact.
"""
import numpy as np

STATE_TOL = {"f32": 1e-3, "f16": 1e-2}
SEG_AGREE = {"f32": 0.9999, "f16": 0.999}


def to_np(t):
    return t.detach().cpu().numpy()


def max_rel_err(got, ref):
    g = np.asarray(got, dtype=np.float64)
    o = np.asarray(ref, dtype=np.float64)
    scale = float(np.max(np.abs(o))) if o.size else 0.0
    diff = float(np.max(np.abs(g - o))) if o.size else 0.0
    return diff / scale if scale > 0 else diff


def elementwise_rel_err(got, ref, floor=1e-6):
    """max over cells and channels of |g - o| / max(|o|, floor * max |o|): the
    elementwise companion of max_rel_err (reported, not bounded)."""
    g = np.asarray(got, dtype=np.float64)
    o = np.asarray(ref, dtype=np.float64)
    if not o.size:
        return 0.0
    den = np.maximum(np.abs(o), floor * float(np.max(np.abs(o))))
    den[den == 0] = 1.0
    return float(np.max(np.abs(g - o) / den))


def assert_state_close(got, ref, dtype: str, tol=None, what="state"):
    tol = STATE_TOL[dtype] if tol is None else tol
    assert np.all(np.isfinite(np.asarray(got, dtype=np.float64))), f"{what}: non-finite values"
    err = max_rel_err(got, ref)
    assert err <= tol, f"{what}: max relative error {err:.3e} > {tol:.1e}"
    return err


def assert_seg_close(got_seg, ref_seg, ref_state, dtype: str, min_agree=None, what="seg"):
    min_agree = SEG_AGREE[dtype] if min_agree is None else min_agree
    got_seg = np.asarray(got_seg)
    ref_seg = np.asarray(ref_seg)
    assert got_seg.shape == ref_seg.shape
    bad = got_seg != ref_seg
    agree = 1.0 - float(np.mean(bad)) if bad.size else 1.0
    o = np.asarray(ref_state, dtype=np.float64)
    margin = np.abs(o[..., -1] - o[..., -2])
    scale = float(np.max(np.abs(o))) if o.size else 0.0
    not_ties = bad & (margin > 2 * STATE_TOL[dtype] * scale)
    assert not np.any(not_ties), f"{what}: {int(not_ties.sum())} clear argmax disagreements"
    allowed = int(np.ceil((1.0 - min_agree) * bad.size - 1e-9))
    assert int(bad.sum()) <= allowed, (f"{what}: agreement {agree:.6f} < {min_agree} "
                                      f"({int(bad.sum())} of {bad.size} cells, {allowed} allowed)")
    return agree
