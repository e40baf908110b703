"""Parity helpers shared by the GPU tests (tolerances are stated here once).

Attention outputs (bf16) are compared with the float64 oracle on the same
bf16 inputs:
  O     : max |dO| <= 2e-2 and mean |dO| <= 2e-3 (absolute);
  LSE   : max |dLSE| <= 1e-3 (a missing or extra key block moves LSE by ~1e-2);
  O     : relative Frobenius error <= 1e-2;
  grads : for g in dQ, dK, dV with s = max |g_ref|: max |dg| <= 2e-2 s and
          mean |dg| <= 2e-3 s; relative Frobenius error <= 2e-2.
Index and copy outputs are compared bit for bit.
"""
import math

import numpy as np
import torch

O_MAX, O_MEAN, LSE_MAX, O_FRO = 2e-2, 2e-3, 1e-3, 1e-2
G_MAX, G_MEAN, G_FRO = 2e-2, 2e-3, 2e-2


def to_np(t):
    return t.detach().float().cpu().numpy() if isinstance(t, torch.Tensor) else np.asarray(t)


def fro(a, b):
    return float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-30))


def check_out(o_gpu, lse_gpu, O_ref, L_ref, label=""):
    o, l = to_np(o_gpu), to_np(lse_gpu)
    sel = ~np.isnan(O_ref)
    e = np.abs(o[sel] - O_ref[sel])
    assert e.max() <= O_MAX and e.mean() <= O_MEAN, f"{label} O err max {e.max():.3e} mean {e.mean():.3e}"
    assert fro(o[sel], O_ref[sel]) <= O_FRO, f"{label} O fro {fro(o[sel], O_ref[sel]):.3e}"
    lsel = ~np.isnan(L_ref)
    fin = np.isfinite(L_ref[lsel])
    assert np.array_equal(np.isfinite(l[lsel]), fin), f"{label} LSE finiteness differs"
    le = np.abs(l[lsel][fin] - L_ref[lsel][fin])
    if le.size:
        assert le.max() <= LSE_MAX, f"{label} LSE err {le.max():.3e}"
    return float(e.max()), float(e.mean())


def check_grad(g_gpu, g_ref, label="", rows=None):
    g = to_np(g_gpu)
    if rows is not None:
        g, g_ref = g[rows], g_ref[rows]
    sel = ~np.isnan(g_ref)
    g, r = g[sel], g_ref[sel]
    s = max(float(np.abs(r).max()), 1e-30)
    e = np.abs(g - r)
    assert e.max() <= G_MAX * s and e.mean() <= G_MEAN * s, \
        f"{label} grad err max {e.max() / s:.3e} mean {e.mean() / s:.3e} (of max |ref| {s:.3e})"
    assert fro(g, r) <= G_FRO, f"{label} grad fro {fro(g, r):.3e}"
    return float(e.max() / s), float(e.mean() / s)


def block_rows(blocks, block, n):
    """Token rows of the listed blocks."""
    return np.concatenate([np.arange(j * block, min(n, (j + 1) * block)) for j in blocks])


def scale_of(d):
    return 1.0 / math.sqrt(d)


# ---------------------------------------------------------------------------
# Top-K block masks: fp32 scores against the exact (float64) selection
# ---------------------------------------------------------------------------
U32 = 2.0 ** -24


def _gamma(n):
    return n * U32 / (1 - n * U32)


def topk_tolerance(q, k, block):
    """Bound on |S_c(fp32) - S_c(exact)| per entry, for any summation order.

    A pooled entry sums at most `block` exact bf16 values in fp32 and divides
    once: |error| <= gamma_block * mean_t |x_td| + u |pool_d|. The fp32 dot
    product over D terms adds gamma_D sum_d |pq_d pk_d|. The first-order sum
    of these is doubled to cover the second-order terms.
    """
    import oracle
    PQ, PK = np.abs(oracle.block_pool(q, block)), np.abs(oracle.block_pool(k, block))
    AQ = oracle.block_pool(np.abs(to_np64(q)), block)
    AK = oracle.block_pool(np.abs(to_np64(k)), block)
    D = PQ.shape[-1]
    g = _gamma(block)
    mm = lambda a, b: a @ np.swapaxes(b, -1, -2)
    return 2.0 * (g * (mm(AQ, PK) + mm(PQ, AK)) + (2 * U32 + _gamma(D)) * mm(PQ, PK))


def to_np64(t):
    return t.detach().to(torch.float64).cpu().numpy() if isinstance(t, torch.Tensor) else np.asarray(t, np.float64)


def check_topk(mask_gpu, ref_mask, scores, tol, k_keep, label="", prefix=0):
    """Every GPU row keeps min(k_keep, Nk) blocks and is a Top-K of the exact
    scores within `tol`; rows whose exact selection is decided by more than
    the tolerance match the oracle exactly. With `prefix` dense leading
    blocks, their rows and columns must be all ones and the rest is checked
    on the remaining blocks. Returns the decided fraction."""
    m = to_np(mask_gpu).astype(np.uint8) if isinstance(mask_gpu, torch.Tensor) else mask_gpu
    if prefix:
        assert m[..., :prefix, :].all() and m[..., :, :prefix].all(), f"{label} prefix not dense"
        sub = lambda a: a[..., prefix:, prefix:]
        return check_topk(sub(m), sub(ref_mask), sub(scores), sub(tol), k_keep, label)
    nk = m.shape[-1]
    assert set(np.unique(m)) <= {0, 1}, f"{label} mask values {np.unique(m)}"
    assert np.all(m.sum(-1) == min(k_keep, nk)), f"{label} row counts"
    if k_keep >= nk:
        assert m.all()
        return 1.0
    sel, ref = m.astype(bool), ref_mask.astype(bool)
    lo = np.where(sel, scores + tol, np.inf).min(-1)
    hi = np.where(~sel, scores - tol, -np.inf).max(-1)
    bad = lo < hi
    assert not bad.any(), f"{label} {int(bad.sum())} rows are not a Top-K within the fp32 bound"
    decided = np.where(ref, scores - tol, np.inf).min(-1) > np.where(~ref, scores + tol, -np.inf).max(-1)
    diff = (sel != ref).any(-1) & decided
    assert not diff.any(), f"{label} {int(diff.sum())} decided rows differ from the oracle"
    return float(decided.mean())
