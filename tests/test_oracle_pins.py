"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-calls the oracle's own formula or library routine: each pin
is an independent route (a different library routine, a closed form worked
out by hand, brute force over scalars, finite differences, or an invariant),
chosen so that a dropped term, a wrong sign or index, or a transposed operand
in the oracle fails at least one of them.
"""
import math

import numpy as np
import pytest
import scipy.sparse as sp
import torch

import oracle
import workloads as W

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


# ---------------------------------------------------------------------------
# Compaction / gather / scatter (Sec. 3.2)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("L,p", [(0, 0.5), (1, 1.0), (1, 0.0), (777, 0.0), (777, 1.0),
                                 (4097, 0.3), (20000, 0.5), (65537, 0.02)])
def test_compact_matches_flatnonzero(L, p):
    rng = np.random.default_rng(L)
    mask = (rng.random(L) < p).astype(np.uint8) * rng.integers(1, 256, L).astype(np.uint8)
    kept, inv, n = oracle.compact(mask)
    ref = np.flatnonzero(mask)
    assert n == ref.size
    assert np.array_equal(kept, ref.astype(np.int32))
    # inverse map: dropped positions are -1, kept positions invert kept_idx
    assert np.all(inv[mask == 0] == -1)
    assert np.array_equal(inv[ref], np.arange(n, dtype=np.int32))


def test_compact_workload_masks():
    for name in ("tiny", "c512"):
        inst = W.make(W.WORKLOADS[name], with_qkv=False)
        kept, inv, n = oracle.compact(inst.fg_mask)
        assert n == inst.n_kept == int(inst.fg_mask.astype(bool).sum())
        assert np.all(np.diff(kept) > 0)


def test_gather_scatter_against_boolean_indexing():
    rng = np.random.default_rng(7)
    L, C = 3000, 40
    mask = (rng.random(L) < 0.37).astype(np.uint8)
    # random 16-bit patterns, NaNs included: compared bitwise
    x = rng.integers(0, 1 << 16, size=(L, C), dtype=np.uint16)
    kept, _, n = oracle.compact(mask)
    packed = oracle.gather(x, kept)
    assert np.array_equal(packed, x[mask.astype(bool)])
    prefill = rng.integers(0, 1 << 16, size=(L, C), dtype=np.uint16)
    out = oracle.scatter(packed, kept, prefill)
    assert np.array_equal(out[mask.astype(bool)], x[mask.astype(bool)])
    assert np.array_equal(out[~mask.astype(bool)], prefill[~mask.astype(bool)])


# ---------------------------------------------------------------------------
# Block index (Eq. 7, the sets S_i of Eq. 8)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("B,H,Nq,Nk,p", [(1, 1, 1, 1, 1.0), (1, 3, 7, 7, 0.3),
                                         (2, 2, 13, 9, 0.5), (1, 4, 33, 33, 0.0),
                                         (1, 2, 50, 50, 1.0)])
def test_block_index_matches_scipy(B, H, Nq, Nk, p):
    rng = np.random.default_rng(B * 1000 + Nq)
    m = (rng.random((B, H, Nq, Nk)) < p).astype(np.uint8)
    rowptr, cols, colptr, rows = oracle.block_index(m)
    # row lists: CSR of each (b, h) slab, offsets chained across slabs
    r_ptr, r_idx, c_ptr, c_idx = [0], [], [0], []
    for b in range(B):
        for h in range(H):
            csr = sp.csr_matrix(m[b, h])
            csr.sort_indices()
            r_ptr.extend((csr.indptr[1:] + r_ptr[-1]).tolist())
            r_idx.extend(csr.indices.tolist())
            csc = sp.csc_matrix(m[b, h])
            csc.sort_indices()
            c_ptr.extend((csc.indptr[1:] + c_ptr[-1]).tolist())
            c_idx.extend(csc.indices.tolist())
    assert np.array_equal(rowptr, np.array(r_ptr, dtype=np.int32))
    assert np.array_equal(cols, np.array(r_idx, dtype=np.int32))
    assert np.array_equal(colptr, np.array(c_ptr, dtype=np.int32))
    assert np.array_equal(rows, np.array(c_idx, dtype=np.int32))
    assert rowptr[-1] == colptr[-1] == int(m.astype(bool).sum())


def test_block_index_brute_force_tiny():
    m = np.array([[[[1, 0, 1], [0, 0, 0], [1, 1, 1]]]], dtype=np.uint8)
    rowptr, cols, colptr, rows = oracle.block_index(m)
    assert rowptr.tolist() == [0, 2, 2, 5]
    assert cols.tolist() == [0, 2, 0, 1, 2]
    assert colptr.tolist() == [0, 2, 3, 5]
    assert rows.tolist() == [0, 2, 2, 0, 2]


def test_synthetic_block_mask_row_counts():
    # Eq. 7 keeps floor(rho * N_k) key blocks per row; the synthetic stand-in
    # keeps the diagonal plus that many others.
    rng = np.random.default_rng(0)
    for rho, nk, koff in (("0.1", 624, 62), ("0.3", 50, 15), ("0.4", 6, 2), ("0.2", 177, 35),
                          ("0.05", 603, 30)):
        assert W.kept_off_diagonal(rho, nk) == koff
        bm = W.block_mask(1, 3, nk, nk, rho, rng)
        assert np.all(bm.sum(-1) == koff + 1)
        assert np.all(bm[0, :, np.arange(nk), np.arange(nk)] == 1)


# ---------------------------------------------------------------------------
# Forward (Eq. 5, Eq. 8)
# ---------------------------------------------------------------------------

def _expand_mask(bm, n, block):
    """Token-level boolean mask [B, H, N, N] from a block mask."""
    tok = np.arange(n) // block
    return bm[:, :, tok][:, :, :, tok].astype(bool)


def _sdpa(q, k, v, tokmask=None):
    """torch's scaled_dot_product_attention in float64 on [B, N, H, D] inputs."""
    t = lambda a: torch.as_tensor(a, dtype=torch.float64).permute(0, 2, 1, 3)
    am = None if tokmask is None else torch.as_tensor(tokmask)
    o = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), attn_mask=am)
    return o.permute(0, 2, 1, 3).numpy()


def test_fwd_hand_worked_example():
    """Three tokens, d = 2, block 2 (a short last block). Scores, softmax and
    outputs below are worked out by hand from Eq. 5 and Eq. 8."""
    s2 = math.sqrt(2.0)
    q = np.array([[s2 * math.log(3.0), 0.0], [0.0, 0.0], [0.0, 0.0]])
    k = np.array([[1.0, 0.0], [0.0, 1.0], [10.0, 10.0]])
    v = np.array([[1.0, 2.0], [5.0, -2.0], [100.0, 100.0]])
    bm = np.array([[[[1, 0], [1, 1]]]], dtype=np.uint8)
    O, L = oracle.bsattn_fwd(q[None, :, None], k[None, :, None], v[None, :, None], bm, 2,
                             1.0 / s2)
    # row 0: scores (ln 3, 0) -> P = (3/4, 1/4); key 2 lies in a skipped block
    assert np.allclose(O[0, 0, 0], [2.0, 1.0], atol=1e-14)
    assert math.isclose(L[0, 0, 0], math.log(4.0), abs_tol=1e-14)
    # row 1: zero query -> uniform over keys 0, 1
    assert np.allclose(O[0, 1, 0], [3.0, 0.0], atol=1e-14)
    assert math.isclose(L[0, 0, 1], math.log(2.0), abs_tol=1e-14)
    # row 2: zero query, both blocks selected -> uniform over keys 0, 1, 2
    assert np.allclose(O[0, 2, 0], [106.0 / 3.0, 100.0 / 3.0], atol=1e-12)
    assert math.isclose(L[0, 0, 2], math.log(3.0), abs_tol=1e-14)


def test_bwd_hand_worked_example():
    """Same three tokens, dO = e_0 on row 0 only. Hand derivation:
    dP = (v_0[0], v_1[0]) = (1, 5); delta = 3/4 + 5/4 = 2;
    dS = P o (dP - delta) = (-3/4, 3/4); dQ_0 = (1/sqrt2) * (-3/4 k_0 + 3/4 k_1);
    dK_c = (1/sqrt2) dS_c q_0; dV_c = P_c dO_0."""
    s2 = math.sqrt(2.0)
    q = np.array([[s2 * math.log(3.0), 0.0], [0.0, 0.0], [0.0, 0.0]])
    k = np.array([[1.0, 0.0], [0.0, 1.0], [10.0, 10.0]])
    v = np.array([[1.0, 2.0], [5.0, -2.0], [100.0, 100.0]])
    do = np.array([[1.0, 0.0], [0.0, 0.0], [0.0, 0.0]])
    bm = np.array([[[[1, 0], [1, 1]]]], dtype=np.uint8)
    ex = lambda a: a[None, :, None]
    dQ, dK, dV = oracle.bsattn_bwd(ex(q), ex(k), ex(v), ex(do), bm, 2, 1.0 / s2)
    c = 3.0 / (4.0 * s2)
    assert np.allclose(dQ[0, :, 0], [[-c, c], [0, 0], [0, 0]], atol=1e-14)
    l3 = math.log(3.0)
    assert np.allclose(dK[0, :, 0], [[-0.75 * l3, 0], [0.75 * l3, 0], [0, 0]], atol=1e-14)
    assert np.allclose(dV[0, :, 0], [[0.75, 0], [0.25, 0], [0, 0]], atol=1e-14)


@pytest.mark.parametrize("n,block,H,D", [(64, 16, 2, 8), (70, 16, 1, 16), (130, 64, 2, 32)])
def test_fwd_all_ones_is_dense_sdpa(n, block, H, D):
    rng = np.random.default_rng(n)
    q, k, v = (rng.standard_normal((1, n, H, D)) for _ in range(3))
    nb = -(-n // block)
    O, L = oracle.bsattn_fwd(q, k, v, np.ones((1, H, nb, nb), np.uint8), block,
                             1.0 / math.sqrt(D))
    assert np.allclose(O, _sdpa(q, k, v), atol=1e-12, rtol=1e-12)
    s = torch.einsum("bnhd,bmhd->bhnm", torch.tensor(q), torch.tensor(k)) / math.sqrt(D)
    assert np.allclose(L, torch.logsumexp(s, dim=-1).numpy(), atol=1e-12)


@pytest.mark.parametrize("seed,n,block,H,D,density", [(1, 70, 16, 2, 16, 0.4),
                                                      (2, 200, 32, 3, 8, 0.25),
                                                      (3, 97, 8, 1, 4, 0.6)])
def test_fwd_masked_matches_sdpa_boolean_mask(seed, n, block, H, D, density):
    rng = np.random.default_rng(seed)
    q, k, v = (rng.standard_normal((1, n, H, D)) * 2.0 for _ in range(3))
    nb = -(-n // block)
    bm = (rng.random((1, H, nb, nb)) < density).astype(np.uint8)
    bm[:, :, np.arange(nb), np.arange(nb)] = 1
    O, _ = oracle.bsattn_fwd(q, k, v, bm, block, 1.0 / math.sqrt(D))
    ref = _sdpa(q, k, v, _expand_mask(bm, n, block))
    assert np.allclose(O, ref, atol=1e-12, rtol=1e-12)


def test_fwd_diagonal_only_is_blockwise_dense():
    rng = np.random.default_rng(11)
    n, block, H, D = 90, 32, 2, 8
    q, k, v = (rng.standard_normal((1, n, H, D)) for _ in range(3))
    nb = -(-n // block)
    bm = np.zeros((1, H, nb, nb), np.uint8)
    bm[:, :, np.arange(nb), np.arange(nb)] = 1
    O, _ = oracle.bsattn_fwd(q, k, v, bm, block, 1.0 / math.sqrt(D))
    for i in range(nb):
        sl = slice(i * block, min(n, (i + 1) * block))
        assert np.allclose(O[:, sl], _sdpa(q[:, sl], k[:, sl], v[:, sl]), atol=1e-12)


def test_fwd_brute_force_scalar_loops_with_empty_row():
    """Pure-Python scalar loops over every (row, key) pair, ragged tail and an
    empty block row included."""
    rng = np.random.default_rng(5)
    n, block, D = 23, 5, 3
    q, k, v = (rng.standard_normal((1, n, 1, D)) for _ in range(3))
    nb = -(-n // block)
    bm = (rng.random((1, 1, nb, nb)) < 0.5).astype(np.uint8)
    bm[0, 0, 2, :] = 0                     # query block 2 attends to nothing
    bm[0, 0, 0, nb - 1] = 1                # a short key block is selected
    scale = 0.7
    O, L = oracle.bsattn_fwd(q, k, v, bm, block, scale)
    for r in range(n):
        allowed = [c for c in range(n) if bm[0, 0, r // block, c // block]]
        if not allowed:
            assert np.all(O[0, r, 0] == 0) and L[0, 0, r] == -np.inf
            continue
        s = {c: scale * sum(q[0, r, 0, d] * k[0, c, 0, d] for d in range(D)) for c in allowed}
        mx = max(s.values())
        z = sum(math.exp(s[c] - mx) for c in allowed)
        for d in range(D):
            o = sum(math.exp(s[c] - mx) * v[0, c, 0, d] for c in allowed) / z
            assert math.isclose(O[0, r, 0, d], o, rel_tol=1e-12, abs_tol=1e-12)
        assert math.isclose(L[0, 0, r], mx + math.log(z), rel_tol=1e-13)


def test_fwd_zero_query_is_mean_of_allowed_values():
    rng = np.random.default_rng(9)
    n, block, H, D = 77, 16, 2, 8
    q = np.zeros((1, n, H, D))
    k, v = (rng.standard_normal((1, n, H, D)) for _ in range(2))
    nb = -(-n // block)
    bm = (rng.random((1, H, nb, nb)) < 0.5).astype(np.uint8)
    bm[:, :, np.arange(nb), np.arange(nb)] = 1
    O, L = oracle.bsattn_fwd(q, k, v, bm, block, 0.3)
    for h in range(H):
        for r in range(n):
            cols = [c for c in range(n) if bm[0, h, r // block, c // block]]
            assert np.allclose(O[0, r, h], v[0, cols, h].mean(axis=0), atol=1e-13)
            assert math.isclose(L[0, h, r], math.log(len(cols)), rel_tol=1e-13)


def test_fwd_invariants_unit_values_and_peaky_scores():
    rng = np.random.default_rng(3)
    n, block, H, D = 150, 32, 2, 16
    q = rng.standard_normal((1, n, H, D)) * 40.0    # large scores: online-max stress
    k = rng.standard_normal((1, n, H, D))
    nb = -(-n // block)
    bm = (rng.random((1, H, nb, nb)) < 0.4).astype(np.uint8)
    bm[:, :, np.arange(nb), np.arange(nb)] = 1
    O, L = oracle.bsattn_fwd(q, k, np.ones((1, n, H, D)), bm, block, 0.25)
    assert np.allclose(O, 1.0, atol=1e-12)        # rows of P sum to one
    assert np.all(np.isfinite(L))
    v = rng.standard_normal((1, n, H, D))
    O2, _ = oracle.bsattn_fwd(q, k, v, bm, block, 0.25)
    tq = torch.tensor(q * 0.25 / (1 / math.sqrt(D)))   # SDPA applies 1/sqrt(D)
    ref = _sdpa(tq.numpy(), k, v, _expand_mask(bm, n, block))
    assert np.allclose(O2, ref, atol=1e-10)


def test_dropped_tokens_never_influence_kept_outputs():
    """Background rows of the full sequence set to NaN: after dropping, every
    kept output is finite and identical to the run with other background."""
    inst = W.make(W.WORKLOADS["tiny"], with_qkv=False)
    L, H, D = inst.wl.seq_len, 2, 16
    rng = np.random.default_rng(1)
    full = rng.standard_normal((L, 3, H, D))
    kept, _, n = oracle.compact(inst.fg_mask)
    a = full.copy()
    a[inst.fg_mask == 0] = np.nan
    b = full.copy()
    b[inst.fg_mask == 0] = 1e6
    nb = -(-n // 64)
    bm = np.ones((1, H, nb, nb), np.uint8)
    outs = []
    for x in (a, b):
        p = oracle.gather(x, kept)
        O, _ = oracle.bsattn_fwd(p[None, :, 0], p[None, :, 1], p[None, :, 2], bm, 64, 0.25)
        outs.append(O)
    assert np.all(np.isfinite(outs[0]))
    assert np.array_equal(outs[0], outs[1])


# ---------------------------------------------------------------------------
# Backward (gradient of Eq. 8, mask constant)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed,n,block,H,D,density", [(1, 70, 16, 2, 8, 0.4),
                                                      (4, 129, 32, 1, 16, 0.3)])
def test_bwd_matches_torch_autograd(seed, n, block, H, D, density):
    rng = np.random.default_rng(seed)
    q, k, v, do = (rng.standard_normal((1, n, H, D)) for _ in range(4))
    nb = -(-n // block)
    bm = (rng.random((1, H, nb, nb)) < density).astype(np.uint8)
    bm[:, :, np.arange(nb), np.arange(nb)] = 1
    tq, tk, tv = (torch.tensor(a, requires_grad=True) for a in (q, k, v))
    t = lambda a: a.permute(0, 2, 1, 3)
    o = torch.nn.functional.scaled_dot_product_attention(
        t(tq), t(tk), t(tv), attn_mask=torch.as_tensor(_expand_mask(bm, n, block)))
    o.permute(0, 2, 1, 3).backward(torch.tensor(do))
    dQ, dK, dV = oracle.bsattn_bwd(q, k, v, do, bm, block, 1.0 / math.sqrt(D))
    assert np.allclose(dQ, tq.grad.numpy(), atol=1e-12)
    assert np.allclose(dK, tk.grad.numpy(), atol=1e-12)
    assert np.allclose(dV, tv.grad.numpy(), atol=1e-12)


def test_fp32_arithmetic_option_matches_fp32_sdpa_and_autograd():
    """The float32 option (CPU-baseline timing only) against torch's float32
    SDPA and autograd on bf16-exact inputs: same definition, fp32 rounding."""
    rng = np.random.default_rng(9)
    n, block, H, D = 150, 32, 2, 16
    q, k, v, do = (torch.tensor(rng.standard_normal((1, n, H, D)), dtype=torch.float32)
                   .to(torch.bfloat16) for _ in range(4))
    nb = -(-n // block)
    bm = (rng.random((1, H, nb, nb)) < 0.4).astype(np.uint8)
    bm[:, :, np.arange(nb), np.arange(nb)] = 1
    tq, tk, tv = (x.float().clone().requires_grad_(True) for x in (q, k, v))
    t = lambda a: a.permute(0, 2, 1, 3)
    o = torch.nn.functional.scaled_dot_product_attention(
        t(tq), t(tk), t(tv), attn_mask=torch.as_tensor(_expand_mask(bm, n, block)))
    o.permute(0, 2, 1, 3).backward(do.float())
    sc = 1.0 / math.sqrt(D)
    O, LSE = oracle.bsattn_fwd(q, k, v, bm, block, sc, dtype=np.float32)
    dQ, dK, dV = oracle.bsattn_bwd(q, k, v, do, bm, block, sc, dtype=np.float32)
    assert O.dtype == np.float32 and dQ.dtype == np.float32
    assert np.allclose(O, o.permute(0, 2, 1, 3).detach().numpy(), atol=2e-6, rtol=1e-5)
    for got, ref in ((dQ, tq.grad), (dK, tk.grad), (dV, tv.grad)):
        assert np.allclose(got, ref.numpy(), atol=2e-5, rtol=1e-4)
    O64, LSE64 = oracle.bsattn_fwd(q, k, v, bm, block, sc)
    assert np.abs(LSE - LSE64).max() < 1e-5


def test_bwd_central_finite_differences():
    rng = np.random.default_rng(21)
    n, block, H, D = 19, 6, 1, 3
    q, k, v, do = (rng.standard_normal((1, n, H, D)) for _ in range(4))
    nb = -(-n // block)
    bm = (rng.random((1, H, nb, nb)) < 0.5).astype(np.uint8)
    bm[0, 0, 1, :] = 0                          # empty row: zero gradients
    bm[0, 0, 0, 0] = bm[0, 0, 3, 3] = 1
    scale = 0.8

    def loss(qq, kk, vv):
        O, _ = oracle.bsattn_fwd(qq, kk, vv, bm, block, scale)
        return float((O * do).sum())

    dQ, dK, dV = oracle.bsattn_bwd(q, k, v, do, bm, block, scale)
    h = 1e-5
    for grad, which in ((dQ, 0), (dK, 1), (dV, 2)):
        for idx in np.ndindex(q.shape):
            args = [q.copy(), k.copy(), v.copy()]
            args[which][idx] += h
            up = loss(*args)
            args[which][idx] -= 2 * h
            dn = loss(*args)
            assert abs((up - dn) / (2 * h) - grad[idx]) < 1e-7, (which, idx)
    assert np.all(dQ[0, block:2 * block] == 0)


def test_bwd_invariants_sum_dk_zero_sum_dv_equals_sum_do():
    rng = np.random.default_rng(8)
    n, block, H, D = 200, 32, 3, 8
    q, k, v, do = (rng.standard_normal((1, n, H, D)) for _ in range(4))
    nb = -(-n // block)
    bm = (rng.random((1, H, nb, nb)) < 0.3).astype(np.uint8)
    bm[:, :, np.arange(nb), np.arange(nb)] = 1
    dQ, dK, dV = oracle.bsattn_bwd(q, k, v, do, bm, block, 0.35)
    assert np.allclose(dK.sum(axis=1), 0.0, atol=1e-11)
    assert np.allclose(dV.sum(axis=1), do.sum(axis=1), atol=1e-11)


# ---------------------------------------------------------------------------
# Top-K block selection (Sec. 3.3, Eq. 6 and Eq. 7)
# ---------------------------------------------------------------------------

def _hand_example():
    """N = 5 tokens, block 2 (blocks {0,1}, {2,3} and the short {4}), H = 1, D = 2.

    pool(Q): (2,0),(0,2) -> (1,1);  (4,0),(2,2) -> (3,1);  (0,-1) -> (0,-1)
    pool(K): (2,0),(2,0) -> (2,0);  (0,2),(0,0) -> (0,1);  (2,2)  -> (2,2)
    S_c = pool(Q) pool(K)^T = [[2, 1, 4], [6, 1, 8], [0, -1, -2]] (worked by hand).
    Averaging the short block over the block size instead of its one token
    would give pool(K)_2 = (1,1) and row 0 = [2, 1, 2]; a transposed S_c would
    give row 0 = [2, 6, 0]: both change the Top-1 answer below.
    """
    q = np.array([[2, 0], [0, 2], [4, 0], [2, 2], [0, -1]], dtype=np.float64)
    k = np.array([[2, 0], [2, 0], [0, 2], [0, 0], [2, 2]], dtype=np.float64)
    return q.reshape(1, 5, 1, 2), k.reshape(1, 5, 1, 2)


def test_topk_hand_worked_example():
    q, k = _hand_example()
    mask1, sc = oracle.topk_block_mask(q, k, 2, 1)
    assert np.array_equal(sc[0, 0], [[2, 1, 4], [6, 1, 8], [0, -1, -2]])
    assert np.array_equal(mask1[0, 0], [[0, 0, 1], [0, 0, 1], [1, 0, 0]])
    mask2, _ = oracle.topk_block_mask(q, k, 2, 2)
    assert np.array_equal(mask2[0, 0], [[1, 0, 1], [1, 0, 1], [1, 1, 0]])
    mask3, _ = oracle.topk_block_mask(q, k, 2, 3)
    assert mask3.all()


def test_topk_ties_go_to_the_lower_block():
    # pool(K) equal for blocks 0 and 1 (and 3): every row has an exact tie at its top
    q = np.ones((1, 8, 1, 2))
    k = np.array([[1, 0], [1, 0], [0, 1], [1, 0], [0, 0], [0, 0], [1, 0], [0, 1]],
                 dtype=np.float64).reshape(1, 8, 1, 2)
    mask, sc = oracle.topk_block_mask(q, k, 2, 1)
    assert np.array_equal(sc[0, 0, 0], [1, 1, 0, 1])
    assert np.array_equal(mask[0, 0], np.tile([1, 0, 0, 0], (4, 1)))
    mask, _ = oracle.topk_block_mask(q, k, 2, 2)
    assert np.array_equal(mask[0, 0], np.tile([1, 1, 0, 0], (4, 1)))


@pytest.mark.parametrize("seed,n,block,H,D,kk", [(1, 37, 8, 2, 4, 2), (2, 64, 16, 1, 3, 1),
                                                   (3, 50, 8, 3, 5, 4), (4, 9, 4, 1, 2, 5)])
def test_topk_brute_force(seed, n, block, H, D, kk):
    """Scalar loops: pooled means token by token, dot products term by term, and
    the rank definition of Top-K (j is kept iff fewer than kk entries beat it,
    an entry beating j when larger, or equal with a lower index). Small
    integer inputs make exact ties common."""
    rng = np.random.default_rng(seed)
    q = rng.integers(-2, 3, (1, n, H, D)).astype(np.float64)
    k = rng.integers(-2, 3, (1, n, H, D)).astype(np.float64)
    nb = -(-n // block)
    mask, sc = oracle.topk_block_mask(q, k, block, kk)
    for h in range(H):
        pq = [[0.0] * D for _ in range(nb)]
        pk = [[0.0] * D for _ in range(nb)]
        for j in range(nb):
            toks = list(range(j * block, min(n, (j + 1) * block)))
            for d in range(D):
                pq[j][d] = sum(q[0, t, h, d] for t in toks) / len(toks)
                pk[j][d] = sum(k[0, t, h, d] for t in toks) / len(toks)
        for i in range(nb):
            row = [sum(pq[i][d] * pk[j][d] for d in range(D)) for j in range(nb)]
            assert np.allclose(sc[0, h, i], row, rtol=0, atol=1e-12)
            for j in range(nb):
                beaten_by = sum(1 for jj in range(nb)
                                if row[jj] > row[j] or (row[jj] == row[j] and jj < j))
                assert mask[0, h, i, j] == (1 if beaten_by < kk else 0), (h, i, j)


def test_topk_invariants():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((2, 300, 3, 16))
    k = rng.standard_normal((2, 300, 3, 16))
    block, nb = 32, 10
    for kk in (1, 3, 9):
        mask, sc = oracle.topk_block_mask(q, k, block, kk)
        assert np.all(mask.sum(axis=-1) == kk)
        # Top-1 is the first maximum (library argmax)
        if kk == 1:
            assert np.array_equal(mask.argmax(axis=-1), sc.argmax(axis=-1))
        # the kept scores are never below a dropped score of the same row
        lo = np.where(mask == 1, sc, np.inf).min(axis=-1)
        hi = np.where(mask == 0, sc, -np.inf).max(axis=-1)
        assert np.all(lo >= hi)
        # a positive power-of-two scale of Q (exact) changes no selection
        m4, _ = oracle.topk_block_mask(4.0 * q, k, block, kk)
        assert np.array_equal(m4, mask)
    full, _ = oracle.topk_block_mask(q, k, block, nb + 5)
    assert full.all()
    # block_pool of a block filled with one vector is that vector, short last block included
    x = np.repeat(rng.standard_normal((1, 10, 2, 4)), 32, axis=1)[:, :300]
    assert np.allclose(oracle.block_pool(x, 32)[0, :, :, :].transpose(1, 0, 2), x[0, ::32], atol=1e-12)


# ---------------------------------------------------------------------------
# Foreground-restricted sampling and training (Sec. 3.2, Eq. 3 and Eq. 4)
# ---------------------------------------------------------------------------

def test_euler_hand_example_and_untouched_background():
    # L = 4 positions, C = 2, positions 1 and 3 retained; dt = t_prev - t_curr = -0.25
    z = np.array([[1.0, 2.0], [3.0, 4.0], [5.0, 6.0], [7.0, 8.0]])
    v = np.array([[4.0, -8.0], [2.0, 0.0]])
    out = oracle.euler_update_fg(z, v, np.array([1, 3]), -0.25)
    assert np.array_equal(out, [[1, 2], [2, 6], [5, 6], [6.5, 8]])
    assert np.array_equal(z, [[1, 2], [3, 4], [5, 6], [7, 8]])   # input not modified


def test_euler_composes_and_matches_torch_index_add():
    rng = np.random.default_rng(3)
    L, C = 500, 16
    z = rng.standard_normal((L, C))
    mask = rng.random(L) < 0.4
    kept = np.flatnonzero(mask)
    v1, v2 = rng.standard_normal((kept.size, C)), rng.standard_normal((kept.size, C))
    # two steps = one step with the combined increment (exact here up to rounding)
    two = oracle.euler_update_fg(oracle.euler_update_fg(z, v1, kept, 0.5), v2, kept, -0.125)
    ref = torch.from_numpy(z).index_add(0, torch.from_numpy(kept), torch.from_numpy(0.5 * v1 - 0.125 * v2))
    assert np.allclose(two, ref.numpy(), rtol=0, atol=1e-12)
    assert np.array_equal(two[~mask], z[~mask])
    assert np.array_equal(oracle.euler_update_fg(z, v1, kept, 0.0), z)


def test_fg_loss_hand_example():
    # two retained positions (2 and 0) of L = 3, C = 2
    eps = np.array([[1.0, 1.0], [9.0, 9.0], [3.0, 0.0]])
    z0 = np.array([[0.5, 2.0], [9.0, 9.0], [1.0, 1.0]])
    kept = np.array([2, 0])
    # targets eps - z0: row 2 -> (2, -1), row 0 -> (0.5, -1)
    v = np.array([[3.0, -1.0], [0.5, 1.0]])
    loss, grad = oracle.fg_flow_loss(v, eps, z0, kept)
    # diffs (1, 0) and (0, 2): sum of squares 5 over n C = 4
    assert loss == 5.0 / 4.0
    assert np.array_equal(grad, [[0.5, 0.0], [0.0, 1.0]])


def test_fg_loss_matches_mse_and_finite_differences():
    rng = np.random.default_rng(4)
    L, C = 300, 8
    eps, z0 = rng.standard_normal((L, C)), rng.standard_normal((L, C))
    kept = np.flatnonzero(rng.random(L) < 0.5)
    v = rng.standard_normal((kept.size, C))
    loss, grad = oracle.fg_flow_loss(v, eps, z0, kept)
    target = torch.from_numpy(eps[kept] - z0[kept])
    vt = torch.from_numpy(v).requires_grad_(True)
    ref = torch.nn.functional.mse_loss(vt, target)
    ref.backward()
    assert abs(loss - ref.item()) <= 1e-12 * max(1.0, ref.item())
    assert np.allclose(grad, vt.grad.numpy(), rtol=0, atol=1e-15)
    # central differences on a few entries
    h = 1e-6
    for k, c in [(0, 0), (3, 5), (kept.size - 1, C - 1)]:
        vp, vm = v.copy(), v.copy()
        vp[k, c] += h
        vm[k, c] -= h
        fd = (oracle.fg_flow_loss(vp, eps, z0, kept)[0] - oracle.fg_flow_loss(vm, eps, z0, kept)[0]) / (2 * h)
        assert abs(fd - grad[k, c]) <= 1e-8
    # the exact velocity gives zero loss; background rows never matter
    assert oracle.fg_flow_loss(eps[kept] - z0[kept], eps, z0, kept)[0] == 0.0
    eps2 = eps.copy()
    eps2[np.setdiff1d(np.arange(L), kept)] = np.nan
    assert oracle.fg_flow_loss(v, eps2, z0, kept)[0] == loss


# ---------------------------------------------------------------------------
# Composite latent (Sec. 3.4, Eq. 9) and token masks (Sec. 3.2)
# ---------------------------------------------------------------------------

def test_composite_hand_example():
    # two views of P = 3 tokens, C = 2; retained positions 1, 3, 5
    bg = np.array([[10, 11], [12, 13], [14, 15]], dtype=np.float32)
    packed = np.array([[1, 2], [3, 4], [5, 6]], dtype=np.float32)
    out = oracle.composite_latent(packed, np.array([1, 3, 5]), bg, 6)
    assert np.array_equal(out, [[10, 11], [1, 2], [14, 15], [3, 4], [12, 13], [5, 6]])


def test_composite_matches_tile_then_index_put():
    rng = np.random.default_rng(8)
    V, P, C = 6, 64, 16
    L = V * P
    bg = rng.standard_normal((P, C)).astype(np.float32)
    kept = np.flatnonzero(rng.random(L) < 0.35)
    packed = rng.standard_normal((kept.size, C)).astype(np.float32)
    ref = torch.from_numpy(bg).repeat(V, 1)
    ref[torch.from_numpy(kept)] = torch.from_numpy(packed)
    out = oracle.composite_latent(packed, kept, bg, L)
    assert np.array_equal(out, ref.numpy())
    # nothing kept -> the tiled background; everything kept -> the packed rows
    assert np.array_equal(oracle.composite_latent(packed[:0], kept[:0], bg, L), np.tile(bg, (V, 1)))
    full = rng.standard_normal((L, C)).astype(np.float32)
    assert np.array_equal(oracle.composite_latent(full, np.arange(L), bg, L), full)


def test_token_mask_hand_example():
    # one 64 x 64 view, patch 16 -> 4 x 4 tokens; one bright pixel in token (1, 2)
    a = np.zeros((1, 64, 64), dtype=np.uint8)
    a[0, 16 + 5, 32 + 15] = 200
    m0 = oracle.token_mask_from_alpha(a, 16, 0)
    assert m0.sum() == 1 and m0[0, 1, 2] == 1
    m1 = oracle.token_mask_from_alpha(a, 16, 1)
    assert np.array_equal(m1[0], [[0, 1, 1, 1], [0, 1, 1, 1], [0, 1, 1, 1], [0, 0, 0, 0]])
    # threshold: a pixel at exactly the threshold is background
    assert oracle.token_mask_from_alpha(a, 16, 1, threshold=200).sum() == 0
    assert oracle.token_mask_from_alpha(a, 16, 1, threshold=199).sum() == 9


def test_token_mask_matches_reshape_max_and_scipy_dilation():
    from scipy import ndimage
    rng = np.random.default_rng(9)
    V, H, W, patch = 3, 96, 128, 16
    a = (rng.random((V, H, W)) < 0.002).astype(np.uint8) * rng.integers(1, 256, (V, H, W)).astype(np.uint8)
    for radius in (0, 1, 2):
        got = oracle.token_mask_from_alpha(a, patch, radius)
        pooled = a.reshape(V, H // patch, patch, W // patch, patch).max(axis=(2, 4)) > 0
        ref = np.stack([ndimage.binary_dilation(pooled[v], structure=np.ones((2 * radius + 1,) * 2))
                        if radius else pooled[v] for v in range(V)]).astype(np.uint8)
        assert np.array_equal(got, ref), radius


def test_topk_dense_prefix_blocks():
    """Text-prefix reading: prefix columns and rows are dense, the Top-K runs
    over the remaining key blocks (checked against the no-prefix selection
    restricted to j >= P, and by brute-force rank)."""
    rng = np.random.default_rng(12)
    q = rng.standard_normal((1, 700, 2, 8))
    k = rng.standard_normal((1, 700, 2, 8))
    block, P, kk = 64, 3, 4
    mask, sc = oracle.topk_block_mask(q, k, block, kk, prefix_blocks=P)
    nb = mask.shape[-1]
    assert mask[:, :, :P, :].all() and mask[:, :, :, :P].all()
    assert np.all(mask[:, :, P:, :].sum(-1) == P + kk)
    for h in range(2):
        for i in range(P, nb):
            row = sc[0, h, i]
            for j in range(P, nb):
                beaten = sum(1 for jj in range(P, nb) if row[jj] > row[j] or (row[jj] == row[j] and jj < j))
                assert mask[0, h, i, j] == (1 if beaten < kk else 0)
    # P = 0 is the plain selection; a prefix covering everything keeps all
    assert np.array_equal(oracle.topk_block_mask(q, k, block, kk, 0)[0], oracle.topk_block_mask(q, k, block, kk)[0])
    assert oracle.topk_block_mask(q, k, block, kk, nb)[0].all()


# ---------------------------------------------------------------------------
# Packed samples of differing lengths (Eq. 8 per sample)
# ---------------------------------------------------------------------------

def _packed_token_mask(cu, bm, block, H):
    """Token-level mask [1, H, T, T] of the whole packed sequence: a pair is
    allowed only inside one sample, and there only where that sample's block
    mask holds (block coordinates measured from the sample's first token)."""
    T = int(cu[-1])
    allow = np.zeros((1, H, T, T), dtype=bool)
    for b in range(len(cu) - 1):
        t0, t1 = int(cu[b]), int(cu[b + 1])
        blk = (np.arange(t0, t1) - t0) // block
        for h in range(H):
            allow[0, h, t0:t1, t0:t1] = bm[b, h][np.ix_(blk, blk)].astype(bool)
    return allow


def _varlen_case(seed, lens, block, H, D, density):
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    T, nb = int(cu[-1]), -(-max(lens) // block)
    q, k, v, do = (rng.standard_normal((T, H, D)) for _ in range(4))
    # random blocks everywhere (entries past a sample's own blocks included,
    # which must be ignored) and the diagonal within each sample, so that no
    # row of the dense reference is fully masked
    bm = (rng.random((len(lens), H, nb, nb)) < density).astype(np.uint8)
    for b, n in enumerate(lens):
        d = np.arange(-(-n // block))
        bm[b][:, d, d] = 1
    return cu, q, k, v, do, bm


@pytest.mark.parametrize("seed,lens,block,H,D", [(1, [37, 70, 16], 16, 2, 8),
                                                 (2, [5, 0, 64, 33], 16, 1, 4),
                                                 (3, [100, 99], 32, 2, 16)])
def test_varlen_fwd_bwd_match_block_diagonal_dense_attention(seed, lens, block, H, D):
    """The packed sequence as ONE dense attention problem whose token mask is
    block-diagonal over the samples: torch's SDPA and autograd in float64
    must reproduce the per-sample oracle (a wrong offset, a leak across
    samples or a mask entry read in the wrong sample's frame fails this)."""
    cu, q, k, v, do, bm = _varlen_case(seed, lens, block, H, D, 0.4)
    scale = 1.0 / math.sqrt(D)
    O, L = oracle.bsattn_fwd_varlen(q, k, v, cu, bm, block, scale)
    allow = torch.as_tensor(_packed_token_mask(cu, bm, block, H))
    tq, tk, tv = (torch.tensor(a[None], requires_grad=True) for a in (q, k, v))
    t = lambda a: a.permute(0, 2, 1, 3)
    o = torch.nn.functional.scaled_dot_product_attention(t(tq), t(tk), t(tv), attn_mask=allow)
    o = o.permute(0, 2, 1, 3)
    assert np.allclose(O, o[0].detach().numpy(), atol=1e-12)
    s = torch.einsum("nhd,mhd->hnm", torch.tensor(q), torch.tensor(k)) * scale
    lse = torch.logsumexp(s.masked_fill(~allow[0], -math.inf), dim=-1).numpy()
    assert np.allclose(L, lse, atol=1e-12)
    o.backward(torch.tensor(do[None]))
    dQ, dK, dV = oracle.bsattn_bwd_varlen(q, k, v, do, cu, bm, block, scale)
    assert np.allclose(dQ, tq.grad[0].numpy(), atol=1e-12)
    assert np.allclose(dK, tk.grad[0].numpy(), atol=1e-12)
    assert np.allclose(dV, tv.grad[0].numpy(), atol=1e-12)


def test_varlen_samples_are_independent():
    """Changing one sample's tokens leaves every other sample's outputs and
    gradients exactly as they were."""
    cu, q, k, v, do, bm = _varlen_case(7, [40, 23, 57], 16, 2, 8, 0.5)
    base = oracle.bsattn_fwd_varlen(q, k, v, cu, bm, 16, 0.3)[0]
    gbase = oracle.bsattn_bwd_varlen(q, k, v, do, cu, bm, 16, 0.3)
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    for a in (q2, k2, v2):
        a[40:63] += 5.0
    O2 = oracle.bsattn_fwd_varlen(q2, k2, v2, cu, bm, 16, 0.3)[0]
    g2 = oracle.bsattn_bwd_varlen(q2, k2, v2, do, cu, bm, 16, 0.3)
    others = np.r_[0:40, 63:120]
    assert np.array_equal(O2[others], base[others])
    assert not np.allclose(O2[40:63], base[40:63])
    for a, b in zip(g2, gbase):
        assert np.array_equal(a[others], b[others])
