"""More attention checks through the C ABI: a diagonal-only mask, gradient
invariants at a mid size and at the full 2K size, the opt-in block-list
validation mode, launches on a non-default stream, and seeded sweeps over
random shapes (uniform and packed batches)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_23169_amd as ut
import workloads as W
from parity import check_grad, check_out

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _run(case, ds_pairs=None):
    q, k, v, do = (case[n].to(DEV) for n in ("q", "k", "v", "do"))
    idx = ut.build_block_index(torch.from_numpy(case["block_mask"]).to(DEV))
    o, lse = ut.bsattn_fwd(q, k, v, idx, case["block"], case["scale"])
    if callable(ds_pairs):
        ds_pairs = ds_pairs(idx["nnz"])
    dq, dk, dv = ut.bsattn_bwd(q, k, v, o, do, lse, idx, case["block"], case["scale"],
                               ds_pairs=ds_pairs)
    torch.cuda.synchronize()
    return q, k, v, do, idx, o, lse, dq, dk, dv


def test_diagonal_only_mask_is_blockwise_dense_attention():
    case = W.random_case(31, 900, 2, 128, 128, 0.0, diag=True)
    *_, o, lse, dq, dk, dv = _run(case)
    O, L = oracle.bsattn_fwd(case["q"], case["k"], case["v"], case["block_mask"], 128, case["scale"])
    check_out(o, lse, O, L, "diagonal")
    dQ, dK, dV = oracle.bsattn_bwd(case["q"], case["k"], case["v"], case["do"], case["block_mask"], 128,
                                   case["scale"])
    for got, ref, nm in ((dq, dQ, "dq"), (dk, dK, "dk"), (dv, dV, "dv")):
        check_grad(got, ref, f"diagonal {nm}")


def _invariants(dk, dv, do, label):
    """Per head: sum over tokens of dK is 0 (rows of dS sum to 0) and of dV is
    that of dO (rows of P sum to 1). P and dS enter the second products as bf16
    (relative 2^-9 each) and the outputs are bf16, hence the 1e-2 bound
    relative to the summed magnitudes."""
    dk, dv, do = (t.float() for t in (dk, dv, do))
    sk = dk.sum(dim=1).abs().amax().item()
    ak = dk.abs().sum(dim=1).amin().item()
    assert sk <= 1e-2 * ak, f"{label}: |sum dK| {sk:.3e} vs sum |dK| {ak:.3e}"
    dd = (dv.sum(dim=1) - do.sum(dim=1)).abs().amax().item()
    ao = do.abs().sum(dim=1).amin().item()
    assert dd <= 1e-2 * ao, f"{label}: |sum dV - sum dO| {dd:.3e} vs sum |dO| {ao:.3e}"


def test_gradient_invariants_mid_size():
    case = W.random_case(32, 5000, 3, 128, 128, 0.3)     # diagonal kept: no empty rows
    q, k, v, do, idx, o, lse, dq, dk, dv = _run(case)
    _invariants(dk, dv, do, "mid")


def test_gradient_invariants_full_size():
    inst = W.make(W.WORKLOADS["c2k_train"].with_rho("0.1"), with_qkv=True, with_do=True)
    case = {"q": inst.q, "k": inst.k, "v": inst.v, "do": inst.do, "block_mask": inst.block_mask,
            "block": 128, "scale": 1 / math.sqrt(128)}
    q, k, v, do, idx, o, lse, dq, dk, dv = _run(case)
    _invariants(dk, dv, do, "2K")


def test_validate_mode(monkeypatch):
    case = W.random_case(33, 700, 2, 64, 64, 0.4)
    q, k, v, do, idx, o_ref, lse_ref, *_ = _run(case)
    B, N, H, D = q.shape
    nb = -(-N // 64)
    o, lse = torch.empty_like(q), torch.empty((B, H, N), dtype=torch.float32, device=DEV)
    monkeypatch.setenv("UT_VALIDATE", "1")
    # valid lists pass and give the same result
    assert ut.ut_bsattn_fwd(q, k, v, o, lse, 64, idx["q_rowptr"], idx["q_cols"], case["scale"]) == ut.UT_OK
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref) and torch.equal(lse, lse_ref)
    # corrupted lists are refused before any launch
    cols = idx["q_cols"].clone()
    cols[3] = nb                                        # out of range
    assert ut.ut_bsattn_fwd(q, k, v, o, lse, 64, idx["q_rowptr"], cols, case["scale"]) == ut.UT_ERR_INVALID_ARG
    assert "outside" in ut.last_error()
    rp = idx["q_rowptr"]
    row = int(np.argmax(np.diff(rp.cpu().numpy()) >= 2))   # a row with two entries or more
    cols = idx["q_cols"].clone()
    a = int(rp[row].item())
    cols[a], cols[a + 1] = cols[a + 1].clone(), cols[a].clone()   # not ascending
    assert ut.ut_bsattn_fwd(q, k, v, o, lse, 64, rp, cols, case["scale"]) == ut.UT_ERR_INVALID_ARG
    assert "ascending" in ut.last_error()
    bad_rp = rp.clone()
    bad_rp[5] = bad_rp[4] - 1                           # decreasing pointers
    assert ut.ut_bsattn_fwd(q, k, v, o, lse, 64, bad_rp, idx["q_cols"], case["scale"]) == ut.UT_ERR_INVALID_ARG
    ws = torch.empty(ut.ut_bsattn_bwd_workspace_size(B, N, H), dtype=torch.uint8, device=DEV)
    dq, dk, dv = (torch.empty_like(q) for _ in range(3))
    kvc = idx["kv_rows"].clone()
    kvc[0] = -1
    st = ut.ut_bsattn_bwd(q, k, v, o_ref, do, lse_ref, dq, dk, dv, 64, idx["q_rowptr"], idx["q_cols"],
                          idx["kv_colptr"], kvc, case["scale"], ws)
    assert st == ut.UT_ERR_INVALID_ARG and "column lists" in ut.last_error()


def test_non_default_stream_matches_default():
    case = W.random_case(34, 1500, 2, 128, 128, 0.3)
    q, k, v, do, idx, o_ref, lse_ref, dq_ref, dk_ref, dv_ref = _run(case)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        o, lse = ut.bsattn_fwd(q, k, v, idx, 128, case["scale"], stream=s)
        dq, dk, dv = ut.bsattn_bwd(q, k, v, o, do, lse, idx, 128, case["scale"], stream=s)
    s.synchronize()
    for a, b in ((o, o_ref), (lse, lse_ref), (dq, dq_ref), (dk, dk_ref), (dv, dv_ref)):
        assert torch.equal(a, b)


def _dq_mode(mrng):
    """One of the backward's dQ splits: every pair's dS tile stored (None),
    none (0), or a random count (the rest recomputed)."""
    m = int(mrng.integers(3))
    if m == 2:
        r = float(mrng.random())
        return "some", lambda nnz: int(r * (nnz + 1))
    return ("all", None) if m == 0 else ("none", 0)


def test_random_shape_sweep():
    """Twenty seeded random configurations (length, heads, head_dim, block,
    batch, density, forced-empty rows, dQ from all, none or some of the
    stored dS tiles), forward and backward against the oracle element by
    element."""
    rng = np.random.default_rng(2024)
    mrng = np.random.default_rng(4048)   # modes drawn apart: the shapes stay as they were
    for case_no in range(20):
        n = int(rng.integers(1, 2500))
        H = int(rng.integers(1, 4))
        D = int(rng.choice([64, 128]))
        blk = int(rng.choice([64, 128]))
        batch = int(rng.integers(1, 3))
        dens = float(rng.uniform(0.05, 1.0))
        nb = -(-n // blk)
        empty = int(rng.integers(0, min(3, nb) + 1))
        seed = int(rng.integers(1 << 30))
        mode, pairs = _dq_mode(mrng)
        label = (f"sweep {case_no}: n={n} H={H} D={D} block={blk} B={batch} density={dens:.2f} "
                 f"empty={empty} dq={mode}")
        print(label, flush=True)
        case = W.random_case(seed, n, H, D, blk, dens, batch=batch, empty_rows=empty)
        q, k, v, do, idx, o, lse, dq, dk, dv = _run(case, pairs)
        O, L = oracle.bsattn_fwd(case["q"], case["k"], case["v"], case["block_mask"], blk, case["scale"])
        check_out(o, lse, O, L, label)
        grads = oracle.bsattn_bwd(case["q"], case["k"], case["v"], case["do"], case["block_mask"], blk,
                                  case["scale"])
        for got, ref, nm in zip((dq, dk, dv), grads, ("dq", "dk", "dv")):
            check_grad(got, ref, f"{label} {nm}")


def test_random_varlen_sweep():
    """Ten seeded random packed batches (1-5 samples of 0-1500 tokens, some
    shorter than a block; dQ from all, none or some of the stored dS tiles)
    against the oracle element by element."""
    rng = np.random.default_rng(2025)
    mrng = np.random.default_rng(4050)
    for case_no in range(10):
        count = int(rng.integers(1, 6))
        lens = [int(x) for x in rng.integers(0, 1500, size=count)]
        if max(lens) == 0:
            lens[0] = 1
        H = int(rng.integers(1, 3))
        D = int(rng.choice([64, 128]))
        blk = int(rng.choice([64, 128]))
        dens = float(rng.uniform(0.1, 0.9))
        mode, pairs = _dq_mode(mrng)
        label = f"varlen sweep {case_no}: lens={lens} H={H} D={D} block={blk} density={dens:.2f} dq={mode}"
        print(label, flush=True)
        c = W.varlen_case(int(rng.integers(1 << 30)), lens, H, D, blk, dens)
        q, k, v, do = (c[x].to(DEV) for x in ("q", "k", "v", "do"))
        cu = torch.from_numpy(c["cu_seqlens"]).to(DEV)
        idx = ut.build_block_index(torch.from_numpy(c["block_mask"]).to(DEV))
        o, lse = ut.bsattn_fwd_varlen(q, k, v, cu, c["max_seqlen"], idx, blk, c["scale"])
        g = ut.bsattn_bwd_varlen(q, k, v, o, do, lse, cu, c["max_seqlen"], idx, blk, c["scale"],
                                 ds_pairs=pairs(idx["nnz"]) if callable(pairs) else pairs)
        torch.cuda.synchronize()
        O, L = oracle.bsattn_fwd_varlen(c["q"], c["k"], c["v"], c["cu_seqlens"], c["block_mask"], blk,
                                        c["scale"])
        check_out(o, lse, O, L, label)
        grads = oracle.bsattn_bwd_varlen(c["q"], c["k"], c["v"], c["do"], c["cu_seqlens"],
                                         c["block_mask"], blk, c["scale"])
        for got, ref, nm in zip(g, grads, ("dq", "dk", "dv")):
            check_grad(got, ref, f"{label} {nm}")


def test_lse_normalises_the_allowed_scores():
    """For sampled query rows, exp(s - LSE) summed over the row's allowed keys
    (scores exact in float64 from the bf16 inputs) is 1; |LSE error| <= 1e-3
    bounds the deviation by about 1e-3."""
    case = W.random_case(41, 3000, 2, 128, 128, 0.3, empty_rows=0)
    q, k, v, do, idx, o, lse, *_ = _run(case)
    Q, K = case["q"].double().numpy()[0], case["k"].double().numpy()[0]
    bm, blk, sc = case["block_mask"][0], 128, case["scale"]
    L = lse.double().cpu().numpy()[0]
    rng = np.random.default_rng(41)
    for h in range(2):
        for r in rng.choice(3000, 40, replace=False):
            keys = np.concatenate([np.arange(j * blk, min(3000, (j + 1) * blk))
                                   for j in np.flatnonzero(bm[h, r // blk])])
            s = Q[r, h] @ K[keys, h].T * sc
            tot = np.exp(s - L[h, r]).sum()
            assert abs(tot - 1.0) <= 2e-3, (h, r, tot)
