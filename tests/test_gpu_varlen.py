"""Packed samples of differing lengths through the C ABI (ut_bsattn_fwd_varlen,
ut_bsattn_bwd_varlen) against the oracle's per-sample Eq. 8: ragged lengths
(short last blocks, a sample shorter than one block, an empty sample, block
mask entries past a sample's end that must be ignored), equal lengths against
the uniform calls bit for bit, a bucket of the 512-canvas workload at full
head count, two 2048-canvas samples at full size (sampled rows), tokens
covered by no sample, and the validation of the offsets."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_23169_amd as ut
import workloads as W
from parity import block_rows, check_grad, check_out

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _dev(case):
    q, k, v, do = (case[n].to(DEV) for n in ("q", "k", "v", "do"))
    cu = torch.from_numpy(case["cu_seqlens"]).to(DEV)
    idx = ut.build_block_index(torch.from_numpy(case["block_mask"]).to(DEV))
    return q, k, v, do, cu, idx


def _run(case, ds_pairs=None):
    q, k, v, do, cu, idx = _dev(case)
    o, lse = ut.bsattn_fwd_varlen(q, k, v, cu, case["max_seqlen"], idx, case["block"], case["scale"])
    if ds_pairs == "half":
        ds_pairs = idx["nnz"] // 2
    dq, dk, dv = ut.bsattn_bwd_varlen(q, k, v, o, do, lse, cu, case["max_seqlen"], idx, case["block"],
                                      case["scale"], ds_pairs=ds_pairs)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


# dS tiles in the backward's workspace: all pairs, none (dQ recomputed), half
@pytest.mark.parametrize("ds_pairs", [None, 0, "half"])
@pytest.mark.parametrize("seed,lens,H,D,block,density", [
    (1, [700, 1300, 257, 0, 128], 2, 128, 128, 0.4),
    (2, [65, 1, 300, 64], 3, 64, 64, 0.5),
    (3, [1000, 999, 1001], 2, 128, 64, 0.3),
    (4, [129, 2000], 1, 64, 128, 0.25),
])
def test_varlen_matches_oracle(seed, lens, H, D, block, density, ds_pairs):
    case = W.varlen_case(seed, lens, H, D, block, density)
    o, lse, dq, dk, dv = _run(case, ds_pairs)
    args = (case["q"], case["k"], case["v"])
    O, L = oracle.bsattn_fwd_varlen(*args, case["cu_seqlens"], case["block_mask"], block,
                                    case["scale"])
    check_out(o, lse, O, L, f"varlen {lens}")
    grads = oracle.bsattn_bwd_varlen(*args, case["do"], case["cu_seqlens"], case["block_mask"], block,
                                     case["scale"])
    for got, ref, nm in zip((dq, dk, dv), grads, ("dq", "dk", "dv")):
        check_grad(got, ref, f"varlen {lens} {nm}")


def test_mask_entries_past_a_sample_are_ignored():
    """The same samples with zeros instead of random entries past each
    sample's own blocks give bit-identical results."""
    lens = [300, 900, 513]
    a = _run(W.varlen_case(5, lens, 2, 128, 128, 0.4, garbage_past_end=True))
    b = _run(W.varlen_case(5, lens, 2, 128, 128, 0.4, garbage_past_end=False))
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_equal_lengths_match_uniform_calls_bit_for_bit():
    B, N, H, D, block = 3, 1000, 2, 128, 128
    case = W.varlen_case(6, [N] * B, H, D, block, 0.4)
    o, lse, dq, dk, dv = _run(case)
    q, k, v, do, cu, idx = _dev(case)
    shp = (B, N, H, D)
    ou, lu = ut.bsattn_fwd(q.view(shp), k.view(shp), v.view(shp), idx, block, case["scale"])
    gu = ut.bsattn_bwd(q.view(shp), k.view(shp), v.view(shp), ou, do.view(shp), lu, idx, block,
                       case["scale"])
    torch.cuda.synchronize()
    assert torch.equal(o.view(shp), ou)
    # varlen LSE is [H, T]; uniform is [B, H, N]
    assert torch.equal(lse.view(H, B, N).permute(1, 0, 2), lu)
    for x, y in zip((dq, dk, dv), gu):
        assert torch.equal(x.view(shp), y)


def test_bucket_of_512_canvas_samples_full_heads():
    """Eight samples of one foreground-count bucket of the 512-canvas workload
    (24 heads, head_dim 128, block 128, ~10% of key blocks); parity on two
    query blocks of every sample (the first and the short last one)."""
    wl = W.WORKLOADS["c512"]
    lens = W.bucket_lengths(11, wl, 8)
    case = W.varlen_case(12, lens, wl.heads, wl.head_dim, wl.block, 0.1)
    o, lse, dq, dk, dv = _run(case)
    cu, bm, blk, sc = case["cu_seqlens"], case["block_mask"], case["block"], case["scale"]
    for b, n in enumerate(lens):
        t0, nb = int(cu[b]), -(-n // blk)
        sl = slice(t0, t0 + n)
        sample = [case[x][None, sl] for x in ("q", "k", "v")]
        qb = [0, nb - 1]
        O, L = oracle.bsattn_fwd(*sample, bm[b:b + 1, :, :nb, :nb], blk, sc, q_blocks=qb)
        rows = block_rows(qb, blk, n)
        check_out(o[sl][rows], lse[:, sl][:, rows], O[0][rows], L[0][:, rows], f"bucket sample {b}")
        dQ, _, _ = oracle.bsattn_bwd(*sample, case["do"][None, sl], bm[b:b + 1, :, :nb, :nb], blk, sc,
                                     q_blocks=qb)
        check_grad(dq[sl], dQ[0], f"bucket sample {b} dq", rows=rows)


def test_two_2k_samples_full_size_sampled():
    """Per-GPU batch 2 at the 2048 canvas: two samples of one foreground-count
    bucket (~77K kept tokens each, 24 heads x 128, block 128, density 0.1 +
    diagonal) packed in one launch pair. The oracle checks, per sample and on
    two heads, the first, a middle and the short last query block (O, LSE,
    dQ), and dK / dV of the last key block from every query block selecting it."""
    wl = W.WORKLOADS["c2k_train"]
    lens = W.bucket_lengths(21, wl, 2)
    case = W.varlen_case_device(22, lens, wl.heads, wl.head_dim, wl.block, 0.1, DEV)
    q, k, v, do = case["q"], case["k"], case["v"], case["do"]
    cu_h, bm, blk, sc = case["cu_seqlens"], case["block_mask"], case["block"], case["scale"]
    cu = torch.from_numpy(cu_h).to(DEV)
    idx = ut.build_block_index(torch.from_numpy(bm).to(DEV))
    o, lse = ut.bsattn_fwd_varlen(q, k, v, cu, case["max_seqlen"], idx, blk, sc)
    dq, dk, dv = ut.bsattn_bwd_varlen(q, k, v, o, do, lse, cu, case["max_seqlen"], idx, blk, sc)
    torch.cuda.synchronize()
    heads = [5, 19]
    ht = torch.tensor(heads, device=DEV)
    for b, n in enumerate(lens):
        t0, nb = int(cu_h[b]), -(-n // blk)
        sl = slice(t0, t0 + n)
        x = [t[sl].index_select(1, ht).unsqueeze(0).cpu() for t in (q, k, v, do)]
        m = np.ascontiguousarray(bm[b:b + 1][:, heads, :nb, :nb])
        qb = [0, nb // 2, nb - 1]
        rows = block_rows(qb, blk, n)
        O, L = oracle.bsattn_fwd(*x[:3], m, blk, sc, q_blocks=qb)
        check_out(o[sl].index_select(1, ht)[rows], lse.index_select(0, ht)[:, sl][:, rows],
                  O[0][rows], L[0][:, rows], f"2K sample {b}")
        jb = nb - 1
        need = sorted(set(qb) | set(np.flatnonzero(m[0, :, :, jb].any(axis=0)).tolist()))
        dQ, dK, dV = oracle.bsattn_bwd(*x, m, blk, sc, q_blocks=need)
        check_grad(dq[sl].index_select(1, ht), dQ[0], f"2K sample {b} dq", rows=rows)
        krows = block_rows([jb], blk, n)
        check_grad(dk[sl].index_select(1, ht), dK[0], f"2K sample {b} dk", rows=krows)
        check_grad(dv[sl].index_select(1, ht), dV[0], f"2K sample {b} dv", rows=krows)


def test_tokens_outside_every_sample_are_untouched():
    """Offsets that stop short of T leave the remaining tokens as they were."""
    case = W.varlen_case(8, [300, 400], 2, 64, 64, 0.5)
    q, k, v, do, cu, idx = _dev(case)
    T, H, D = 1000, 2, 64
    pad = lambda t: torch.cat([t, torch.ones(T - t.shape[0], H, D, dtype=t.dtype, device=DEV)])
    q, k, v = pad(q), pad(k), pad(v)
    o = torch.full_like(q, 7.0)
    lse = torch.full((H, T), 7.0, dtype=torch.float32, device=DEV)
    st = ut.ut_bsattn_fwd_varlen(q, k, v, o, lse, cu, case["max_seqlen"], 64, idx["q_rowptr"],
                                 idx["q_cols"], case["scale"])
    torch.cuda.synchronize()
    assert st == ut.UT_OK
    assert torch.all(o[700:] == 7.0) and torch.all(lse[:, 700:] == 7.0)
    O, L = oracle.bsattn_fwd_varlen(case["q"], case["k"], case["v"], case["cu_seqlens"],
                                    case["block_mask"], 64, case["scale"])
    check_out(o[:700], lse[:, :700], O, L, "short offsets")


def test_validate_mode_checks_offsets(monkeypatch):
    case = W.varlen_case(9, [200, 300], 2, 64, 64, 0.5)
    q, k, v, do, cu, idx = _dev(case)
    T, H = q.shape[0], q.shape[1]
    o, lse = torch.empty_like(q), torch.empty((H, T), dtype=torch.float32, device=DEV)
    call = lambda c, maxlen=300: ut.ut_bsattn_fwd_varlen(q, k, v, o, lse, c, maxlen, 64,
                                                         idx["q_rowptr"], idx["q_cols"], case["scale"])
    monkeypatch.setenv("UT_VALIDATE", "1")
    assert call(cu) == ut.UT_OK
    torch.cuda.synchronize()
    bad = {"decreasing": [0, 300, 200], "not ending at T": [0, 200, 400],
           "not starting at 0": [10, 200, 500]}
    for what, c in bad.items():
        assert call(torch.tensor(c, dtype=torch.int32, device=DEV)) == ut.UT_ERR_INVALID_ARG, what
    assert call(cu, maxlen=299) == ut.UT_ERR_INVALID_ARG
    assert "max_seqlen" in ut.last_error()
