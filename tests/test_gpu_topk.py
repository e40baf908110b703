"""GPU Top-K block selection (Sec. 3.3, Eq. 6-7) through the C ABI against the
float64 oracle. The GPU ranks fp32 scores, so a row is compared exactly
wherever the exact selection is decided by more than the fp32 error bound of
the pooling and the dot products (`parity.topk_tolerance`); every other row
must still be a valid Top-K within that bound. Constructed ties check the
lower-index rule exactly."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_23169_amd as ut
import workloads as W
from parity import check_out, check_topk, topk_tolerance

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _qk(seed, n, H, D, block):
    c = W.random_case(seed, n, H, D, block, 1.0)
    return c["q"], c["k"]


def _run(q, k, block, kk, prefix=0):
    m = ut.topk_block_mask(q.to(DEV), k.to(DEV), block, kk, prefix_blocks=prefix)
    torch.cuda.synchronize()
    return m.cpu().numpy()


CASES = [  # seed, N, H, D, block, k_keep
    (1, 384, 2, 64, 64, 2),
    (2, 700, 3, 128, 128, 2),      # ragged last block
    (3, 1000, 2, 64, 64, 5),
    (4, 5000, 4, 128, 128, 7),
    (5, 3000, 2, 128, 32, 20),     # 94 blocks: two 64-lane chunks per row
    (6, 50, 2, 128, 128, 1),       # a single (short) block
    (7, 2000, 2, 128, 16, 40),     # 125 blocks
    (8, 30000, 1, 128, 16, 90),    # 1875 blocks: four rows per workgroup
    (9, 70000, 1, 64, 16, 300),    # 4375 blocks: one row per workgroup
    (10, 2000, 2, 96, 64, 5),      # head_dim 96: the fused multiply-add path, 16 rows per group
    (11, 900, 3, 24, 32, 3),       # head_dim 24
    (12, 61000, 1, 128, 64, 100),  # 954 blocks, head_dim 128: past the MFMA path's LDS limit
]


@pytest.mark.parametrize("seed,n,H,D,block,kk", CASES)
def test_topk_matches_oracle(seed, n, H, D, block, kk):
    q, k = _qk(seed, n, H, D, block)
    got = _run(q, k, block, kk)
    ref, sc = oracle.topk_block_mask(q, k, block, kk)
    frac = check_topk(got, ref, sc, topk_tolerance(q, k, block), kk, f"case {seed}")
    assert frac > 0.5, f"case {seed}: only {frac:.2f} of the rows are decided"


def test_topk_keep_all_and_keep_one():
    q, k = _qk(11, 900, 2, 64, 64)
    nb = -(-900 // 64)
    assert _run(q, k, 64, nb).all()
    assert _run(q, k, 64, nb + 10).all()
    got = _run(q, k, 64, 1)
    ref, sc = oracle.topk_block_mask(q, k, 64, 1)
    check_topk(got, ref, sc, topk_tolerance(q, k, 64), 1, "keep one")


def test_topk_exact_ties_lower_block_first():
    # key blocks 0, 3 and 5 hold identical tokens: identical fp32 pooled rows, exact ties
    q, k = _qk(12, 512, 2, 64, 64)
    k = k.clone()
    k[:, 3 * 64:4 * 64] = k[:, 0:64]
    k[:, 5 * 64:6 * 64] = k[:, 0:64]
    got = _run(q, k, 64, 1)
    ref, sc = oracle.topk_block_mask(q, k, 64, 1)
    assert np.array_equal(sc[..., 0], sc[..., 3]) and np.array_equal(sc[..., 0], sc[..., 5])
    # wherever a tied block wins, block 0 is the one kept
    tied_win = sc[..., 0] >= sc.max(-1)
    assert tied_win.any()
    assert np.all(got[..., 0][tied_win] == 1) and np.all(got[..., 3][tied_win] == 0)
    for kk in (1, 2, 3):
        got = _run(q, k, 64, kk)
        ref, _ = oracle.topk_block_mask(q, k, 64, kk)
        # exact ties resolve identically; other rows must be decided or valid
        check_topk(got, ref, sc, topk_tolerance(q, k, 64), kk, f"ties k={kk}")


@pytest.mark.parametrize("wl_name,rho", [("c1k", "0.2"), ("c2k_train", "0.1")])
def test_topk_full_size_workloads(wl_name, rho):
    wl = W.WORKLOADS[wl_name].with_rho(rho)
    inst = W.make(wl, with_qkv=True)
    nb = -(-inst.n_kept // wl.block)
    kk = W.kept_off_diagonal(rho, nb)   # floor(rho N_k) blocks
    got = _run(inst.q, inst.k, wl.block, kk)
    ref, sc = oracle.topk_block_mask(inst.q, inst.k, wl.block, kk)
    frac = check_topk(got, ref, sc, topk_tolerance(inst.q, inst.k, wl.block), kk, wl_name)
    assert frac > 0.5


def test_topk_mask_drives_attention_end_to_end():
    """Top-K mask -> block lists -> forward, against the oracle's own mask and
    forward (the rows used are all decided, so both sides select the same)."""
    c = W.random_case(18, 1500, 2, 128, 128, 1.0)   # seed 18: every row decided
    q, k = c["q"], c["k"]
    v = c["v"]
    kk = 4
    ref, sc = oracle.topk_block_mask(q, k, 128, kk)
    mask = ut.topk_block_mask(q.to(DEV), k.to(DEV), 128, kk)
    frac = check_topk(mask.cpu().numpy(), ref, sc, topk_tolerance(q, k, 128), kk, "e2e")
    assert frac == 1.0, "pick a case whose rows are all decided"
    idx = ut.build_block_index(mask)
    scale = 1 / math.sqrt(128)
    o, lse = ut.bsattn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), idx, 128, scale)
    O, L = oracle.bsattn_fwd(q, k, v, ref, 128, scale)
    check_out(o, lse, O, L, "e2e")


@pytest.mark.parametrize("seed,n,H,D,block,kk,P", [
    (21, 2000, 2, 128, 128, 3, 4),     # MFMA path
    (22, 1212, 3, 64, 64, 5, 8),
    (23, 3000, 2, 96, 64, 6, 2),       # fused multiply-add path
    (24, 900, 1, 128, 128, 20, 3),     # k_keep beyond the remaining blocks: dense
])
def test_topk_dense_text_prefix(seed, n, H, D, block, kk, P):
    q, k = _qk(seed, n, H, D, block)
    got = _run(q, k, block, kk, P)
    ref, sc = oracle.topk_block_mask(q, k, block, kk, prefix_blocks=P)
    check_topk(got, ref, sc, topk_tolerance(q, k, block), kk, f"prefix {seed}", prefix=P)


def test_topk_text_prefix_full_size():
    """512 text tokens ahead of the 2K workload's 77,060 foreground tokens:
    four dense leading blocks, k = floor(0.1 N_k) among the rest."""
    inst = W.make(W.WORKLOADS["c2k_train"].with_rho("0.1"), with_qkv=True)
    g = torch.Generator().manual_seed(25)
    txt = lambda: torch.randn((1, 512, 24, 128), generator=g).to(torch.bfloat16)
    q, k = torch.cat([txt(), inst.q], 1), torch.cat([txt(), inst.k], 1)
    nb = -(-q.shape[1] // 128)
    kk = W.kept_off_diagonal("0.1", nb)
    got = _run(q, k, 128, kk, 4)
    ref, sc = oracle.topk_block_mask(q, k, 128, kk, prefix_blocks=4)
    assert check_topk(got, ref, sc, topk_tolerance(q, k, 128), kk, "text prefix", prefix=4) > 0.5
