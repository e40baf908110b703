"""GPU parity of block-sparse attention forward and backward against the
float64 oracle, through the C ABI. Small cases are compared element by
element (several tiles, ragged tails, empty rows, every head_dim / block
pair); the full-size workloads are compared on sampled heads and blocks that
the oracle computes exactly (a query block's rows, or a key block's complete
gradient from every query block that selects it)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_23169_amd as ut
import workloads as W
from parity import block_rows, check_grad, check_out, to_np

pytestmark = pytest.mark.gpu
DEV = "cuda"


# dS tiles the backward's workspace makes room for: every pair (dQ from the
# stored tiles), none (dQ recomputed) or half (the first query blocks stored,
# the rest recomputed)
MODES = {"stored": None, "recompute": 0, "partial": "half"}


def run_gpu(case, backward=True, ds_pairs=None):
    q, k, v = (case[n].to(DEV) for n in ("q", "k", "v"))
    idx = ut.build_block_index(torch.from_numpy(case["block_mask"]).to(DEV))
    o, lse = ut.bsattn_fwd(q, k, v, idx, case["block"], case["scale"])
    out = {"o": o, "lse": lse, "idx": idx}
    if backward:
        do = case["do"].to(DEV)
        if ds_pairs == "half":
            ds_pairs = idx["nnz"] // 2
        out["dq"], out["dk"], out["dv"] = ut.bsattn_bwd(q, k, v, o, do, lse, idx, case["block"],
                                                        case["scale"], ds_pairs=ds_pairs)
    torch.cuda.synchronize()
    return out


SMALL = [  # seed, N, H, D, block, density, batch, empty_rows
    (1, 700, 3, 128, 128, 0.4, 1, 0),
    (2, 700, 3, 64, 64, 0.4, 1, 0),
    (3, 700, 2, 128, 64, 0.3, 1, 1),
    (4, 700, 2, 64, 128, 0.5, 1, 1),
    (5, 50, 2, 128, 128, 1.0, 1, 0),      # N below one block
    (6, 512, 2, 128, 128, 0.5, 2, 0),     # exact multiple, batch 2
    (7, 1000, 2, 128, 128, 0.2, 1, 3),    # several empty rows
    (8, 1300, 4, 128, 128, 1.0, 1, 0),    # dense (all ones)
    (9, 1, 2, 128, 128, 1.0, 1, 0),       # a single token
    (10, 129, 2, 128, 128, 0.5, 1, 0),    # last block of one token
    (11, 65, 2, 64, 64, 1.0, 1, 0),       # the same at block 64
    (12, 64, 1, 64, 64, 1.0, 3, 0),       # one full block, batch 3
]


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("seed,n,H,D,block,density,batch,empty", SMALL)
def test_small_fwd_bwd_elementwise(seed, n, H, D, block, density, batch, empty, mode):
    case = W.random_case(seed, n, H, D, block, density, batch=batch, empty_rows=empty)
    g = run_gpu(case, ds_pairs=MODES[mode])
    O, L = oracle.bsattn_fwd(case["q"], case["k"], case["v"], case["block_mask"], block, case["scale"])
    check_out(g["o"], g["lse"], O, L, f"fwd {seed}")
    dQ, dK, dV = oracle.bsattn_bwd(case["q"], case["k"], case["v"], case["do"], case["block_mask"],
                                   block, case["scale"])
    for got, ref, nm in ((g["dq"], dQ, "dq"), (g["dk"], dK, "dk"), (g["dv"], dV, "dv")):
        check_grad(got, ref, f"{nm} {seed} {mode}")
    if empty:
        # empty rows: O = 0, LSE = -inf, dQ = 0 exactly
        bm = case["block_mask"]
        for b, h, i in zip(*np.nonzero(bm.sum(-1) == 0)):
            rows = np.arange(i * block, min(n, (i + 1) * block))
            assert np.all(to_np(g["o"])[b, rows, h] == 0)
            assert np.all(np.isneginf(to_np(g["lse"])[b, h, rows]))
            assert np.all(to_np(g["dq"])[b, rows, h] == 0)


def test_peaky_scores_online_rescaling():
    case = W.random_case(11, 900, 2, 128, 128, 0.5)
    case["q"] = (case["q"].float() * 4).to(torch.bfloat16)
    g = run_gpu(case)
    O, L = oracle.bsattn_fwd(case["q"], case["k"], case["v"], case["block_mask"], 128, case["scale"])
    check_out(g["o"], g["lse"], O, L, "peaky")
    dQ, dK, dV = oracle.bsattn_bwd(case["q"], case["k"], case["v"], case["do"], case["block_mask"],
                                   128, case["scale"])
    check_grad(g["dq"], dQ, "peaky dq")
    check_grad(g["dk"], dK, "peaky dk")
    check_grad(g["dv"], dV, "peaky dv")


@pytest.mark.parametrize("seed,boost", [(13, 60.0), (14, 400.0)])
def test_later_key_block_far_above_first_tile_max(seed, boost):
    """Keys of the last block aligned with the queries make later tiles score
    far above the first tile's maximum (2^(thousands) in log2 units for the
    larger boost): the forward must take a new max and rescale rather than
    overflow."""
    case = W.random_case(seed, 900, 2, 128, 128, 0.6)
    q = case["q"].float() * 4
    k = case["k"].float().clone()
    k[0, -200:] = q[0, :200] / q[0, :200].norm(dim=-1, keepdim=True) * boost
    case["q"], case["k"] = q.to(torch.bfloat16), k.to(torch.bfloat16)
    g = run_gpu(case, backward=False)
    O, L = oracle.bsattn_fwd(case["q"], case["k"], case["v"], case["block_mask"], 128, case["scale"])
    assert torch.isfinite(g["o"]).all() and torch.isfinite(g["lse"]).all()
    check_out(g["o"], g["lse"], O, L, f"boost {boost}")


def test_unit_values_give_unit_outputs_and_determinism():
    case = W.random_case(12, 1100, 3, 128, 128, 0.3)
    case["v"] = torch.ones_like(case["v"])
    g1 = run_gpu(case)
    assert torch.all(g1["o"] == 1.0)
    g2 = run_gpu(case)
    for nm in ("o", "lse", "dq", "dk", "dv"):
        assert torch.equal(g1[nm].view(torch.int16) if g1[nm].dtype == torch.bfloat16 else g1[nm],
                           g2[nm].view(torch.int16) if g2[nm].dtype == torch.bfloat16 else g2[nm]), nm


def test_dropped_tokens_never_influence_kept_outputs():
    """Full-grid inputs whose background rows are NaN or huge: after the drop,
    the kept outputs are finite and bit-identical."""
    wl = W.WORKLOADS["tiny"]
    inst = W.make(wl)
    Lfull, H, D = wl.seq_len, wl.heads, wl.head_dim
    kept, _, n = oracle.compact(inst.fg_mask)
    outs = []
    for bg in (float("nan"), 3.0e4):
        full = torch.full((Lfull, 3, H, D), bg, dtype=torch.bfloat16)
        for s, t in enumerate((inst.q, inst.k, inst.v)):
            full[torch.from_numpy(kept.astype(np.int64)), s] = t[0]
        d = ut.drop_background(torch.from_numpy(inst.fg_mask).to(DEV), full.to(DEV))
        p = d["x_packed"]
        q, k, v = (p[:, s].unsqueeze(0).contiguous() for s in range(3))
        idx = ut.build_block_index(torch.from_numpy(inst.block_mask).to(DEV))
        o, lse = ut.bsattn_fwd(q, k, v, idx, wl.block, 1 / math.sqrt(D))
        outs.append((o.view(torch.int16).cpu(), lse.cpu()))
    assert torch.isfinite(outs[0][1]).all()
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


# ---------------------------------------------------------------------------
# Workloads at their real sizes
# ---------------------------------------------------------------------------

_CACHE = {}


def workload(name, rho=None):
    key = (name, rho)
    if key not in _CACHE:
        _CACHE.clear()
        wl = W.WORKLOADS[name] if rho is None else W.WORKLOADS[name].with_rho(rho)
        inst = W.make(wl, with_do=True)
        case = {"q": inst.q, "k": inst.k, "v": inst.v, "do": inst.do,
                "block_mask": inst.block_mask, "block": wl.block, "scale": 1 / math.sqrt(wl.head_dim),
                "n": inst.n_kept, "wl": wl}
        case["gpu"] = run_gpu(case, backward=True)
        _CACHE[key] = case
    return _CACHE[key]


def _heads(case, heads):
    """Inputs restricted to some heads (the oracle's work is per head)."""
    sl = lambda t: t[:, :, heads, :].contiguous()
    return sl(case["q"]), sl(case["k"]), sl(case["v"]), sl(case["do"]), case["block_mask"][:, heads]


def test_tiny_full():
    c = workload("tiny")
    O, L = oracle.bsattn_fwd(c["q"], c["k"], c["v"], c["block_mask"], c["block"], c["scale"])
    check_out(c["gpu"]["o"], c["gpu"]["lse"], O, L, "tiny")
    dQ, dK, dV = oracle.bsattn_bwd(c["q"], c["k"], c["v"], c["do"], c["block_mask"], c["block"],
                                   c["scale"])
    check_grad(c["gpu"]["dq"], dQ, "tiny dq")
    check_grad(c["gpu"]["dk"], dK, "tiny dk")
    check_grad(c["gpu"]["dv"], dV, "tiny dv")


@pytest.mark.parametrize("name,rho,heads,nq,nk", [
    ("c512", None, [0, 23], 12, 3),
    ("c1k", None, [7], 8, 3),
    ("c2k", None, [0, 13], 8, 0),
    ("c2k_train", "0.05", [3], 6, 3),
    ("c2k_train", "0.1", [21], 6, 2),
    ("c2k_train", "0.2", [9], 6, 2),
    ("c2k_train", "1", [17], 3, 0),
])
def test_workload_sampled(name, rho, heads, nq, nk):
    c = workload(name, rho)
    n, blk = c["n"], c["block"]
    nb = -(-n // blk)
    rng = np.random.default_rng(nb)
    qb = sorted(set(rng.choice(nb - 1, nq - 1, replace=False).tolist()) | {nb - 1})
    q, k, v, do, bm = _heads(c, heads)
    O, L = oracle.bsattn_fwd(q, k, v, bm, blk, c["scale"], q_blocks=qb)
    g = c["gpu"]
    rows = block_rows(qb, blk, n)
    ht = torch.tensor(heads, device=DEV)
    sel = lambda t, r: t.index_select(1, torch.from_numpy(r).to(DEV)).index_select(2, ht)
    check_out(sel(g["o"], rows), g["lse"].index_select(1, ht)[:, :, torch.from_numpy(rows).to(DEV)],
              O[:, rows], L[:, :, rows], name)
    if not c["wl"].backward:
        return
    # dQ of the sampled query blocks; dK/dV of sampled key blocks, each from
    # every query block that selects it
    kb = sorted(set(rng.choice(nb - 1, max(nk - 1, 0), replace=False).tolist()) | {nb - 1}) if nk else []
    need = set(qb)
    for j in kb:
        need |= set(np.flatnonzero(bm[0, :, :, j].any(axis=0)).tolist())
    dQ, dK, dV = oracle.bsattn_bwd(q, k, v, do, bm, blk, c["scale"], q_blocks=sorted(need))
    check_grad(sel(g["dq"], rows), dQ[:, rows], f"{name} dq")
    if kb:
        krows = block_rows(kb, blk, n)
        check_grad(sel(g["dk"], krows), dK[:, krows], f"{name} dk")
        check_grad(sel(g["dv"], krows), dV[:, krows], f"{name} dv")

def test_full_size_unit_values():
    """2048-canvas forward with V = 1: every kept output is exactly 1."""
    c = workload("c2k")
    v1 = torch.ones_like(c["q"]).to(DEV)
    q, k = c["q"].to(DEV), c["k"].to(DEV)
    o, lse = ut.bsattn_fwd(q, k, v1, c["gpu"]["idx"], c["block"], c["scale"])
    assert torch.all(o == 1.0) and torch.isfinite(lse).all()
    assert torch.equal(lse, c["gpu"]["lse"])   # LSE does not depend on V
