"""GPU parity of Background Token Dropping: compaction, gather and scatter are
compared with the oracle bit for bit (row bytes compared as int16)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_23169_amd as ut
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _mask(L, p, seed):
    rng = np.random.default_rng(seed)
    m = (rng.random(L) < p).astype(np.uint8)
    return m * rng.integers(1, 256, L).astype(np.uint8)   # any nonzero byte keeps


@pytest.mark.parametrize("L,p", [(1, 1.0), (1, 0.0), (15, 0.5), (16, 1.0), (17, 0.5),
                                 (4095, 0.3), (4096, 0.5), (4097, 0.9), (100000, 0.0),
                                 (100000, 1.0), (212992, 0.37), (1 << 20, 0.05)])
def test_compaction_bit_exact(L, p):
    m = _mask(L, p, L)
    kept_ref, inv_ref, n_ref = oracle.compact(m)
    d = ut.drop_background(torch.from_numpy(m).to(DEV))
    assert d["n_kept"] == n_ref
    assert np.array_equal(d["kept_idx"].cpu().numpy(), kept_ref)
    assert np.array_equal(d["inv_idx"].cpu().numpy(), inv_ref)


def test_compaction_unaligned_mask_pointer():
    m = _mask(9000, 0.5, 3)
    buf = torch.zeros(9001, dtype=torch.uint8, device=DEV)
    buf[1:] = torch.from_numpy(m).to(DEV)
    view = buf[1:]                                  # 1-byte offset pointer
    kept_ref, _, n_ref = oracle.compact(m)
    d = ut.drop_background(view)
    assert d["n_kept"] == n_ref and np.array_equal(d["kept_idx"].cpu().numpy(), kept_ref)


@pytest.mark.parametrize("L,row_elems,p", [(777, 8, 0.4), (5000, 24, 0.6), (4096, 3072, 0.35),
                                           (33, 64, 1.0), (50, 64, 0.0),
                                           # ~180K kept rows: more than one pass of the
                                           # gather grid, so waves take several rows
                                           (300000, 8, 0.6)])
def test_gather_scatter_bit_exact(L, row_elems, p):
    rng = np.random.default_rng(L + row_elems)
    m = _mask(L, p, L)
    bits = rng.integers(0, 1 << 16, size=(L, row_elems), dtype=np.uint16)   # NaNs included
    x = torch.from_numpy(bits.view(np.int16)).to(DEV).view(torch.bfloat16)
    kept_ref, _, n = oracle.compact(m)
    d = ut.drop_background(torch.from_numpy(m).to(DEV), x)
    assert d["n_kept"] == n
    got = d["x_packed"].view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, oracle.gather(bits, kept_ref))
    # write back into a sentinel-filled grid: kept rows replaced, others untouched
    pre = rng.integers(0, 1 << 16, size=(L, row_elems), dtype=np.uint16)
    full = torch.from_numpy(pre.view(np.int16)).to(DEV).view(torch.bfloat16)
    if n:
        packed = torch.from_numpy(rng.integers(0, 1 << 16, size=(n, row_elems), dtype=np.uint16)
                                  .view(np.int16)).to(DEV).view(torch.bfloat16)
        ut.scatter_foreground(packed, d["kept_idx"], full)
        ref = oracle.scatter(packed.view(torch.int16).cpu().numpy().view(np.uint16), kept_ref, pre)
    else:
        ref = pre
    assert np.array_equal(full.view(torch.int16).cpu().numpy().view(np.uint16), ref)


def test_capacity_overflow_reports_true_count():
    L = 10000
    m = _mask(L, 0.5, 9)
    kept_ref, _, n = oracle.compact(m)
    cap = n // 2
    kept = torch.full((cap,), -7, dtype=torch.int32, device=DEV)
    n_dev = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = torch.empty(ut.ut_drop_background_workspace_size(L), dtype=torch.uint8, device=DEV)
    st, nh = ut.ut_drop_background(torch.from_numpy(m).to(DEV), None, None, kept, None, n_dev, ws,
                                   n_kept_host=True)
    assert st == ut.UT_ERR_CAPACITY and nh == n and int(n_dev.item()) == n
    assert np.array_equal(kept.cpu().numpy(), kept_ref[:cap])


def test_full_size_hidden_state_gather_scatter():
    """The 2048-canvas workload: 212,992 x 3072 bf16 hidden state."""
    wl = W.WORKLOADS["c2k"]
    inst = W.make(wl, with_qkv=False, with_hidden=True)
    kept_ref, inv_ref, n = oracle.compact(inst.fg_mask)
    x = inst.hidden.to(DEV)
    d = ut.drop_background(torch.from_numpy(inst.fg_mask).to(DEV), x)
    assert d["n_kept"] == n == inst.n_kept
    assert np.array_equal(d["inv_idx"].cpu().numpy(), inv_ref)
    h16 = inst.hidden.view(torch.int16).numpy()
    assert np.array_equal(d["x_packed"].view(torch.int16).cpu().numpy(), oracle.gather(h16, kept_ref))
    # scatter the packed rows (negated bits) into a zero grid
    packed = (~d["x_packed"].view(torch.int16)).view(torch.bfloat16).contiguous()
    out = torch.zeros_like(x)
    ut.scatter_foreground(packed, d["kept_idx"], out)
    ref = oracle.scatter(packed.view(torch.int16).cpu().numpy(), kept_ref,
                         np.zeros_like(h16))
    assert np.array_equal(out.view(torch.int16).cpu().numpy(), ref)
