"""GPU parity of the block index: row and column lists bit-exact vs the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_23169_amd as ut
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _check(bm):
    rp, cols, cp, rows = oracle.block_index(bm)
    idx = ut.build_block_index(torch.from_numpy(bm).to(DEV))
    nnz = idx["nnz"]
    assert nnz == rp[-1]
    assert np.array_equal(idx["q_rowptr"].cpu().numpy(), rp)
    assert np.array_equal(idx["kv_colptr"].cpu().numpy(), cp)
    assert np.array_equal(idx["q_cols"][:nnz].cpu().numpy(), cols)
    assert np.array_equal(idx["kv_rows"][:nnz].cpu().numpy(), rows)


@pytest.mark.parametrize("B,H,Nq,Nk,p", [(1, 1, 1, 1, 1.0), (1, 1, 1, 1, 0.0), (1, 3, 7, 7, 0.3),
                                         (2, 2, 13, 70, 0.5), (1, 4, 65, 63, 0.2),
                                         (1, 2, 130, 130, 1.0), (1, 1, 200, 200, 0.0),
                                         (3, 5, 64, 64, 0.5), (1, 2, 129, 1, 0.7),
                                         # more than 16 row tiles: waves of the column
                                         # lists walk two or three tiles each
                                         (1, 2, 1100, 90, 0.3), (1, 1, 3000, 40, 0.1),
                                         (1, 1, 2048, 64, 1.0),
                                         # 17,600 row counts: the scan takes two passes
                                         (2, 8, 1100, 33, 0.05),
                                         # 1,500 columns: three passes of row chunks
                                         (1, 1, 50, 1500, 0.4)])
def test_random_masks(B, H, Nq, Nk, p):
    rng = np.random.default_rng(B * 100 + H * 10 + Nq)
    _check((rng.random((B, H, Nq, Nk)) < p).astype(np.uint8) * 3)


@pytest.mark.parametrize("name,rho", [("tiny", None), ("c512", None), ("c1k", None), ("c2k", None),
                                      ("c2k_train", "0.05"), ("c2k_train", "0.2"),
                                      ("c2k_train", "1")])
def test_workload_masks(name, rho):
    wl = W.WORKLOADS[name]
    if rho:
        wl = wl.with_rho(rho)
    _check(W.make(wl, with_qkv=False).block_mask)


def test_capacity_overflow():
    bm = np.ones((1, 2, 10, 10), np.uint8)
    dev = torch.from_numpy(bm).to(DEV)
    rp = torch.empty(21, dtype=torch.int32, device=DEV)
    cp = torch.empty(21, dtype=torch.int32, device=DEV)
    cols = torch.empty(150, dtype=torch.int32, device=DEV)
    rows = torch.empty(150, dtype=torch.int32, device=DEV)
    st, nnz = ut.ut_build_block_index(dev, rp, cols, cp, rows, nnz_host=True)
    assert st == ut.UT_ERR_CAPACITY and nnz == 200
    assert np.array_equal(rp.cpu().numpy(), np.arange(0, 201, 10))
