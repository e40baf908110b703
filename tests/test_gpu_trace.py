"""The tracing aid on the GPU: with tracing on, each attention launch is
recorded under its kernel's name with a positive duration; the per-kernel
times of one backward call add up to no more than the call's own span
measured with events on the same stream; tracing off records nothing."""
import math

import numpy as np
import pytest
import torch

import paper_2609_23169_amd as ut

pytestmark = pytest.mark.gpu
DEV = "cuda"


def test_trace_records_attention_kernels():
    n, H, D, blk = 3000, 4, 128, 128
    g = torch.Generator(device=DEV).manual_seed(3)
    q, k, v, do = (torch.randn((1, n, H, D), generator=g, device=DEV).to(torch.bfloat16)
                   for _ in range(4))
    nb = -(-n // blk)
    bm = (np.random.default_rng(3).random((1, H, nb, nb)) < 0.4).astype(np.uint8)
    bm[0][:, np.arange(nb), np.arange(nb)] = 1
    idx = ut.build_block_index(torch.from_numpy(bm).to(DEV))
    scale = 1 / math.sqrt(D)
    torch.cuda.synchronize()
    ut.trace_read()                       # drop anything recorded before
    assert ut.ut_trace_enable(True) == ut.UT_OK
    try:
        o, lse = ut.bsattn_fwd(q, k, v, idx, blk, scale)
        ws = torch.empty(ut.ut_bsattn_bwd_workspace_size(1, n, H), dtype=torch.uint8, device=DEV)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        ut.bsattn_bwd(q, k, v, o, do, lse, idx, blk, scale, workspace=ws)
        e1.record()
        torch.cuda.synchronize()
        rec = {r["name"]: r for r in ut.trace_read()}
    finally:
        ut.ut_trace_enable(False)
    for name in ("bsattn_fwd<128,128>", "bwd_prep<128>", "bwd_dkdv<128,128>", "bwd_dq<128,128>"):
        assert name in rec, (name, sorted(rec))
        assert rec[name]["count"] == 1 and rec[name]["total_ms"] > 0
        assert rec[name]["min_ms"] == rec[name]["max_ms"] == rec[name]["total_ms"]
    span = e0.elapsed_time(e1)
    inner = sum(rec[x]["total_ms"] for x in ("bwd_prep<128>", "bwd_dkdv<128,128>", "bwd_dq<128,128>"))
    assert inner <= span * 1.02 + 0.01, (inner, span)
    # tracing off: nothing more is recorded
    ut.bsattn_fwd(q, k, v, idx, blk, scale)
    torch.cuda.synchronize()
    assert ut.trace_read() == []
