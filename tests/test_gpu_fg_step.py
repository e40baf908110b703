"""GPU foreground-only Euler update (Eq. 4) and foreground flow-matching loss
(Eq. 3) through the C ABI against the float64 oracle.

Euler: every element is one fp32 fused multiply-add, so a kept row is within
one fp32 ulp of the exact result (the oracle's float64 value rounded to fp32
can differ from the single rounding only at a rounding tie), and every other
row is bit-identical to the input. Loss: differences and squares in fp64,
summed in a fixed order, so loss and gradient agree with the oracle to one
fp32 ulp after their final rounding, and two runs agree bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_23169_amd as ut
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"


def ulp_close(got, ref64, ulps=1):
    """|got - fp32(ref64)| <= ulps fp32 spacings of fp32(ref64), elementwise."""
    ref32 = np.asarray(ref64).astype(np.float32)
    spacing = np.spacing(np.abs(ref32)).astype(np.float64)
    return np.all(np.abs(np.asarray(got).astype(np.float64) - ref32.astype(np.float64)) <= ulps * spacing)


def case(seed, L, C, frac, vdtype, xdtype=torch.float32):
    g = torch.Generator().manual_seed(seed)
    kept = torch.nonzero(torch.rand(L, generator=g) < frac).flatten().to(torch.int32)
    z = torch.randn((L, C), generator=g)
    v = torch.randn((kept.numel(), C), generator=g).to(vdtype)
    eps = torch.randn((L, C), generator=g).to(xdtype)
    z0 = torch.randn((L, C), generator=g).to(xdtype)
    return kept, z, v, eps, z0


SHAPES = [(1, 5000, 64, 0.4), (2, 777, 4, 0.9), (3, 3000, 12, 0.05), (4, 64, 16, 1.0),
          (5, 1, 8, 1.0), (6, 4096, 64, 0.0)]


@pytest.mark.parametrize("vdtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("seed,L,C,frac", SHAPES)
def test_euler_update(seed, L, C, frac, vdtype):
    kept, z, v, _, _ = case(seed, L, C, frac, vdtype)
    dt = -0.0625 + 0.001 * seed
    zg = z.to(DEV)
    ut.euler_update_foreground(zg, v.to(DEV), kept.to(DEV), dt)
    got = zg.cpu().numpy()
    ref = oracle.euler_update_fg(z, v, kept.numpy(), float(np.float32(dt)))
    mask = np.zeros(L, bool)
    mask[kept.numpy()] = True
    assert np.array_equal(got[~mask].view(np.uint32), z.numpy()[~mask].view(np.uint32))
    assert ulp_close(got[mask], ref[mask])


@pytest.mark.parametrize("vdtype,xdtype", [(torch.bfloat16, torch.float32), (torch.float32, torch.float32),
                                           (torch.bfloat16, torch.bfloat16)])
@pytest.mark.parametrize("seed,L,C,frac", SHAPES)
def test_fg_flow_loss(seed, L, C, frac, vdtype, xdtype):
    kept, _, v, eps, z0 = case(seed, L, C, frac, vdtype, xdtype)
    args = (v.to(DEV), eps.to(DEV), z0.to(DEV), kept.to(DEV))
    loss, grad = ut.fg_flow_loss(*args)
    loss2, _ = ut.fg_flow_loss(*args, with_grad=False)
    torch.cuda.synchronize()
    ref_loss, ref_grad = oracle.fg_flow_loss(v, eps, z0, kept.numpy())
    assert ulp_close(loss.cpu().numpy(), np.array([ref_loss]))
    assert loss.cpu().numpy().view(np.uint32) == loss2.cpu().numpy().view(np.uint32)   # deterministic
    assert ulp_close(grad.cpu().numpy(), ref_grad)


def test_loss_never_reads_background_rows():
    kept, _, v, eps, z0 = case(7, 2000, 64, 0.3, torch.bfloat16)
    mask = torch.zeros(2000, dtype=torch.bool)
    mask[kept.long()] = True
    eps_nan, z0_nan = eps.clone(), z0.clone()
    eps_nan[~mask] = float("nan")
    z0_nan[~mask] = float("nan")
    a, _ = ut.fg_flow_loss(v.to(DEV), eps.to(DEV), z0.to(DEV), kept.to(DEV))
    b, _ = ut.fg_flow_loss(v.to(DEV), eps_nan.to(DEV), z0_nan.to(DEV), kept.to(DEV))
    assert a.item() == b.item()


def test_full_size_target_grid():
    """The 2048-canvas target views: 6 x 128 x 128 token grid, 64 latent channels,
    the retained target positions of the workload's foreground masks."""
    wl = W.WORKLOADS["c2k"]
    inst = W.make(wl)
    L = 6 * wl.grid * wl.grid
    kept = torch.from_numpy(np.flatnonzero(inst.fg_mask[:L]).astype(np.int32))
    g = torch.Generator().manual_seed(11)
    C = 64
    z = torch.randn((L, C), generator=g)
    v = torch.randn((kept.numel(), C), generator=g).to(torch.bfloat16)
    eps = torch.randn((L, C), generator=g)
    zg = z.to(DEV)
    ut.euler_update_foreground(zg, v.to(DEV), kept.to(DEV), -1.0 / 28)
    ref = oracle.euler_update_fg(z, v, kept.numpy(), float(np.float32(-1.0 / 28)))
    assert ulp_close(zg.cpu().numpy(), ref)
    loss, grad = ut.fg_flow_loss(v.to(DEV), eps.to(DEV), z.to(DEV), kept.to(DEV))
    rl, rg = oracle.fg_flow_loss(v, eps, z, kept.numpy())
    assert ulp_close(loss.cpu().numpy(), np.array([rl])) and ulp_close(grad.cpu().numpy(), rg)
