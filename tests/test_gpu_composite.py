"""GPU composite latent (Eq. 9) and alpha-to-token-grid masks (Sec. 3.2)
through the C ABI against the oracle, bit for bit (both are byte and index
work)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_23169_amd as ut
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"


def inverse_map(mask):
    kept = np.flatnonzero(mask)
    inv = np.full(mask.size, -1, dtype=np.int32)
    inv[kept] = np.arange(kept.size, dtype=np.int32)
    return kept, inv


@pytest.mark.parametrize("seed,V,P,C,frac,dtype", [
    (1, 6, 256, 64, 0.4, torch.float32), (2, 6, 256, 64, 0.4, torch.bfloat16), (3, 2, 7, 8, 0.5, torch.float32),
    (4, 1, 33, 16, 0.0, torch.bfloat16), (5, 3, 100, 32, 1.0, torch.float32), (6, 13, 64, 4, 0.3, torch.float32)])
def test_composite_bit_exact(seed, V, P, C, frac, dtype):
    rng = np.random.default_rng(seed)
    L = V * P
    kept, inv = inverse_map(rng.random(L) < frac)
    bg = torch.from_numpy(rng.standard_normal((P, C)).astype(np.float32)).to(dtype)
    packed = torch.from_numpy(rng.standard_normal((kept.size, C)).astype(np.float32)).to(dtype)
    got = ut.composite_latent(packed.to(DEV), torch.from_numpy(inv).to(DEV), bg.to(DEV), kept.size).cpu()
    u16 = torch.int16 if dtype == torch.bfloat16 else torch.int32
    ref = oracle.composite_latent(packed.view(u16).numpy(), kept, bg.view(u16).numpy(), L)
    assert np.array_equal(got.view(u16).numpy(), ref)


def test_composite_full_size_target_grid():
    wl = W.WORKLOADS["c2k"]
    inst = W.make(wl)
    P = wl.grid * wl.grid
    L = 6 * P
    kept, inv = inverse_map(inst.fg_mask[:L])
    rng = np.random.default_rng(21)
    bg = rng.standard_normal((P, 64)).astype(np.float32)
    packed = rng.standard_normal((kept.size, 64)).astype(np.float32)
    got = ut.composite_latent(torch.from_numpy(packed).to(DEV), torch.from_numpy(inv).to(DEV),
                              torch.from_numpy(bg).to(DEV), kept.size).cpu().numpy()
    ref = oracle.composite_latent(packed, kept, bg, L)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def _alpha(seed, V, H, W):
    """Ellipse-like foreground plus sparse specks, as in rendered alpha channels."""
    rng = np.random.default_rng(seed)
    yy, xx = np.mgrid[0:H, 0:W]
    a = np.zeros((V, H, W), dtype=np.uint8)
    for v in range(V):
        cy, cx = rng.uniform(0.3, 0.7) * H, rng.uniform(0.3, 0.7) * W
        ry, rx = rng.uniform(0.15, 0.35) * H, rng.uniform(0.15, 0.35) * W
        inside = ((yy - cy) / ry) ** 2 + ((xx - cx) / rx) ** 2 <= 1.0
        a[v][inside] = 255
        specks = rng.random((H, W)) < 2e-5
        a[v][specks] = rng.integers(1, 255, int(specks.sum()))
    return a


@pytest.mark.parametrize("V,H,W,patch,thr,radius", [
    (2, 256, 384, 16, 0, 1), (3, 512, 512, 16, 0, 0), (1, 256, 256, 32, 0, 2),
    (2, 192, 160, 16, 100, 1), (1, 64, 64, 16, 254, 3)])
def test_token_mask_bit_exact(V, H, W, patch, thr, radius):
    a = _alpha(V * 7 + H, V, H, W)
    got = ut.token_mask_from_alpha(torch.from_numpy(a).to(DEV), patch, thr, radius).cpu().numpy()
    ref = oracle.token_mask_from_alpha(a, patch, radius, threshold=thr)
    assert np.array_equal(got, ref)


def test_token_mask_full_size_2048():
    """Seven distinct 2048 x 2048 alpha masks (6 target/condition views and the
    reference) -> 128 x 128 token grids, dilation radius 1."""
    a = _alpha(31, 7, 2048, 2048)
    got = ut.token_mask_from_alpha(torch.from_numpy(a).to(DEV), 16, 0, 1).cpu().numpy()
    ref = oracle.token_mask_from_alpha(a, 16, 1)
    assert np.array_equal(got, ref)
