"""Seeded synthetic inputs shaped like UltraTex's multi-view workloads.

This module only draws inputs. It holds none of the method's arithmetic (no
compaction, no block lists, no attention), so the CPU oracle and the HIP path
can both consume its output without sharing any code of the method.

Layout of the unified sequence (paper, Sec. 3.1 "In-Context Multi-View
Diffusion"): `m` noisy target views, then `m` normal-map condition views, then
one reference view, each a g x g token grid (canvas / 8 for the VAE, / 2 for
the 2x2 patchify, so g = canvas / 16). At a 2048 canvas g = 128 and the
sequence is 13 x 16,384 = 212,992 tokens.

Foreground masks (Sec. 3.2 "Mask Construction and Sequence Compression"): the
m target-view masks are shared by the m condition views; the reference view
has its own mask. The real masks come from rendered alpha channels, which are
not available here; each distinct mask is a seeded filled ellipse whose area
is a seeded fraction of the grid, in the foreground-ratio ranges of the
workloads (the dataset statistics are in the supplementary "Foreground Ratio
Statistics").

Block masks (Sec. 3.3, Eq. 7): the paper keeps exactly floor(rho * N_k) key
blocks per (head, query block) by Top-K over pooled scores. The synthetic
stand-in keeps the diagonal block plus exactly min(floor(rho * N_k), N_k - 1)
other key blocks drawn uniformly without replacement, so every row carries a
fixed count like the paper's Top-K and the work is deterministic per seed.

Random streams: numpy SeedSequence(seed).spawn(7) in the fixed order
[fg masks, Q, K, V, dO, block mask, hidden state].
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from fractions import Fraction

import numpy as np

STREAMS = ("fg", "q", "k", "v", "do", "block", "hidden")


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: sequence layout, attention shape, sparsity."""

    name: str
    seed: int
    m_views: int           # target views (= condition views); +1 reference
    grid: int              # tokens per side of one view's token grid
    fg_lo: float           # foreground fraction range per distinct mask
    fg_hi: float
    disk: bool             # True: circles (axis ratio 1); False: ellipses
    heads: int
    head_dim: int
    block: int
    rho: str               # retention ratio as an exact decimal string
    backward: bool
    hidden: int = 0        # hidden width of the gather/scatter state (0: none)
    batch: int = 1

    @property
    def views(self) -> int:
        return 2 * self.m_views + 1

    @property
    def seq_len(self) -> int:
        return self.views * self.grid * self.grid

    def with_rho(self, rho: str) -> "Workload":
        return replace(self, rho=rho, name=f"{self.name.split('@')[0]}@rho={rho}")


# The five workloads: a tiny CPU-checkable case and the 512 / 1K / 2K canvases.
WORKLOADS = {
    "tiny": Workload("tiny", 1, 1, 16, 0.5, 0.5, True, 2, 64, 64, "0.4", True),
    "c512": Workload("c512", 2, 6, 32, 0.40, 0.55, False, 24, 128, 128, "0.3", False),
    "c1k": Workload("c1k", 3, 6, 64, 0.35, 0.50, False, 24, 128, 128, "0.2", True),
    "c2k": Workload("c2k", 4, 6, 128, 0.30, 0.45, False, 24, 128, 128, "0.1", False,
                    hidden=3072),
    "c2k_train": Workload("c2k_train", 5, 6, 128, 0.30, 0.45, False, 24, 128, 128, "0.1",
                          True, hidden=3072),
}
TRAIN_RHOS = ("0.05", "0.1", "0.2", "1")


def streams(seed: int) -> dict:
    ss = np.random.SeedSequence(seed).spawn(len(STREAMS))
    return {name: np.random.default_rng(s) for name, s in zip(STREAMS, ss)}


def _ellipse_mask(g: int, frac: float, cx: float, cy: float, ratio: float,
                  theta: float) -> np.ndarray:
    """Filled ellipse on a g x g grid; the token (y, x) is kept iff its centre
    (x + 1/2, y + 1/2) lies inside. The scale is bisected until the kept count
    is within 0.5% of round(frac * g^2) (or as close as the grid allows)."""
    target = int(round(frac * g * g))
    ys, xs = np.mgrid[0:g, 0:g].astype(np.float64)
    dx, dy = xs + 0.5 - cx, ys + 0.5 - cy
    c, s = math.cos(theta), math.sin(theta)
    u = dx * c + dy * s
    w = -dx * s + dy * c
    # Inside test for semi-axes (a, ratio * a): (u/a)^2 + (w/(ratio a))^2 <= 1,
    # i.e. rad <= a^2 with rad = u^2 + (w/ratio)^2. Count is monotone in a.
    rad = u * u + (w / ratio) ** 2
    lo, hi = 0.0, float(4 * g * g)
    best = None
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        cnt = int((rad <= mid).sum())
        if best is None or abs(cnt - target) < abs(best[1] - target):
            best = (mid, cnt)
        if abs(cnt - target) <= 0.005 * target:
            break
        if cnt < target:
            lo = mid
        else:
            hi = mid
    return (rad <= best[0]).astype(np.uint8)


def fg_masks(wl: Workload, rng: np.random.Generator | None = None) -> np.ndarray:
    """Per-view token-grid foreground masks, uint8 [views, g, g], with the
    target masks shared by the condition views and an own reference mask."""
    rng = rng if rng is not None else streams(wl.seed)["fg"]
    g, m = wl.grid, wl.m_views
    distinct = []
    for _ in range(m + 1):
        frac = rng.uniform(wl.fg_lo, wl.fg_hi)
        cx, cy = rng.uniform(0.35 * g, 0.65 * g, size=2)
        ratio = 1.0 if wl.disk else rng.uniform(0.6, 1.0)
        theta = rng.uniform(0.0, math.pi)
        distinct.append(_ellipse_mask(g, frac, cx, cy, ratio, theta))
    views = distinct[:m] + distinct[:m] + [distinct[m]]
    return np.stack(views).astype(np.uint8)


def kept_off_diagonal(rho: str, nk: int) -> int:
    """Off-diagonal key blocks kept per row: min(floor(rho * N_k), N_k - 1),
    with rho taken as an exact decimal so that e.g. 0.3 * 50 is exactly 15."""
    return min(math.floor(Fraction(rho) * nk), nk - 1)


def block_mask(batch: int, heads: int, nq: int, nk: int, rho: str,
               rng: np.random.Generator) -> np.ndarray:
    """uint8 [B, H, Nq, Nk]: diagonal plus exactly kept_off_diagonal(rho, Nk)
    off-diagonal key blocks per row, uniform without replacement."""
    if Fraction(rho) >= 1:
        return np.ones((batch, heads, nq, nk), dtype=np.uint8)
    koff = kept_off_diagonal(rho, nk)
    out = np.zeros((batch, heads, nq, nk), dtype=np.uint8)
    diag = np.arange(min(nq, nk))
    out[:, :, diag, diag] = 1
    if koff > 0:
        keys = rng.random((batch, heads, nq, nk))
        # the diagonal can never be drawn as an off-diagonal block
        keys[:, :, diag, diag] = np.inf
        pick = np.argpartition(keys, koff - 1, axis=-1)[..., :koff]
        np.put_along_axis(out, pick, 1, axis=-1)
    return out


@dataclass
class Instance:
    """All inputs of one workload instance (host arrays / CPU tensors)."""

    wl: Workload
    fg_mask: np.ndarray          # uint8 [L] flat, view-major then row-major
    n_kept: int
    block_mask: np.ndarray       # uint8 [B, H, Nq, Nk]
    q: "object" = None           # torch bf16 [B, N, H, D] (CPU)
    k: "object" = None
    v: "object" = None
    do: "object" = None
    hidden: "object" = None      # torch bf16 [L, C] of random bit patterns
    extras: dict = field(default_factory=dict)


def _bf16_normal(rng: np.random.Generator, shape) -> "object":
    import torch
    x = rng.standard_normal(shape, dtype=np.float32)
    return torch.from_numpy(x).to(torch.bfloat16)   # round-to-nearest-even


def make(wl: Workload, with_qkv: bool = True, with_do: bool | None = None,
         with_hidden: bool = False) -> Instance:
    """Draw one instance. N (the kept-token count) follows from the masks."""
    st = streams(wl.seed)
    fg = fg_masks(wl, st["fg"]).reshape(-1)
    n = int(np.count_nonzero(fg))
    nb = -(-n // wl.block)
    bm = block_mask(wl.batch, wl.heads, nb, nb, wl.rho, st["block"])
    inst = Instance(wl, fg, n, bm)
    shape = (wl.batch, n, wl.heads, wl.head_dim)
    if with_qkv:
        inst.q = _bf16_normal(st["q"], shape)
        inst.k = _bf16_normal(st["k"], shape)
        inst.v = _bf16_normal(st["v"], shape)
    if with_do if with_do is not None else (with_qkv and wl.backward):
        inst.do = _bf16_normal(st["do"], shape)
    if with_hidden and wl.hidden:
        import torch
        bits = st["hidden"].integers(0, 1 << 16, size=(wl.seq_len, wl.hidden),
                                     dtype=np.uint16)
        inst.hidden = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16)
    return inst


def random_case(seed: int, n: int, heads: int, head_dim: int, block: int,
                density: float, batch: int = 1, diag: bool = True,
                empty_rows: int = 0) -> dict:
    """Small seeded attention case for parity tests: bf16 Q/K/V/dO [B,N,H,D]
    and a block mask with per-entry density (diagonal optional) and a number of
    rows forced empty."""
    import torch
    rng = np.random.default_rng(seed)
    shape = (batch, n, heads, head_dim)
    q, k, v, do = (_bf16_normal(rng, shape) for _ in range(4))
    nb = -(-n // block)
    bm = (rng.random((batch, heads, nb, nb)) < density).astype(np.uint8)
    if diag:
        idx = np.arange(nb)
        bm[:, :, idx, idx] = 1
    for _ in range(empty_rows):
        b, h, i = rng.integers(0, batch), rng.integers(0, heads), rng.integers(0, nb)
        bm[b, h, i, :] = 0
    return {"q": q, "k": k, "v": v, "do": do, "block_mask": bm, "n": n,
            "block": block, "scale": 1.0 / math.sqrt(head_dim)}


def varlen_case(seed: int, lens, heads: int, head_dim: int, block: int, density: float,
                garbage_past_end: bool = True) -> dict:
    """Seeded packed batch of samples with the given token counts: bf16
    Q/K/V/dO [T, H, D] back to back, int32 offsets cu_seqlens [B + 1], and a
    block mask [B, H, Nb, Nb] (Nb from the longest sample) with per-entry
    density and the diagonal set within each sample. With garbage_past_end the
    entries past a sample's own blocks are random too (they must be ignored);
    otherwise they are 0."""
    rng = np.random.default_rng(seed)
    lens = [int(x) for x in lens]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T, nb = int(cu[-1]), max(1, -(-max(lens) // block))
    q, k, v, do = (_bf16_normal(rng, (T, heads, head_dim)) for _ in range(4))
    bm = (rng.random((len(lens), heads, nb, nb)) < density).astype(np.uint8)
    for b, n in enumerate(lens):
        own = -(-n // block)
        if not garbage_past_end:
            bm[b, :, own:, :] = 0
            bm[b, :, :, own:] = 0
        d = np.arange(own)
        bm[b][:, d, d] = 1
    return {"q": q, "k": k, "v": v, "do": do, "cu_seqlens": cu, "block_mask": bm,
            "lens": lens, "max_seqlen": max(max(lens), 1), "block": block,
            "scale": 1.0 / math.sqrt(head_dim)}


def varlen_case_device(seed: int, lens, heads: int, head_dim: int, block: int, density: float,
                       device) -> dict:
    """`varlen_case` for sizes too large to draw on the host: Q/K/V/dO come
    from a seeded torch generator on `device` (N(0, 1) in fp32, rounded to
    bf16); the offsets and the block mask (entries past each sample's blocks
    zero) come from numpy as in `varlen_case`."""
    import torch
    rng = np.random.default_rng(seed)
    lens = [int(x) for x in lens]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T, nb = int(cu[-1]), max(1, -(-max(lens) // block))
    bm = (rng.random((len(lens), heads, nb, nb)) < density).astype(np.uint8)
    for b, n in enumerate(lens):
        own = -(-n // block)
        bm[b, :, own:, :] = 0
        bm[b, :, :, own:] = 0
        d = np.arange(own)
        bm[b][:, d, d] = 1
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    q, k, v, do = (torch.randn((T, heads, head_dim), generator=g, device=device).to(torch.bfloat16)
                   for _ in range(4))
    return {"q": q, "k": k, "v": v, "do": do, "cu_seqlens": cu, "block_mask": bm, "lens": lens,
            "max_seqlen": max(max(lens), 1), "block": block, "scale": 1.0 / math.sqrt(head_dim)}


def bucket_lengths(seed: int, wl: Workload, count: int) -> list:
    """Kept-token counts of `count` samples of one foreground-count bucket of a
    workload: each sample's count is its own draw of the workload's foreground
    masks (Sec. 4.1 buckets training samples by this count). The counts are
    sorted, as bucketing by count would order them."""
    rng = np.random.default_rng(seed)
    return sorted(int(fg_masks(wl, rng).sum()) for _ in range(count))


def block_sizes(n: int, block: int) -> np.ndarray:
    """Real token count of each block of an N-token sequence (last may be short)."""
    nb = -(-n // block)
    return np.array([min(n, (j + 1) * block) - j * block for j in range(nb)],
                    dtype=np.int64)


def retained_flops_fwd(block_mask: np.ndarray, n: int, block: int, head_dim: int) -> int:
    """Algorithmic forward FLOPs over retained block pairs only: Q_i K_j^T and
    P_ij V_j cost 2 * r_i * c_j * d each, r_i and c_j the real token counts of
    blocks i and j. The backward's five products (S recompute, dV, dP, dQ, dK)
    count 2.5x this. Skipped pairs and dense-equivalent work are not counted."""
    sz = block_sizes(n, block)
    pairs = np.einsum("bhij,i,j->", np.asarray(block_mask, dtype=np.int64), sz, sz)
    return int(4 * head_dim * pairs)
