"""CPU oracle for the UltraTex foreground hot path -- TEST INFRASTRUCTURE ONLY.

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this module. The product path (the HIP library and its Python
binding) never imports, calls or links it, and this module imports nothing of
the product path: the two share no code. Inputs come from `workloads`, which
holds none of the method's arithmetic.

Every function is a plain, slow, direct statement of what the paper defines,
in float64 (bf16 inputs are upcast exactly). Where the paper is silent the
reading taken is stated in the docstring.

Paper sections (arXiv 2609.23169, "UltraTex"):
  * Background Token Dropping: Sec. 3.2, "Mask Construction and Sequence
    Compression" (retained positions M_fg, the Gather_{M_fg} operator that
    concatenates them) and "Efficient Inference" (Eq. 4: only positions in M_fg
    are written back; Eq. 9: the composite latent keeps every other position).
  * Block-Sparse Attention: Sec. 3.3, Eq. 5 (dense softmax attention with
    scale 1/sqrt(d)), the b_q / b_kv block partition, Eq. 7 (binary block mask
    M_c) and Eq. 8 (each query block attends only to its selected key blocks).
  * Foreground-restricted training and sampling: Sec. 3.2, Eq. 3 (the flow
    matching loss over the gathered foreground target tokens, with the target
    velocity eps - z_tgt of Eq. 1-2) and Eq. 4 (the Euler step applied only
    at the retained positions).
  * Foreground-aware decoding input: Sec. 3.4, Eq. 9 (the composite latent:
    denoised foreground at the retained positions, the canonical background
    latent tile-repeated over the views elsewhere) and the mask construction
    of Sec. 3.2 (alpha masks brought to the 1/16 token grid and slightly
    dilated).
  * Top-K block selection: Sec. 3.3, Eq. 6 (compressed scores from
    mean-pooled query and key blocks) and Eq. 7 (row-wise Top-K over the key
    blocks gives the block mask).
  * The backward pass: the paper trains its third stage with block-sparse
    attention but prints no gradient formula; the oracle differentiates Eq. 8
    with the mask held constant (the standard softmax-attention gradient
    restricted to the retained pairs).
  * Batches of differing lengths: training buckets samples by their
    foreground token count (Sec. 4.1, Implementation Details), so the kept
    counts within a batch are close but not equal. The reading taken: the
    samples are packed back to back and each is its own Eq. 8 problem.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "compact", "gather", "scatter", "block_index",
    "bsattn_fwd", "bsattn_bwd", "bsattn_fwd_varlen", "bsattn_bwd_varlen",
    "block_pool", "topk_block_mask",
    "euler_update_fg", "fg_flow_loss",
    "composite_latent", "token_mask_from_alpha",
]


# ---------------------------------------------------------------------------
# Background Token Dropping (Sec. 3.2)
# ---------------------------------------------------------------------------

def compact(fg_mask) -> tuple[np.ndarray, np.ndarray, int]:
    """The retained set M_fg of a flat per-view foreground mask.

    Returns (kept_idx, inv_idx, n_kept): kept_idx lists the positions p with a
    nonzero mask byte in ascending p (the paper concatenates the retained
    tokens; ascending original order is the reading taken, view-major and
    row-major as the unified sequence is laid out); inv_idx[p] is the packed
    index of p, or -1 for a dropped position.
    """
    flags = np.asarray(fg_mask).reshape(-1).tolist()
    inv = np.full(len(flags), -1, dtype=np.int32)
    kept = []
    for p, f in enumerate(flags):
        if f != 0:
            inv[p] = len(kept)
            kept.append(p)
    return np.asarray(kept, dtype=np.int32), inv, len(kept)


def gather(x_full: np.ndarray, kept_idx: np.ndarray) -> np.ndarray:
    """Gather_{M_fg}: packed row k is full row kept_idx[k] (a byte copy)."""
    return np.asarray(x_full)[np.asarray(kept_idx, dtype=np.int64)]


def scatter(x_packed: np.ndarray, kept_idx: np.ndarray,
            x_full_prefilled: np.ndarray) -> np.ndarray:
    """Write packed row k back to full row kept_idx[k]; every other row keeps
    its prior contents (the background noise of Eq. 4, or z_bg of Eq. 9)."""
    out = np.array(x_full_prefilled, copy=True)
    out[np.asarray(kept_idx, dtype=np.int64)] = x_packed
    return out


# ---------------------------------------------------------------------------
# Block index (Sec. 3.3, Eq. 7 and the sets S_i of Eq. 8)
# ---------------------------------------------------------------------------

def block_index(block_mask: np.ndarray):
    """Row lists S_i and their transpose from a block mask [B, H, Nq, Nk].

    Returns (rowptr, cols, colptr, rows) as int32 arrays. Row r = (b*H + h)*Nq
    + i lists S_i = {j : M_c[b,h,i,j] = 1} in ascending j between rowptr[r]
    and rowptr[r+1]. Column c = (b*H + h)*Nk + j lists {i : M_c[b,h,i,j] = 1}
    in ascending i between colptr[c] and colptr[c+1].
    """
    m = np.asarray(block_mask)
    B, H, Nq, Nk = m.shape
    rowptr, cols = [0], []
    for b in range(B):
        for h in range(H):
            for i in range(Nq):
                s_i = np.flatnonzero(m[b, h, i, :])
                cols.extend(s_i.tolist())
                rowptr.append(len(cols))
    colptr, rows = [0], []
    for b in range(B):
        for h in range(H):
            for j in range(Nk):
                t_j = np.flatnonzero(m[b, h, :, j])
                rows.extend(t_j.tolist())
                colptr.append(len(rows))
    as32 = lambda a: np.asarray(a, dtype=np.int32)
    return as32(rowptr), as32(cols), as32(colptr), as32(rows)


# ---------------------------------------------------------------------------
# Block-sparse attention (Sec. 3.3, Eq. 5 and Eq. 8)
# ---------------------------------------------------------------------------

def _f64(x, dtype=np.float64) -> np.ndarray:
    """Exact upcast of a bf16 torch tensor (or any array) to float64 (or to
    float32, also exact for bf16 inputs)."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            tt = torch.float64 if np.dtype(dtype) == np.float64 else torch.float32
            return x.detach().to(tt).numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.asarray(x, dtype=dtype)


def _block_tokens(j: int, block: int, n: int) -> np.ndarray:
    """Token rows of block j: the partition of Sec. 3.3, with a shorter last
    block when N is not a multiple of the block size (the paper assumes
    divisibility; a ragged tail is the reading taken)."""
    return np.arange(j * block, min(n, (j + 1) * block))


def _selected_keys(mask_row: np.ndarray, block: int, n: int) -> np.ndarray:
    """Token indices of all key blocks in S_i, ascending."""
    sel = np.flatnonzero(mask_row)
    if sel.size == 0:
        return np.zeros(0, dtype=np.int64)
    return np.concatenate([_block_tokens(j, block, n) for j in sel])


def bsattn_fwd(q, k, v, block_mask, block: int, scale: float,
               q_blocks=None, dtype=np.float64):
    """Eq. 8: O_i = softmax(Q_i K_{S_i}^T * scale) V_{S_i} per (batch, head,
    query block i), plus the natural-log log-sum-exp of each query row's
    scaled scores over the keys it attends to.

    q, k, v: [B, N, H, D]; block_mask: [B, H, Nq, Nk] with Nq = Nk =
    ceil(N / block). q_blocks: optional iterable of query-block indices to
    compute (rows of other blocks are left NaN). A query block whose S_i is
    empty attends to nothing: its rows are O = 0 and LSE = -inf (the paper
    never produces such a row; this is the reading taken).

    Returns (O [B, N, H, D], LSE [B, H, N]) in float64. dtype=np.float32
    runs the same arithmetic in float32 (used only to time a CPU baseline;
    every check uses float64).
    """
    Q, K, V = _f64(q, dtype), _f64(k, dtype), _f64(v, dtype)
    m = np.asarray(block_mask)
    B, N, H, D = Q.shape
    Nq = m.shape[2]
    O = np.full((B, N, H, D), np.nan, dtype=dtype)
    LSE = np.full((B, H, N), np.nan, dtype=dtype)
    blocks = range(Nq) if q_blocks is None else q_blocks
    for b in range(B):
        for h in range(H):
            for i in blocks:
                rows = _block_tokens(i, block, N)
                keys = _selected_keys(m[b, h, i], block, N)
                if keys.size == 0:
                    O[b, rows, h, :] = 0.0
                    LSE[b, h, rows] = -np.inf
                    continue
                S = (Q[b, rows, h, :] @ K[b, keys, h, :].T) * Q.dtype.type(scale)
                mx = S.max(axis=1, keepdims=True)
                E = np.exp(S - mx)
                l = E.sum(axis=1, keepdims=True)
                O[b, rows, h, :] = (E @ V[b, keys, h, :]) / l
                LSE[b, h, rows] = mx[:, 0] + np.log(l[:, 0])
    return O, LSE


def bsattn_bwd(q, k, v, dout, block_mask, block: int, scale: float,
               q_blocks=None, dtype=np.float64):
    """Gradients of Eq. 8 for a loss whose gradient w.r.t. O is dout.

    The block mask is a constant. With P = softmax(S) over the retained keys of
    each row, S = Q K^T * scale:
        dV = P^T dO,   dP = dO V^T,   delta_r = sum_c P_rc dP_rc,
        dS = P o (dP - delta),   dQ = scale * dS K,   dK = scale * dS^T Q.
    Pairs outside the mask contribute nothing. Rows with an empty S_i have
    zero gradients.

    q_blocks: optional subset of query blocks whose contributions are summed
    (dQ of other rows is NaN; dK and dV then hold only the listed blocks'
    contributions). Returns (dQ, dK, dV) [B, N, H, D] float64 (float32 with
    dtype=np.float32, as for bsattn_fwd).
    """
    Q, K, V, dO = _f64(q, dtype), _f64(k, dtype), _f64(v, dtype), _f64(dout, dtype)
    m = np.asarray(block_mask)
    B, N, H, D = Q.shape
    Nq = m.shape[2]
    sc = Q.dtype.type(scale)
    dQ = np.full((B, N, H, D), np.nan, dtype=dtype)
    dK = np.zeros((B, N, H, D), dtype=dtype)
    dV = np.zeros((B, N, H, D), dtype=dtype)
    blocks = range(Nq) if q_blocks is None else q_blocks
    for b in range(B):
        for h in range(H):
            for i in blocks:
                rows = _block_tokens(i, block, N)
                keys = _selected_keys(m[b, h, i], block, N)
                dQ[b, rows, h, :] = 0.0
                if keys.size == 0:
                    continue
                Qi, Kk, Vk, dOi = Q[b, rows, h], K[b, keys, h], V[b, keys, h], dO[b, rows, h]
                S = (Qi @ Kk.T) * sc
                E = np.exp(S - S.max(axis=1, keepdims=True))
                P = E / E.sum(axis=1, keepdims=True)
                dP = dOi @ Vk.T
                delta = (P * dP).sum(axis=1, keepdims=True)
                dS = P * (dP - delta)
                dQ[b, rows, h, :] = sc * (dS @ Kk)
                dK[b, keys, h, :] += sc * (dS.T @ Qi)
                dV[b, keys, h, :] += P.T @ dOi
    return dQ, dK, dV



def _varlen_samples(cu_seqlens, block: int):
    """(b, first token, length, blocks) of each packed sample."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    for b in range(cu.size - 1):
        n = int(cu[b + 1] - cu[b])
        yield b, int(cu[b]), n, -(-n // block)


def bsattn_fwd_varlen(q, k, v, cu_seqlens, block_mask, block: int, scale: float):
    """Eq. 8 over packed samples of differing lengths.

    q, k, v: [T, H, D], sample b being tokens cu_seqlens[b] .. cu_seqlens[b+1]
    - 1; block_mask: [B, H, Nb, Nb] for the longest sample. Sample b is the
    uniform problem of `bsattn_fwd` on its own tokens with the leading
    ceil(n_b / block) rows and columns of block_mask[b]; entries past them do
    not exist for it and are ignored (reading taken). Tokens attend only
    within their own sample. Returns (O [T, H, D], LSE [H, T]) in float64;
    tokens outside every sample stay NaN.
    """
    Q, K, V = _f64(q), _f64(k), _f64(v)
    m = np.asarray(block_mask)
    T, H, D = Q.shape
    O = np.full((T, H, D), np.nan)
    LSE = np.full((H, T), np.nan)
    for b, t0, n, nb in _varlen_samples(cu_seqlens, block):
        if n == 0:
            continue
        sl = slice(t0, t0 + n)
        Ob, Lb = bsattn_fwd(Q[None, sl], K[None, sl], V[None, sl], m[b:b + 1, :, :nb, :nb],
                            block, scale)
        O[sl] = Ob[0]
        LSE[:, sl] = Lb[0]
    return O, LSE


def bsattn_bwd_varlen(q, k, v, dout, cu_seqlens, block_mask, block: int, scale: float):
    """Gradients of `bsattn_fwd_varlen`: each sample's gradients are those of
    its own uniform problem (`bsattn_bwd`). Returns (dQ, dK, dV) [T, H, D]
    float64; tokens outside every sample stay NaN."""
    Q, K, V, dO = _f64(q), _f64(k), _f64(v), _f64(dout)
    m = np.asarray(block_mask)
    out = [np.full(Q.shape, np.nan) for _ in range(3)]
    for b, t0, n, nb in _varlen_samples(cu_seqlens, block):
        if n == 0:
            continue
        sl = slice(t0, t0 + n)
        grads = bsattn_bwd(Q[None, sl], K[None, sl], V[None, sl], dO[None, sl],
                           m[b:b + 1, :, :nb, :nb], block, scale)
        for g, full in zip(grads, out):
            full[sl] = g[0]
    return tuple(out)


# ---------------------------------------------------------------------------
# Top-K block selection (Sec. 3.3, Eq. 6 and Eq. 7)
# ---------------------------------------------------------------------------

def block_pool(x, block: int) -> np.ndarray:
    """pool(.) of Eq. 6: the mean of each block's token rows, per head.

    x [B, N, H, D] -> [B, H, ceil(N / block), D] float64. A short last block is
    averaged over its real tokens (the reading taken for a ragged tail).
    """
    X = _f64(x)
    B, N, H, D = X.shape
    nb = -(-N // block)
    out = np.zeros((B, H, nb, D))
    for b in range(B):
        for h in range(H):
            for j in range(nb):
                rows = _block_tokens(j, block, N)
                out[b, h, j] = X[b, rows, h, :].sum(axis=0) / rows.size
    return out


def topk_block_mask(q, k, block: int, k_keep: int, prefix_blocks: int = 0):
    """Eq. 6-7: per (b, h), S_c = pool(Q) pool(K)^T and M_c[i, j] = 1 for the
    k_keep largest entries of row i of S_c.

    Readings: the paper keeps floor(rho N_k) blocks and the caller passes that
    count as k_keep (k_keep >= N_k keeps every block); equal scores are ranked
    lower j first (the paper does not order ties); no block is forced, the
    diagonal included. A stable sort of the negated row is the selection step.
    prefix_blocks = P > 0 models the always-kept text tokens at the head of
    the joint sequence (512 in the paper's token counts): the first P key
    blocks are kept for every row, the first P query blocks keep every block,
    and the k_keep best blocks are chosen among j >= P.
    Returns (mask uint8 [B, H, Nq, Nk], S_c float64 [B, H, Nq, Nk]).
    """
    PQ, PK = block_pool(q, block), block_pool(k, block)
    B, H, nq, _ = PQ.shape
    nk = PK.shape[2]
    P = min(prefix_blocks, nk)
    Sc = np.zeros((B, H, nq, nk))
    mask = np.zeros((B, H, nq, nk), dtype=np.uint8)
    for b in range(B):
        for h in range(H):
            Sc[b, h] = PQ[b, h] @ PK[b, h].T
            for i in range(nq):
                if i < P:
                    mask[b, h, i, :] = 1
                    continue
                mask[b, h, i, :P] = 1
                order = P + np.argsort(-Sc[b, h, i, P:], kind="stable")
                mask[b, h, i, order[:min(k_keep, nk - P)]] = 1
    return mask, Sc


# ---------------------------------------------------------------------------
# Foreground-restricted sampling and training (Sec. 3.2, Eq. 3 and Eq. 4)
# ---------------------------------------------------------------------------

def euler_update_fg(z, v, kept_idx, dt: float) -> np.ndarray:
    """Eq. 4: z_i <- z_i + (t_prev - t_curr) v_i for every retained position i;
    every other position keeps its value (the initial noise).

    z [L, C] full-grid latent, v [n, C] packed velocities (row k belongs to
    position kept_idx[k]), dt = t_prev - t_curr. Returns the new z in float64.
    """
    Z = _f64(z).copy()
    V = _f64(v)
    for k, i in enumerate(np.asarray(kept_idx).tolist()):
        Z[i, :] = Z[i, :] + dt * V[k, :]
    return Z


def fg_flow_loss(v, eps, z0, kept_idx):
    """Eq. 3: the flow matching loss over the foreground target tokens only,
    || v_hat - Gather_{M_fg}(eps - z_tgt) ||^2, with the target velocity
    eps - z_tgt of Eq. 1-2.

    Reading: the squared norm is averaged over the n retained tokens and the
    C channels (a mean squared error; the paper writes the norm inside an
    expectation and fixes no normalisation). Returns (loss, grad) with
    grad = d loss / d v_hat = 2 (v_hat - target) / (n C), float64.
    """
    V, E, Z = _f64(v), _f64(eps), _f64(z0)
    idx = np.asarray(kept_idx).tolist()
    n, C = V.shape
    target = np.stack([E[i, :] - Z[i, :] for i in idx]) if n else np.zeros((0, C))
    diff = V - target
    loss = float((diff * diff).sum() / (n * C)) if n else 0.0
    grad = 2.0 * diff / (n * C) if n else np.zeros((0, C))
    return loss, grad


# ---------------------------------------------------------------------------
# Composite latent (Sec. 3.4, Eq. 9) and token masks (Sec. 3.2)
# ---------------------------------------------------------------------------

def composite_latent(x_packed, kept_idx, z_bg, L: int) -> np.ndarray:
    """Eq. 9: z_mix_i = z_fg_i at a retained position i (packed row k for
    i = kept_idx[k]) and the canonical background latent elsewhere. z_bg holds
    one view's token grid [P, C]; tile-repeating it over the views gives
    position i the background row i mod P. Returns [L, C] in z_bg's dtype
    (a copy: no arithmetic)."""
    xp, bg = np.asarray(x_packed), np.asarray(z_bg)
    P = bg.shape[0]
    out = np.empty((L,) + bg.shape[1:], dtype=bg.dtype)
    kept = {int(i): k for k, i in enumerate(np.asarray(kept_idx).tolist())}
    for i in range(L):
        out[i] = xp[kept[i]] if i in kept else bg[i % P]
    return out


def token_mask_from_alpha(alpha, patch: int, radius: int, threshold: int = 0) -> np.ndarray:
    """Sec. 3.2: per-view alpha masks brought to the token grid and dilated.

    Readings (the paper names neither rule): a token is foreground when any
    pixel of its patch x patch block has alpha > threshold, and the dilation
    is a (2 radius + 1)^2 square, clipped at the view border.
    alpha [V, H, W] with H, W multiples of patch -> uint8 [V, H/patch, W/patch].
    """
    a = np.asarray(alpha)
    V, Hp, Wp = a.shape
    gh, gw = Hp // patch, Wp // patch
    pooled = np.zeros((V, gh, gw), dtype=bool)
    for v in range(V):
        for y in range(gh):
            for x in range(gw):
                blk = a[v, y * patch:(y + 1) * patch, x * patch:(x + 1) * patch]
                pooled[v, y, x] = bool((blk > threshold).any())
    out = np.zeros((V, gh, gw), dtype=np.uint8)
    for v in range(V):
        for y in range(gh):
            for x in range(gw):
                y0, y1 = max(0, y - radius), min(gh, y + radius + 1)
                x0, x1 = max(0, x - radius), min(gw, x + radius + 1)
                out[v, y, x] = 1 if pooled[v, y0:y1, x0:x1].any() else 0
    return out
