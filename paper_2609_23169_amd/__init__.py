"""Python binding of libultratex.so: UltraTex's foreground hot path on MI355X.

The functions `ut_*` mirror the C ABI in include/ultratex.h one to one: they
take torch tensors, check device, dtype and sizes (a raw pointer cannot carry
its size), pass the pointers and the current HIP stream, and return the
ut_status code. Every step of the path runs in the HIP kernels of the
library; there is no CPU fallback, and importing the package without the
built library raises.

The helpers below the raw calls (`drop_background`, `build_block_index`,
`bsattn_fwd`, ...) allocate the outputs and workspaces with torch and raise
UltraTexError on a non-zero status.
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# UT_LIBRARY selects another build of the same library (the sanitized host
# build of _build.py); by default the in-tree libultratex.so.
LIB_PATH = os.environ.get("UT_LIBRARY") or os.path.join(HERE, "libultratex.so")

UT_OK, UT_ERR_INVALID_ARG, UT_ERR_UNSUPPORTED, UT_ERR_WORKSPACE, UT_ERR_CAPACITY, UT_ERR_HIP = range(6)
UT_BF16, UT_F32 = 0, 1
STATUS_NAMES = ["UT_OK", "UT_ERR_INVALID_ARG", "UT_ERR_UNSUPPORTED", "UT_ERR_WORKSPACE",
                "UT_ERR_CAPACITY", "UT_ERR_HIP"]

# Every symbol the header declares (checked by the CPU test suite).
EXPORTS = [
    "ut_last_error", "ut_abi_version", "ut_trace_enable", "ut_trace_read",
    "ut_drop_background_workspace_size", "ut_drop_background",
    "ut_scatter_foreground", "ut_build_block_index_workspace_size", "ut_build_block_index",
    "ut_bsattn_fwd", "ut_bsattn_bwd_workspace_size", "ut_bsattn_bwd_workspace_size_stored",
    "ut_bsattn_bwd", "ut_bsattn_bwd_noalloc",
    "ut_bsattn_fwd_varlen", "ut_bsattn_bwd_varlen_workspace_size",
    "ut_bsattn_bwd_varlen_workspace_size_stored", "ut_bsattn_bwd_varlen",
    "ut_topk_block_mask_workspace_size", "ut_topk_block_mask",
    "ut_euler_update_foreground", "ut_fg_flow_loss_workspace_size", "ut_fg_flow_loss",
    "ut_composite_latent", "ut_token_mask_workspace_size", "ut_token_mask_from_alpha",
]


class UltraTexError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} -> {STATUS_NAMES[status] if 0 <= status < 6 else status}: {msg}")
        self.status = status


class KernelTime(ctypes.Structure):
    """ut_kernel_time of the C ABI."""
    _fields_ = [("name", ctypes.c_char * 48), ("count", ctypes.c_int64), ("total_ms", ctypes.c_double),
                ("min_ms", ctypes.c_double), ("max_ms", ctypes.c_double)]


_c = ctypes
_vp, _i32, _i64, _f32, _sz = _c.c_void_p, _c.c_int32, _c.c_int64, _c.c_float, _c.c_size_t
_SIGS = {
    "ut_last_error": (_c.c_char_p, []),
    "ut_abi_version": (_c.c_int, []),
    "ut_trace_enable": (_c.c_int, [_c.c_int]),
    "ut_trace_read": (_c.c_int, [_c.POINTER(KernelTime), _c.c_int]),
    "ut_drop_background_workspace_size": (_sz, [_i64]),
    "ut_drop_background": (_c.c_int, [_vp, _i64, _vp, _i64, _vp, _i64, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "ut_scatter_foreground": (_c.c_int, [_vp, _vp, _i64, _i64, _vp, _vp]),
    "ut_build_block_index_workspace_size": (_sz, [_i32, _i32, _i32, _i32]),
    "ut_build_block_index": (_c.c_int, [_vp, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _i64, _vp, _vp, _sz,
                                        _vp]),
    "ut_bsattn_fwd": (_c.c_int, [_vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _f32, _vp]),
    "ut_bsattn_bwd_workspace_size": (_sz, [_i32, _i32, _i32]),
    "ut_bsattn_bwd_workspace_size_stored": (_sz, [_i32, _i32, _i32, _i32, _i64]),
    "ut_bsattn_bwd": (_c.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32,
                                 _vp, _vp, _vp, _vp, _f32, _vp, _sz, _vp]),
    "ut_bsattn_bwd_noalloc": (_c.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32,
                                         _i32, _vp, _vp, _vp, _vp, _f32, _vp]),
    "ut_bsattn_fwd_varlen": (_c.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _i32, _i64, _i32, _i32, _i32, _i32,
                                        _vp, _vp, _f32, _vp]),
    "ut_bsattn_bwd_varlen_workspace_size": (_sz, [_i64, _i32]),
    "ut_bsattn_bwd_varlen_workspace_size_stored": (_sz, [_i32, _i64, _i32, _i32, _i32, _i64]),
    "ut_bsattn_bwd_varlen": (_c.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i64, _i32,
                                        _i32, _i32, _i32, _vp, _vp, _vp, _vp, _f32, _vp, _sz, _vp]),
    "ut_topk_block_mask_workspace_size": (_sz, [_i32, _i32, _i32, _i32, _i32]),
    "ut_topk_block_mask": (_c.c_int, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _sz,
                                      _vp]),
    "ut_euler_update_foreground": (_c.c_int, [_vp, _i64, _i64, _vp, _c.c_int, _vp, _i64, _f32, _vp]),
    "ut_fg_flow_loss_workspace_size": (_sz, []),
    "ut_composite_latent": (_c.c_int, [_vp, _i64, _vp, _i64, _vp, _i64, _i64, _vp, _vp]),
    "ut_token_mask_workspace_size": (_sz, [_i32, _i32, _i32, _i32]),
    "ut_token_mask_from_alpha": (_c.c_int, [_vp, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _sz, _vp]),
    "ut_fg_flow_loss": (_c.c_int, [_vp, _c.c_int, _vp, _vp, _c.c_int, _i64, _i64, _vp, _i64, _vp, _vp,
                                   _vp, _sz, _vp]),
}

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -c "
                               f"'import __graft_entry__ as g; g.build()'`")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(l, name)
            f.restype, f.argtypes = res, args
        _lib = l
    return _lib


def last_error() -> str:
    return lib().ut_last_error().decode()


def ut_trace_enable(on: bool) -> int:
    return lib().ut_trace_enable(1 if on else 0)


def trace_read() -> list:
    """Per-kernel launch timings recorded since the last read (waits for
    them): [{"name", "count", "total_ms", "min_ms", "max_ms"}, ...]."""
    cap = 128   # the library launches fewer distinct kernels than this
    buf = (KernelTime * cap)()
    n = lib().ut_trace_read(buf, cap)
    if n < 0:
        raise UltraTexError("ut_trace_read", UT_ERR_HIP, last_error())
    return [{"name": k.name.decode(), "count": int(k.count), "total_ms": k.total_ms,
             "min_ms": k.min_ms, "max_ms": k.max_ms} for k in buf[:min(n, cap)]]


def _p(t):
    """Pointer of a device tensor (None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch.Tensor")
    if not t.is_cuda:
        raise ValueError("tensor must live in GPU memory")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _need(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


# ---------------------------------------------------------------------------
# Raw calls: same names and argument order as the C ABI, tensors for pointers.
# ---------------------------------------------------------------------------

def ut_drop_background_workspace_size(L: int) -> int:
    return int(lib().ut_drop_background_workspace_size(L))


def ut_drop_background(fg_mask, x_full, x_packed, kept_idx, inv_idx, n_kept, workspace,
                       n_kept_host: bool = False, stream=None):
    """Returns (status, n_kept or None)."""
    L = fg_mask.numel()
    _need(fg_mask.dtype == torch.uint8, "fg_mask must be uint8")
    capacity = kept_idx.numel()
    _need(kept_idx.dtype == torch.int32 and n_kept.dtype == torch.int32 and n_kept.numel() >= 1,
          "kept_idx and n_kept must be int32")
    row_bytes = 0
    if x_full is not None:
        _need(x_packed is not None, "x_packed needed with x_full")
        _need(x_full.dim() >= 1 and x_full.shape[0] == L, "x_full must have L rows")
        row_bytes = _nbytes(x_full) // L
        _need(x_packed.shape[0] >= capacity and _nbytes(x_packed) >= capacity * row_bytes
              and x_packed.dtype == x_full.dtype, "x_packed must hold capacity rows")
    if inv_idx is not None:
        _need(inv_idx.dtype == torch.int32 and inv_idx.numel() >= L, "inv_idx must be int32 [L]")
    host = ctypes.c_int64(-1)
    ws_bytes = _nbytes(workspace) if workspace is not None else 0
    st = lib().ut_drop_background(_p(fg_mask), L, _p(x_full), row_bytes, _p(x_packed), capacity,
                                  _p(kept_idx), _p(inv_idx), _p(n_kept),
                                  ctypes.byref(host) if n_kept_host else None,
                                  _p(workspace), ws_bytes, _stream(stream))
    return st, (host.value if n_kept_host else None)


def ut_scatter_foreground(x_packed, kept_idx, n_kept: int, x_full, stream=None) -> int:
    L = x_full.shape[0]
    row_bytes = _nbytes(x_full) // max(L, 1)
    _need(kept_idx.dtype == torch.int32 and kept_idx.numel() >= n_kept, "kept_idx int32 [n_kept]")
    _need(x_packed.dtype == x_full.dtype and _nbytes(x_packed) >= n_kept * row_bytes,
          "x_packed must hold n_kept rows of x_full's width")
    return lib().ut_scatter_foreground(_p(x_packed), _p(kept_idx), n_kept, row_bytes, _p(x_full),
                                       _stream(stream))


def ut_build_block_index_workspace_size(B: int, H: int, Nq: int, Nk: int) -> int:
    return int(lib().ut_build_block_index_workspace_size(B, H, Nq, Nk))


def ut_build_block_index(block_mask, q_rowptr, q_cols, kv_colptr, kv_rows, nnz_host: bool = False,
                         workspace=None, stream=None):
    """Returns (status, nnz or None). The build needs no scratch (its size
    query returns 0), so `workspace` may stay None."""
    _need(block_mask.dtype == torch.uint8 and block_mask.dim() == 4, "block_mask uint8 [B,H,Nq,Nk]")
    B, H, Nq, Nk = block_mask.shape
    _need(q_rowptr.numel() >= B * H * Nq + 1 and kv_colptr.numel() >= B * H * Nk + 1,
          "row/column pointer arrays too short")
    cap = min(q_cols.numel(), kv_rows.numel())
    for t in (q_rowptr, q_cols, kv_colptr, kv_rows):
        _need(t.dtype == torch.int32, "index arrays must be int32")
    host = ctypes.c_int64(-1)
    ws_bytes = _nbytes(workspace) if workspace is not None else 0
    st = lib().ut_build_block_index(_p(block_mask), B, H, Nq, Nk, _p(q_rowptr), _p(q_cols),
                                    _p(kv_colptr), _p(kv_rows), cap,
                                    ctypes.byref(host) if nnz_host else None, _p(workspace),
                                    ws_bytes, _stream(stream))
    return st, (host.value if nnz_host else None)


def _attn_shape(q, block):
    _need(q.dim() == 4, "q/k/v must be [B, N, H, D]")
    B, N, H, D = q.shape
    return B, N, H, D, -(-N // block)


def _check_attn(q, k, v, block, rowptr, cols):
    B, N, H, D, nb = _attn_shape(q, block)
    for t in (q, k, v):
        _need(t.shape == q.shape and t.dtype == torch.bfloat16, "q, k, v: bf16 [B,N,H,D], same shape")
    _need(rowptr.dtype == torch.int32 and rowptr.numel() >= B * H * nb + 1, "rowptr int32 [B*H*Nq+1]")
    _need(cols.dtype == torch.int32, "cols int32")
    return B, N, H, D, nb


def ut_bsattn_fwd(q, k, v, o, lse, block: int, q_rowptr, q_cols, softmax_scale: float,
                  stream=None) -> int:
    B, N, H, D, nb = _check_attn(q, k, v, block, q_rowptr, q_cols)
    _need(o.shape == q.shape and o.dtype == torch.bfloat16, "o: bf16 [B,N,H,D]")
    _need(lse.dtype == torch.float32 and lse.numel() >= B * H * N, "lse: fp32 [B,H,N]")
    return lib().ut_bsattn_fwd(_p(q), _p(k), _p(v), _p(o), _p(lse), B, N, H, D, block,
                               _p(q_rowptr), _p(q_cols), softmax_scale, _stream(stream))


def ut_bsattn_bwd_workspace_size(B: int, N: int, H: int) -> int:
    return int(lib().ut_bsattn_bwd_workspace_size(B, N, H))


def ut_bsattn_bwd_workspace_size_stored(B: int, N: int, H: int, block: int, nnz: int) -> int:
    """Workspace bytes with room for the bf16 dS tiles of nnz retained pairs:
    with it, dQ of every query block comes from the tiles the dK/dV pass
    stores instead of a recompute of S and dP."""
    return int(lib().ut_bsattn_bwd_workspace_size_stored(B, N, H, block, nnz))


def ut_bsattn_bwd(q, k, v, o, dout, lse, dq, dk, dv, block: int, q_rowptr, q_cols, kv_colptr,
                  kv_rows, softmax_scale: float, workspace, stream=None) -> int:
    B, N, H, D, nb = _check_attn(q, k, v, block, q_rowptr, q_cols)
    for t in (o, dout, dq, dk, dv):
        _need(t.shape == q.shape and t.dtype == torch.bfloat16, "o, dout, dq, dk, dv: bf16 [B,N,H,D]")
    _need(lse.dtype == torch.float32 and lse.numel() >= B * H * N, "lse: fp32 [B,H,N]")
    _need(kv_colptr.dtype == torch.int32 and kv_colptr.numel() >= B * H * nb + 1, "kv_colptr int32")
    _need(kv_rows.dtype == torch.int32, "kv_rows int32")
    ws_bytes = _nbytes(workspace) if workspace is not None else 0
    return lib().ut_bsattn_bwd(_p(q), _p(k), _p(v), _p(o), _p(dout), _p(lse), _p(dq), _p(dk), _p(dv),
                               B, N, H, D, block, _p(q_rowptr), _p(q_cols), _p(kv_colptr),
                               _p(kv_rows), softmax_scale, _p(workspace), ws_bytes, _stream(stream))


def ut_bsattn_bwd_noalloc(q, k, v, o, dout, lse, dq, dk, dv, block: int, q_rowptr, q_cols, kv_colptr,
                          kv_rows, softmax_scale: float, stream=None) -> int:
    """ut_bsattn_bwd with the library's built-in scratch instead of a workspace
    (no device allocation; B*H*N up to 4,194,304 query rows)."""
    B, N, H, D, nb = _check_attn(q, k, v, block, q_rowptr, q_cols)
    for t in (o, dout, dq, dk, dv):
        _need(t.shape == q.shape and t.dtype == torch.bfloat16, "o, dout, dq, dk, dv: bf16 [B,N,H,D]")
    _need(lse.dtype == torch.float32 and lse.numel() >= B * H * N, "lse: fp32 [B,H,N]")
    _need(kv_colptr.dtype == torch.int32 and kv_colptr.numel() >= B * H * nb + 1, "kv_colptr int32")
    _need(kv_rows.dtype == torch.int32, "kv_rows int32")
    return lib().ut_bsattn_bwd_noalloc(_p(q), _p(k), _p(v), _p(o), _p(dout), _p(lse), _p(dq), _p(dk),
                                       _p(dv), B, N, H, D, block, _p(q_rowptr), _p(q_cols),
                                       _p(kv_colptr), _p(kv_rows), softmax_scale, _stream(stream))


def _check_varlen(q, k, v, cu_seqlens, max_seqlen, block, rowptr, cols):
    _need(q.dim() == 3, "q: bf16 [T, H, D] (packed samples)")
    T, H, D = q.shape
    for t in (q, k, v):
        _need(t.shape == q.shape and t.dtype == torch.bfloat16, "q, k, v: bf16 [T,H,D], same shape")
    _need(cu_seqlens.dtype == torch.int32 and cu_seqlens.dim() == 1 and cu_seqlens.numel() >= 2,
          "cu_seqlens: int32 [B+1]")
    B = cu_seqlens.numel() - 1
    _need(block > 0 and max_seqlen > 0, "block and max_seqlen must be positive")
    nb = -(-max_seqlen // block)
    _need(rowptr.dtype == torch.int32 and rowptr.numel() >= B * H * nb + 1, "rowptr int32 [B*H*Nb+1]")
    _need(cols.dtype == torch.int32, "cols int32")
    return B, T, H, D, nb


def ut_bsattn_fwd_varlen(q, k, v, o, lse, cu_seqlens, max_seqlen: int, block: int, q_rowptr, q_cols,
                         softmax_scale: float, stream=None) -> int:
    B, T, H, D, nb = _check_varlen(q, k, v, cu_seqlens, max_seqlen, block, q_rowptr, q_cols)
    _need(o.shape == q.shape and o.dtype == torch.bfloat16, "o: bf16 [T,H,D]")
    _need(lse.dtype == torch.float32 and lse.numel() >= H * T, "lse: fp32 [H,T]")
    return lib().ut_bsattn_fwd_varlen(_p(q), _p(k), _p(v), _p(o), _p(lse), _p(cu_seqlens), B, T,
                                      max_seqlen, H, D, block, _p(q_rowptr), _p(q_cols), softmax_scale,
                                      _stream(stream))


def ut_bsattn_bwd_varlen_workspace_size(T: int, H: int) -> int:
    return int(lib().ut_bsattn_bwd_varlen_workspace_size(T, H))


def ut_bsattn_bwd_varlen_workspace_size_stored(B: int, T: int, max_seqlen: int, H: int, block: int,
                                               nnz: int) -> int:
    return int(lib().ut_bsattn_bwd_varlen_workspace_size_stored(B, T, max_seqlen, H, block, nnz))


def ut_bsattn_bwd_varlen(q, k, v, o, dout, lse, dq, dk, dv, cu_seqlens, max_seqlen: int, block: int,
                         q_rowptr, q_cols, kv_colptr, kv_rows, softmax_scale: float, workspace,
                         stream=None) -> int:
    B, T, H, D, nb = _check_varlen(q, k, v, cu_seqlens, max_seqlen, block, q_rowptr, q_cols)
    for t in (o, dout, dq, dk, dv):
        _need(t.shape == q.shape and t.dtype == torch.bfloat16, "o, dout, dq, dk, dv: bf16 [T,H,D]")
    _need(lse.dtype == torch.float32 and lse.numel() >= H * T, "lse: fp32 [H,T]")
    _need(kv_colptr.dtype == torch.int32 and kv_colptr.numel() >= B * H * nb + 1, "kv_colptr int32")
    _need(kv_rows.dtype == torch.int32, "kv_rows int32")
    ws_bytes = _nbytes(workspace) if workspace is not None else 0
    return lib().ut_bsattn_bwd_varlen(_p(q), _p(k), _p(v), _p(o), _p(dout), _p(lse), _p(dq), _p(dk),
                                      _p(dv), _p(cu_seqlens), B, T, max_seqlen, H, D, block,
                                      _p(q_rowptr), _p(q_cols), _p(kv_colptr), _p(kv_rows),
                                      softmax_scale, _p(workspace), ws_bytes, _stream(stream))


def ut_topk_block_mask_workspace_size(B: int, N: int, H: int, D: int, block: int) -> int:
    return int(lib().ut_topk_block_mask_workspace_size(B, N, H, D, block))


def ut_topk_block_mask(q, k, block: int, k_keep: int, block_mask, workspace, prefix_blocks: int = 0,
                       stream=None) -> int:
    _need(q.dim() == 4 and k.shape == q.shape, "q, k: [B, N, H, D], same shape")
    _need(q.dtype == torch.bfloat16 and k.dtype == torch.bfloat16, "q, k: bf16")
    B, N, H, D = q.shape
    nb = -(-N // block)
    _need(block_mask.dtype == torch.uint8 and block_mask.numel() >= B * H * nb * nb,
          "block_mask: uint8 [B, H, Nk, Nk]")
    ws_bytes = _nbytes(workspace) if workspace is not None else 0
    return lib().ut_topk_block_mask(_p(q), _p(k), B, N, H, D, block, k_keep, prefix_blocks,
                                    _p(block_mask), _p(workspace), ws_bytes, _stream(stream))


def _dtype_code(t) -> int:
    if t.dtype == torch.bfloat16:
        return UT_BF16
    _need(t.dtype == torch.float32, "tensors must be bf16 or fp32")
    return UT_F32


def ut_euler_update_foreground(z, v, kept_idx, n_kept: int, dt: float, stream=None) -> int:
    _need(z.dtype == torch.float32 and z.dim() == 2, "z: fp32 [L, C]")
    L, C = z.shape
    _need(v.dim() == 2 and v.shape[1] == C and v.shape[0] >= n_kept, "v: [n_kept, C]")
    _need(kept_idx.dtype == torch.int32 and kept_idx.numel() >= n_kept, "kept_idx: int32 [n_kept]")
    return lib().ut_euler_update_foreground(_p(z), L, C, _p(v), _dtype_code(v), _p(kept_idx),
                                            n_kept, dt, _stream(stream))


def ut_fg_flow_loss_workspace_size() -> int:
    return int(lib().ut_fg_flow_loss_workspace_size())


def ut_fg_flow_loss(v, eps, z0, kept_idx, n_kept: int, loss, grad, workspace, stream=None) -> int:
    _need(eps.dim() == 2 and z0.shape == eps.shape and z0.dtype == eps.dtype, "eps, z0: [L, C], same dtype")
    L, C = eps.shape
    _need(v.dim() == 2 and v.shape[1] == C and v.shape[0] >= n_kept, "v: [n_kept, C]")
    _need(kept_idx.dtype == torch.int32 and kept_idx.numel() >= n_kept, "kept_idx: int32 [n_kept]")
    _need(loss.dtype == torch.float32 and loss.numel() >= 1, "loss: fp32 [1]")
    if grad is not None:
        _need(grad.dtype == torch.float32 and grad.numel() >= n_kept * C, "grad: fp32 [n_kept, C]")
    ws_bytes = _nbytes(workspace) if workspace is not None else 0
    return lib().ut_fg_flow_loss(_p(v), _dtype_code(v), _p(eps), _p(z0), _dtype_code(eps), L, C,
                                 _p(kept_idx), n_kept, _p(loss), _p(grad) if grad is not None else None,
                                 _p(workspace), ws_bytes, _stream(stream))


def ut_composite_latent(x_packed, n_kept: int, inv_idx, z_bg, z_mix, stream=None) -> int:
    _need(z_mix.dim() >= 1 and inv_idx.dtype == torch.int32 and inv_idx.numel() == z_mix.shape[0],
          "inv_idx: int32 [L], z_mix: [L, ...]")
    L = z_mix.shape[0]
    row_bytes = _nbytes(z_mix) // L
    _need(z_bg.dtype == z_mix.dtype and _nbytes(z_bg) % row_bytes == 0, "z_bg: [P, ...] rows like z_mix")
    _need(x_packed.dtype == z_mix.dtype and _nbytes(x_packed) >= n_kept * row_bytes, "x_packed rows")
    return lib().ut_composite_latent(_p(x_packed) if n_kept else None, n_kept, _p(inv_idx), L, _p(z_bg),
                                     _nbytes(z_bg) // row_bytes, row_bytes, _p(z_mix), _stream(stream))


def ut_token_mask_workspace_size(V: int, Hp: int, Wp: int, patch: int) -> int:
    return int(lib().ut_token_mask_workspace_size(V, Hp, Wp, patch))


def ut_token_mask_from_alpha(alpha, patch: int, threshold: int, radius: int, token_mask, workspace,
                             stream=None) -> int:
    _need(alpha.dtype == torch.uint8 and alpha.dim() == 3, "alpha: uint8 [V, Hp, Wp]")
    V, Hp, Wp = alpha.shape
    _need(token_mask.dtype == torch.uint8 and token_mask.numel() >= V * (Hp // patch) * (Wp // patch),
          "token_mask: uint8 [V, Hp/patch, Wp/patch]")
    ws_bytes = _nbytes(workspace) if workspace is not None else 0
    return lib().ut_token_mask_from_alpha(_p(alpha), V, Hp, Wp, patch, threshold, radius, _p(token_mask),
                                          _p(workspace), ws_bytes, _stream(stream))


# ---------------------------------------------------------------------------
# Allocating helpers (raise on error)
# ---------------------------------------------------------------------------

def _raise(fn: str, st: int):
    if st != UT_OK:
        raise UltraTexError(fn, st, last_error())


def drop_background(fg_mask, x_full=None, capacity=None, with_inv=True, stream=None):
    """Compaction (+ gather when x_full is given). Synchronises once to learn
    n_kept. Returns dict(kept_idx, inv_idx, n_kept, x_packed)."""
    dev = fg_mask.device
    L = fg_mask.numel()
    cap = L if capacity is None else capacity
    kept = torch.empty(cap, dtype=torch.int32, device=dev)
    inv = torch.empty(L, dtype=torch.int32, device=dev) if with_inv else None
    n_dev = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(max(ut_drop_background_workspace_size(L), 4), dtype=torch.uint8, device=dev)
    packed = None
    if x_full is not None:
        packed = torch.empty((cap,) + tuple(x_full.shape[1:]), dtype=x_full.dtype, device=dev)
    st, n = ut_drop_background(fg_mask, x_full, packed, kept, inv, n_dev, ws, n_kept_host=True,
                               stream=stream)
    _raise("ut_drop_background", st)
    return {"kept_idx": kept[:n], "inv_idx": inv, "n_kept": n,
            "x_packed": packed[:n] if packed is not None else None}


def scatter_foreground(x_packed, kept_idx, x_full, stream=None):
    """In place: x_full[kept_idx[k]] = x_packed[k]."""
    _raise("ut_scatter_foreground",
           ut_scatter_foreground(x_packed, kept_idx, kept_idx.numel(), x_full, stream))
    return x_full


def build_block_index(block_mask, stream=None):
    """Row and column lists of a block mask. Synchronises once to learn nnz."""
    B, H, Nq, Nk = block_mask.shape
    dev = block_mask.device
    cap = int(B * H * Nq * Nk)
    rowptr = torch.empty(B * H * Nq + 1, dtype=torch.int32, device=dev)
    colptr = torch.empty(B * H * Nk + 1, dtype=torch.int32, device=dev)
    cols = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    rows = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    st, nnz = ut_build_block_index(block_mask, rowptr, cols, colptr, rows, nnz_host=True,
                                   stream=stream)
    _raise("ut_build_block_index", st)
    return {"q_rowptr": rowptr, "q_cols": cols[:max(nnz, 1)], "kv_colptr": colptr,
            "kv_rows": rows[:max(nnz, 1)], "nnz": nnz}


def bsattn_fwd(q, k, v, index, block: int, softmax_scale: float, stream=None):
    B, N, H, D = q.shape
    o = torch.empty_like(q)
    lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    _raise("ut_bsattn_fwd", ut_bsattn_fwd(q, k, v, o, lse, block, index["q_rowptr"],
                                          index["q_cols"], softmax_scale, stream))
    return o, lse


def _ds_pairs(index, ds_pairs, block: int, base: int, device) -> int:
    """dS tiles to make room for: all retained pairs by default, unless that
    would take more than half of the device memory still free."""
    if ds_pairs is None:
        ds_pairs = int(index.get("nnz", 0))
        free, _ = torch.cuda.mem_get_info(device)
        if base + ds_pairs * 2 * block * block > free // 2:
            ds_pairs = 0
    return max(int(ds_pairs), 0)


def bsattn_bwd(q, k, v, o, dout, lse, index, block: int, softmax_scale: float, workspace=None,
               stream=None, ds_pairs=None):
    """Gradients of bsattn_fwd. Without a workspace, one is allocated with
    room for the dS tiles of `ds_pairs` pairs (default: every pair of the
    index, if that fits in half the free device memory; 0: recompute dQ)."""
    B, N, H, D = q.shape
    dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
    if workspace is None:
        base = ut_bsattn_bwd_workspace_size(B, N, H)
        n = _ds_pairs(index, ds_pairs, block, base, q.device)
        size = ut_bsattn_bwd_workspace_size_stored(B, N, H, block, n) if n else base
        workspace = torch.empty(size, dtype=torch.uint8, device=q.device)
    _raise("ut_bsattn_bwd", ut_bsattn_bwd(q, k, v, o, dout, lse, dq, dk, dv, block,
                                          index["q_rowptr"], index["q_cols"], index["kv_colptr"],
                                          index["kv_rows"], softmax_scale, workspace, stream))
    return dq, dk, dv


def bsattn_fwd_varlen(q, k, v, cu_seqlens, max_seqlen: int, index, block: int, softmax_scale: float,
                      stream=None):
    """Packed samples q, k, v [T, H, D]; index over a [B, H, Nb, Nb] block
    mask, Nb = ceil(max_seqlen / block). Returns (o [T, H, D], lse [H, T])."""
    T, H, D = q.shape
    o = torch.zeros_like(q)
    lse = torch.empty((H, T), dtype=torch.float32, device=q.device)
    _raise("ut_bsattn_fwd_varlen",
           ut_bsattn_fwd_varlen(q, k, v, o, lse, cu_seqlens, max_seqlen, block, index["q_rowptr"],
                                index["q_cols"], softmax_scale, stream))
    return o, lse


def bsattn_bwd_varlen(q, k, v, o, dout, lse, cu_seqlens, max_seqlen: int, index, block: int,
                      softmax_scale: float, workspace=None, stream=None, ds_pairs=None):
    T, H, D = q.shape
    dq, dk, dv = torch.zeros_like(q), torch.zeros_like(q), torch.zeros_like(q)
    if workspace is None:
        base = max(ut_bsattn_bwd_varlen_workspace_size(T, H), 16)
        n = _ds_pairs(index, ds_pairs, block, base, q.device) if T > 0 else 0
        B = cu_seqlens.numel() - 1
        size = (ut_bsattn_bwd_varlen_workspace_size_stored(B, T, max_seqlen, H, block, n) if n
                else base)
        workspace = torch.empty(size, dtype=torch.uint8, device=q.device)
    _raise("ut_bsattn_bwd_varlen",
           ut_bsattn_bwd_varlen(q, k, v, o, dout, lse, dq, dk, dv, cu_seqlens, max_seqlen, block,
                                index["q_rowptr"], index["q_cols"], index["kv_colptr"], index["kv_rows"],
                                softmax_scale, workspace, stream))
    return dq, dk, dv


def topk_block_mask(q, k, block: int, k_keep: int, prefix_blocks: int = 0, workspace=None, stream=None):
    """Block mask [B, H, Nk, Nk] uint8 of the k_keep best key blocks per query
    block (plus the dense leading prefix blocks, if any)."""
    B, N, H, D = q.shape
    nb = -(-N // block)
    mask = torch.empty((B, H, nb, nb), dtype=torch.uint8, device=q.device)
    if workspace is None:
        workspace = torch.empty(max(ut_topk_block_mask_workspace_size(B, N, H, D, block), 16),
                                dtype=torch.uint8, device=q.device)
    _raise("ut_topk_block_mask", ut_topk_block_mask(q, k, block, k_keep, mask, workspace, prefix_blocks,
                                                    stream))
    return mask


def euler_update_foreground(z, v, kept_idx, dt: float, stream=None):
    """In place: z[kept_idx[k]] += dt * v[k] (Eq. 4). Returns z."""
    _raise("ut_euler_update_foreground",
           ut_euler_update_foreground(z, v, kept_idx, kept_idx.numel(), dt, stream))
    return z


def fg_flow_loss(v, eps, z0, kept_idx, with_grad: bool = True, workspace=None, stream=None):
    """(loss [1] fp32, grad [n, C] fp32 or None) of Eq. 3 on the device."""
    n, C = kept_idx.numel(), eps.shape[1]
    loss = torch.empty(1, dtype=torch.float32, device=eps.device)
    grad = torch.empty((n, C), dtype=torch.float32, device=eps.device) if with_grad else None
    if workspace is None:
        workspace = torch.empty(ut_fg_flow_loss_workspace_size(), dtype=torch.uint8, device=eps.device)
    _raise("ut_fg_flow_loss", ut_fg_flow_loss(v, eps, z0, kept_idx, n, loss, grad, workspace, stream))
    return loss, grad


def composite_latent(x_packed, inv_idx, z_bg, n_kept: int, stream=None):
    """z_mix [L, ...] of Eq. 9 (packed rows where kept, tiled z_bg elsewhere)."""
    L = inv_idx.numel()
    z_mix = torch.empty((L,) + tuple(z_bg.shape[1:]), dtype=z_bg.dtype, device=z_bg.device)
    _raise("ut_composite_latent", ut_composite_latent(x_packed, n_kept, inv_idx, z_bg, z_mix, stream))
    return z_mix


def token_mask_from_alpha(alpha, patch: int = 16, threshold: int = 0, radius: int = 1, stream=None):
    """uint8 [V, Hp/patch, Wp/patch] token-grid foreground masks."""
    V, Hp, Wp = alpha.shape
    out = torch.empty((V, Hp // patch, Wp // patch), dtype=torch.uint8, device=alpha.device)
    ws = torch.empty(max(ut_token_mask_workspace_size(V, Hp, Wp, patch), 1), dtype=torch.uint8,
                     device=alpha.device)
    _raise("ut_token_mask_from_alpha", ut_token_mask_from_alpha(alpha, patch, threshold, radius, out, ws,
                                                                stream))
    return out
