// Host side of the C ABI declared in include/ultratex.h: argument validation,
// workspace sizing, status codes and the per-thread error message. Every
// check runs before any launch; no exception leaves this file.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "common.h"

namespace ut {
namespace {
thread_local char g_last_error[512] = "";

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
}  // namespace

ut_status fail(ut_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

ut_status check_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return UT_OK;
  return fail(UT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// ptr[0] = 0, ptr non-decreasing, ptr[rows] = the number of entries given, and
// each row's entries strictly ascending in [0, limit).
ut_status check_lists(const char* fn, const char* what, const int32_t* ptr, const int32_t* idx,
                      int64_t n_idx, int64_t rows, int32_t limit) {
  if (ptr[0] != 0)
    return fail(UT_ERR_INVALID_ARG, "%s: %s: pointers start at %d, not 0", fn, what, ptr[0]);
  for (int64_t r = 0; r < rows; ++r)
    if (ptr[r + 1] < ptr[r])
      return fail(UT_ERR_INVALID_ARG, "%s: %s: pointers decrease at row %lld", fn, what,
                  (long long)r);
  if (!idx) return UT_OK;   // pointers only
  if (ptr[rows] != n_idx)
    return fail(UT_ERR_INVALID_ARG, "%s: %s: pointers end at %d, not at the %lld entries", fn,
                what, ptr[rows], (long long)n_idx);
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t e = ptr[r]; e < ptr[r + 1]; ++e) {
      if (idx[e] < 0 || idx[e] >= limit)
        return fail(UT_ERR_INVALID_ARG, "%s: %s: row %lld holds %d, outside [0, %d)", fn, what,
                    (long long)r, idx[e], limit);
      if (e > ptr[r] && idx[e] <= idx[e - 1])
        return fail(UT_ERR_INVALID_ARG, "%s: %s: row %lld is not strictly ascending", fn, what,
                    (long long)r);
    }
  return UT_OK;
}

ut_status check_cu_seqlens(const char* fn, const int32_t* cu, int32_t B, int64_t T,
                           int32_t max_seqlen) {
  if (cu[0] != 0 || cu[B] != T)
    return fail(UT_ERR_INVALID_ARG, "%s: cu_seqlens must run from 0 to T = %lld (got %d .. %d)",
                fn, (long long)T, cu[0], cu[B]);
  for (int32_t b = 0; b < B; ++b) {
    if (cu[b + 1] < cu[b])
      return fail(UT_ERR_INVALID_ARG, "%s: cu_seqlens decreases at sample %d", fn, b);
    if (cu[b + 1] - cu[b] > max_seqlen)
      return fail(UT_ERR_INVALID_ARG, "%s: sample %d has %d tokens > max_seqlen %d", fn, b,
                  cu[b + 1] - cu[b], max_seqlen);
  }
  return UT_OK;
}

namespace {

ut_status check_attn_common(const char* fn, int32_t B, int32_t N, int32_t H, int32_t D,
                            int32_t block, float scale) {
  if (B < 1 || N < 1 || H < 1)
    return fail(UT_ERR_INVALID_ARG, "%s: B, N, H must be >= 1 (got %d, %d, %d)", fn, B, N, H);
  if (D != 64 && D != 128)
    return fail(UT_ERR_UNSUPPORTED, "%s: head_dim %d unsupported (64 or 128)", fn, D);
  if (block != 64 && block != 128)
    return fail(UT_ERR_UNSUPPORTED, "%s: block %d unsupported (64 or 128)", fn, block);
  // the kernels keep a running maximum of the scaled scores and mask keys with
  // -inf scores; both need a positive scale
  if (!std::isfinite(scale) || !(scale > 0.f))
    return fail(UT_ERR_INVALID_ARG, "%s: softmax_scale must be finite and > 0 (got %g)", fn,
                (double)scale);
  const int64_t nblk = (N + block - 1) / block;
  if ((int64_t)B * H * nblk >= (int64_t)1 << 31 || (int64_t)B * N * H * D >= (int64_t)1 << 40)
    return fail(UT_ERR_INVALID_ARG, "%s: problem too large", fn);
  // the kernels bound their tile loads with 32-bit buffer ranges over one
  // sample's rows
  if ((int64_t)N * H * D * 2 >= (int64_t)1 << 31)
    return fail(UT_ERR_UNSUPPORTED, "%s: one sample's Q/K/V of %d x %d x %d bf16 reach 2 GiB", fn,
                N, H, D);
  return UT_OK;
}

ut_status check_ptr(const char* fn, const char* name, const void* p, uintptr_t align) {
  if (!p) return fail(UT_ERR_INVALID_ARG, "%s: %s is NULL", fn, name);
  if (!aligned(p, align))
    return fail(UT_ERR_INVALID_ARG, "%s: %s must be %zu-byte aligned", fn, name, (size_t)align);
  return UT_OK;
}

#define UT_TRY(x)                     \
  do {                                \
    ut_status _s = (x);               \
    if (_s != UT_OK) return _s;       \
  } while (0)

// ---- backward workspace: statistics planes, then the stored dS tiles ----
// Layout past the statistics (each part 256-byte aligned): a flag per query
// block row, the row-list entry -> tile map, then the tiles of 2 block^2 bytes.
constexpr size_t kDsAlign = 256;
size_t align_up(size_t x) { return (x + kDsAlign - 1) / kDsAlign * kDsAlign; }
size_t tiles_bytes(int64_t m, int32_t block) {
  return align_up((size_t)m * 4) + (size_t)m * 2 * block * block;
}

// Size with room for the dS tiles of nnz pairs (0 for invalid arguments).
size_t stored_size(size_t stats_bytes, int64_t rows, int32_t block, int64_t nnz) {
  if (stats_bytes == 0 || rows < 1 || (block != 64 && block != 128) || nnz < 0 ||
      nnz > ((int64_t)1 << 31) - 1)
    return 0;
  return align_up(stats_bytes) + align_up((size_t)rows * 4) + tiles_bytes(nnz, block);
}

// The tiles a workspace of `bytes` holds past the statistics (none: recompute dQ).
DsTiles ds_region(void* workspace, size_t bytes, size_t stats_bytes, int64_t rows, int32_t block) {
  DsTiles r;
  const size_t off = align_up(stats_bytes), flags = align_up((size_t)rows * 4);
  if (!workspace || bytes <= off + flags) return r;
  const size_t rem = bytes - off - flags;
  int64_t m = std::min<int64_t>((int64_t)(rem / ((size_t)2 * block * block + 4)),
                                ((int64_t)1 << 31) - 1);
  while (m > 0 && tiles_bytes(m, block) > rem) --m;
  if (m <= 0) return r;
  char* base = static_cast<char*>(workspace) + off;
  r.row_ok = reinterpret_cast<int32_t*>(base);
  r.map = reinterpret_cast<int32_t*>(base + flags);
  r.tiles = base + flags + align_up((size_t)m * 4);
  r.max_pairs = m;
  return r;
}
}  // namespace
}  // namespace ut

using namespace ut;

extern "C" {

const char* ut_last_error(void) { return g_last_error; }

int ut_abi_version(void) { return UT_ABI_VERSION; }

size_t ut_drop_background_workspace_size(int64_t L) {
  if (L < 1) return 0;
  return (size_t)compact_tiles(L) * sizeof(int32_t);
}

ut_status ut_drop_background(const uint8_t* fg_mask, int64_t L, const void* x_full,
                             int64_t row_bytes, void* x_packed, int64_t capacity,
                             int32_t* kept_idx, int32_t* inv_idx, int32_t* n_kept,
                             int64_t* n_kept_host, void* workspace, size_t workspace_bytes,
                             hipStream_t stream) {
  static const char* fn = "ut_drop_background";
  g_last_error[0] = 0;
  if (L < 1 || L >= ((int64_t)1 << 31))
    return fail(UT_ERR_INVALID_ARG, "%s: L must be in [1, 2^31) (got %lld)", fn, (long long)L);
  if (capacity < 0) return fail(UT_ERR_INVALID_ARG, "%s: capacity < 0", fn);
  UT_TRY(check_ptr(fn, "fg_mask", fg_mask, 1));
  UT_TRY(check_ptr(fn, "n_kept", n_kept, 4));
  if (capacity > 0) UT_TRY(check_ptr(fn, "kept_idx", kept_idx, 4));
  if (inv_idx) UT_TRY(check_ptr(fn, "inv_idx", inv_idx, 4));
  if ((x_full == nullptr) != (x_packed == nullptr))
    return fail(UT_ERR_INVALID_ARG, "%s: x_full and x_packed must both be NULL or both set", fn);
  if (x_full) {
    if (row_bytes <= 0 || row_bytes % 16 != 0)
      return fail(UT_ERR_INVALID_ARG, "%s: row_bytes must be a positive multiple of 16 (got %lld)",
                  fn, (long long)row_bytes);
    UT_TRY(check_ptr(fn, "x_full", x_full, 16));
    UT_TRY(check_ptr(fn, "x_packed", x_packed, 16));
  }
  const size_t need = ut_drop_background_workspace_size(L);
  if (!workspace || workspace_bytes < need)
    return fail(UT_ERR_WORKSPACE, "%s: workspace of %zu bytes required (got %zu)", fn, need,
                workspace ? workspace_bytes : (size_t)0);
  UT_TRY(check_ptr(fn, "workspace", workspace, 4));

  UT_TRY(check_hip(launch_compact(fg_mask, L, capacity, kept_idx, inv_idx, n_kept,
                                  static_cast<int32_t*>(workspace), stream),
                   "compaction launch"));
  if (x_full)
    UT_TRY(check_hip(launch_gather(x_full, row_bytes, x_packed, capacity, kept_idx, n_kept, stream),
                     "gather launch"));
  if (n_kept_host) {
    int32_t n = 0;
    UT_TRY(check_hip(hipMemcpyAsync(&n, n_kept, sizeof(n), hipMemcpyDeviceToHost, stream),
                     "n_kept copy"));
    UT_TRY(check_hip(hipStreamSynchronize(stream), "stream sync"));
    *n_kept_host = n;
    if (n > capacity)
      return fail(UT_ERR_CAPACITY, "%s: %d kept positions exceed capacity %lld", fn, n,
                  (long long)capacity);
  }
  return UT_OK;
}

ut_status ut_scatter_foreground(const void* x_packed, const int32_t* kept_idx, int64_t n_kept,
                                int64_t row_bytes, void* x_full, hipStream_t stream) {
  static const char* fn = "ut_scatter_foreground";
  g_last_error[0] = 0;
  if (n_kept < 0 || n_kept >= ((int64_t)1 << 31))
    return fail(UT_ERR_INVALID_ARG, "%s: n_kept out of range", fn);
  if (row_bytes <= 0 || row_bytes % 16 != 0)
    return fail(UT_ERR_INVALID_ARG, "%s: row_bytes must be a positive multiple of 16", fn);
  if (n_kept == 0) return UT_OK;
  UT_TRY(check_ptr(fn, "x_packed", x_packed, 16));
  UT_TRY(check_ptr(fn, "x_full", x_full, 16));
  UT_TRY(check_ptr(fn, "kept_idx", kept_idx, 4));
  return check_hip(launch_scatter(x_packed, kept_idx, n_kept, row_bytes, x_full, stream),
                   "scatter launch");
}

size_t ut_build_block_index_workspace_size(int32_t B, int32_t H, int32_t Nq, int32_t Nk) {
  // the counts are scanned in place inside q_rowptr / kv_colptr: no scratch
  (void)B, (void)H, (void)Nq, (void)Nk;
  return 0;
}

ut_status ut_build_block_index(const uint8_t* block_mask, int32_t B, int32_t H, int32_t Nq,
                               int32_t Nk, int32_t* q_rowptr, int32_t* q_cols,
                               int32_t* kv_colptr, int32_t* kv_rows, int64_t cap,
                               int64_t* nnz_host, void* workspace, size_t workspace_bytes,
                               hipStream_t stream) {
  static const char* fn = "ut_build_block_index";
  g_last_error[0] = 0;
  if (B < 1 || H < 1 || Nq < 1 || Nk < 1)
    return fail(UT_ERR_INVALID_ARG, "%s: B, H, Nq, Nk must be >= 1", fn);
  if ((int64_t)B * H > 65535)
    return fail(UT_ERR_INVALID_ARG, "%s: B*H must be <= 65535 (got %lld)", fn,
                (long long)B * H);
  // list offsets are int32: the mask may not hold 2^31 entries
  if ((int64_t)B * H * Nq * Nk >= ((int64_t)1 << 31))
    return fail(UT_ERR_INVALID_ARG, "%s: B*H*Nq*Nk = %lld reaches 2^31 (int32 offsets)", fn,
                (long long)B * H * Nq * Nk);
  if (cap < 0) return fail(UT_ERR_INVALID_ARG, "%s: cap < 0", fn);
  UT_TRY(check_ptr(fn, "block_mask", block_mask, 1));
  UT_TRY(check_ptr(fn, "q_rowptr", q_rowptr, 4));
  UT_TRY(check_ptr(fn, "kv_colptr", kv_colptr, 4));
  if (cap > 0) {
    UT_TRY(check_ptr(fn, "q_cols", q_cols, 4));
    UT_TRY(check_ptr(fn, "kv_rows", kv_rows, 4));
  }
  const size_t need = ut_build_block_index_workspace_size(B, H, Nq, Nk);
  if (workspace_bytes < need || (need > 0 && !workspace))
    return fail(UT_ERR_WORKSPACE, "%s: workspace of %zu bytes required (got %zu)", fn, need,
                workspace ? workspace_bytes : (size_t)0);
  UT_TRY(check_hip(launch_block_index(block_mask, B, H, Nq, Nk, q_rowptr, q_cols, kv_colptr,
                                      kv_rows, cap, stream),
                   "block index launch"));
  if (nnz_host) {
    int32_t nnz = 0;
    UT_TRY(check_hip(hipMemcpyAsync(&nnz, q_rowptr + (int64_t)B * H * Nq, sizeof(nnz),
                                    hipMemcpyDeviceToHost, stream),
                     "nnz copy"));
    UT_TRY(check_hip(hipStreamSynchronize(stream), "stream sync"));
    *nnz_host = nnz;
    if (nnz < 0 || nnz > cap)
      return fail(UT_ERR_CAPACITY, "%s: %d retained pairs exceed cap %lld", fn, nnz,
                  (long long)cap);
  }
  return UT_OK;
}

namespace {
// Opt-in checking of the block lists' contents (environment UT_VALIDATE set to
// anything but "0"): a debugging aid, since it waits for the stream.
bool validate_mode() {
  const char* e = std::getenv("UT_VALIDATE");
  return e && e[0] && !(e[0] == '0' && e[1] == 0);
}

// Copies a compressed list pair to the host and checks it with check_lists.
ut_status validate_lists(const char* fn, const char* what, const int32_t* ptr, const int32_t* idx,
                         int64_t rows, int32_t limit, hipStream_t stream) {
  std::vector<int32_t> p((size_t)rows + 1);
  UT_TRY(check_hip(hipMemcpyAsync(p.data(), ptr, p.size() * sizeof(int32_t), hipMemcpyDeviceToHost,
                                  stream),
                   "validate copy"));
  UT_TRY(check_hip(hipStreamSynchronize(stream), "validate sync"));
  // well-formed pointers first, so that p[rows] is a sane entry count
  UT_TRY(check_lists(fn, what, p.data(), nullptr, 0, rows, limit));
  std::vector<int32_t> v((size_t)p[rows]);
  if (!v.empty()) {
    UT_TRY(check_hip(hipMemcpyAsync(v.data(), idx, v.size() * sizeof(int32_t),
                                    hipMemcpyDeviceToHost, stream),
                     "validate copy"));
    UT_TRY(check_hip(hipStreamSynchronize(stream), "validate sync"));
  }
  return check_lists(fn, what, p.data(), v.data(), (int64_t)v.size(), rows, limit);
}
}  // namespace

ut_status ut_bsattn_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
                        int32_t B, int32_t N, int32_t H, int32_t D, int32_t block,
                        const int32_t* q_rowptr, const int32_t* q_cols, float softmax_scale,
                        hipStream_t stream) {
  static const char* fn = "ut_bsattn_fwd";
  g_last_error[0] = 0;
  UT_TRY(check_attn_common(fn, B, N, H, D, block, softmax_scale));
  UT_TRY(check_ptr(fn, "q", q, 16));
  UT_TRY(check_ptr(fn, "k", k, 16));
  UT_TRY(check_ptr(fn, "v", v, 16));
  UT_TRY(check_ptr(fn, "o", o, 16));
  UT_TRY(check_ptr(fn, "lse", lse, 4));
  UT_TRY(check_ptr(fn, "q_rowptr", q_rowptr, 4));
  UT_TRY(check_ptr(fn, "q_cols", q_cols, 4));
  const AttnShape sh{B, N, H, D, block, (N + block - 1) / block, softmax_scale, nullptr,
                     (int64_t)B * N};
  if (validate_mode())
    UT_TRY(validate_lists(fn, "row lists", q_rowptr, q_cols, (int64_t)B * H * sh.nblk, sh.nblk,
                          stream));
  return check_hip(launch_bsattn_fwd(q, k, v, o, lse, sh, q_rowptr, q_cols, stream),
                   "forward launch");
}

size_t ut_bsattn_bwd_workspace_size(int32_t B, int32_t N, int32_t H) {
  if (B < 1 || N < 1 || H < 1) return 0;
  return (size_t)B * H * N * 2 * sizeof(float);   // {LSE log2 e, delta} per query row
}


size_t ut_bsattn_bwd_workspace_size_stored(int32_t B, int32_t N, int32_t H, int32_t block,
                                           int64_t nnz) {
  if (block < 1) return 0;
  return stored_size(ut_bsattn_bwd_workspace_size(B, N, H),
                     (int64_t)B * H * (((int64_t)N + block - 1) / block), block, nnz);
}

ut_status ut_bsattn_bwd(const void* q, const void* k, const void* v, const void* o,
                        const void* dout, const float* lse, void* dq, void* dk, void* dv,
                        int32_t B, int32_t N, int32_t H, int32_t D, int32_t block,
                        const int32_t* q_rowptr, const int32_t* q_cols,
                        const int32_t* kv_colptr, const int32_t* kv_rows, float softmax_scale,
                        void* workspace, size_t workspace_bytes, hipStream_t stream) {
  static const char* fn = "ut_bsattn_bwd";
  g_last_error[0] = 0;
  UT_TRY(check_attn_common(fn, B, N, H, D, block, softmax_scale));
  const struct { const char* n; const void* p; uintptr_t a; } ptrs[] = {
      {"q", q, 16},   {"k", k, 16},   {"v", v, 16},         {"o", o, 16},
      {"dout", dout, 16}, {"lse", lse, 4}, {"dq", dq, 16},   {"dk", dk, 16},
      {"dv", dv, 16}, {"q_rowptr", q_rowptr, 4}, {"q_cols", q_cols, 4},
      {"kv_colptr", kv_colptr, 4}, {"kv_rows", kv_rows, 4}};
  for (const auto& p : ptrs) UT_TRY(check_ptr(fn, p.n, p.p, p.a));
  const size_t need = ut_bsattn_bwd_workspace_size(B, N, H);
  if (!workspace || workspace_bytes < need)
    return fail(UT_ERR_WORKSPACE, "%s: workspace of %zu bytes required (got %zu)", fn, need,
                workspace ? workspace_bytes : (size_t)0);
  UT_TRY(check_ptr(fn, "workspace", workspace, 16));
  const AttnShape sh{B, N, H, D, block, (N + block - 1) / block, softmax_scale, nullptr,
                     (int64_t)B * N};
  if (validate_mode()) {
    UT_TRY(validate_lists(fn, "row lists", q_rowptr, q_cols, (int64_t)B * H * sh.nblk, sh.nblk,
                          stream));
    UT_TRY(validate_lists(fn, "column lists", kv_colptr, kv_rows, (int64_t)B * H * sh.nblk,
                          sh.nblk, stream));
  }
  const DsTiles ds = ds_region(workspace, workspace_bytes, need, (int64_t)B * H * sh.nblk, block);
  return check_hip(launch_bsattn_bwd(q, k, v, o, dout, lse, dq, dk, dv, sh, q_rowptr, q_cols,
                                     kv_colptr, kv_rows, static_cast<float*>(workspace), ds,
                                     stream),
                   "backward launch");
}

ut_status ut_bsattn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o,
                                const void* dout, const float* lse, void* dq, void* dk, void* dv,
                                int32_t B, int32_t N, int32_t H, int32_t D, int32_t block,
                                const int32_t* q_rowptr, const int32_t* q_cols,
                                const int32_t* kv_colptr, const int32_t* kv_rows,
                                float softmax_scale, hipStream_t stream) {
  static const char* fn = "ut_bsattn_bwd_noalloc";
  g_last_error[0] = 0;
  UT_TRY(check_attn_common(fn, B, N, H, D, block, softmax_scale));
  const struct { const char* n; const void* p; uintptr_t a; } ptrs[] = {
      {"q", q, 16},   {"k", k, 16},   {"v", v, 16},         {"o", o, 16},
      {"dout", dout, 16}, {"lse", lse, 4}, {"dq", dq, 16},   {"dk", dk, 16},
      {"dv", dv, 16}, {"q_rowptr", q_rowptr, 4}, {"q_cols", q_cols, 4},
      {"kv_colptr", kv_colptr, 4}, {"kv_rows", kv_rows, 4}};
  for (const auto& p : ptrs) UT_TRY(check_ptr(fn, p.n, p.p, p.a));
  const size_t need = ut_bsattn_bwd_workspace_size(B, N, H);
  if (need > kNoallocScratchBytes)
    return fail(UT_ERR_WORKSPACE,
                "%s: B*H*N = %lld query rows need %zu bytes of scratch; the built-in scratch "
                "holds %zu bytes (%zu rows): use ut_bsattn_bwd with a workspace",
                fn, (long long)B * H * N, need, kNoallocScratchBytes,
                kNoallocScratchBytes / (2 * sizeof(float)));
  float* ws = nullptr;
  UT_TRY(check_hip(noalloc_scratch(stream, &ws), "scratch address"));
  const AttnShape sh{B, N, H, D, block, (N + block - 1) / block, softmax_scale, nullptr,
                     (int64_t)B * N};
  return check_hip(launch_bsattn_bwd(q, k, v, o, dout, lse, dq, dk, dv, sh, q_rowptr, q_cols,
                                     kv_colptr, kv_rows, ws, DsTiles{}, stream),
                   "backward launch");
}

namespace {
// Sample offsets of the variable-length calls: B + 1 device int32 values.
// Under UT_VALIDATE they are copied to the host and must start at 0, end at
// T and never decrease, with no sample longer than max_seqlen.
ut_status check_varlen(const char* fn, const int32_t* cu_seqlens, int32_t B, int64_t T,
                       int32_t max_seqlen, hipStream_t stream) {
  UT_TRY(check_ptr(fn, "cu_seqlens", cu_seqlens, 4));
  if (T < 0 || T >= ((int64_t)1 << 31))
    return fail(UT_ERR_INVALID_ARG, "%s: T = %lld outside [0, 2^31)", fn, (long long)T);
  if (!validate_mode()) return UT_OK;
  std::vector<int32_t> cu((size_t)B + 1);
  UT_TRY(check_hip(hipMemcpyAsync(cu.data(), cu_seqlens, cu.size() * sizeof(int32_t),
                                  hipMemcpyDeviceToHost, stream),
                   "validate copy"));
  UT_TRY(check_hip(hipStreamSynchronize(stream), "validate sync"));
  return check_cu_seqlens(fn, cu.data(), B, T, max_seqlen);
}
}  // namespace

ut_status ut_bsattn_fwd_varlen(const void* q, const void* k, const void* v, void* o, float* lse,
                               const int32_t* cu_seqlens, int32_t B, int64_t T,
                               int32_t max_seqlen, int32_t H, int32_t D, int32_t block,
                               const int32_t* q_rowptr, const int32_t* q_cols,
                               float softmax_scale, hipStream_t stream) {
  static const char* fn = "ut_bsattn_fwd_varlen";
  g_last_error[0] = 0;
  UT_TRY(check_attn_common(fn, B, max_seqlen, H, D, block, softmax_scale));
  UT_TRY(check_varlen(fn, cu_seqlens, B, T, max_seqlen, stream));
  if (T * H * D >= (int64_t)1 << 40) return fail(UT_ERR_INVALID_ARG, "%s: problem too large", fn);
  if (T == 0) return UT_OK;
  UT_TRY(check_ptr(fn, "q", q, 16));
  UT_TRY(check_ptr(fn, "k", k, 16));
  UT_TRY(check_ptr(fn, "v", v, 16));
  UT_TRY(check_ptr(fn, "o", o, 16));
  UT_TRY(check_ptr(fn, "lse", lse, 4));
  UT_TRY(check_ptr(fn, "q_rowptr", q_rowptr, 4));
  UT_TRY(check_ptr(fn, "q_cols", q_cols, 4));
  const AttnShape sh{B, max_seqlen, H, D, block, (max_seqlen + block - 1) / block,
                     softmax_scale, cu_seqlens, T};
  if (validate_mode())
    UT_TRY(validate_lists(fn, "row lists", q_rowptr, q_cols, (int64_t)B * H * sh.nblk, sh.nblk,
                          stream));
  return check_hip(launch_bsattn_fwd(q, k, v, o, lse, sh, q_rowptr, q_cols, stream),
                   "forward launch");
}

size_t ut_bsattn_bwd_varlen_workspace_size(int64_t T, int32_t H) {
  if (T < 1 || H < 1) return 0;
  return (size_t)T * H * 2 * sizeof(float);
}

size_t ut_bsattn_bwd_varlen_workspace_size_stored(int32_t B, int64_t T, int32_t max_seqlen,
                                                  int32_t H, int32_t block, int64_t nnz) {
  if (B < 1 || max_seqlen < 1 || block < 1) return 0;
  return stored_size(ut_bsattn_bwd_varlen_workspace_size(T, H),
                     (int64_t)B * H * (((int64_t)max_seqlen + block - 1) / block), block, nnz);
}

ut_status ut_bsattn_bwd_varlen(const void* q, const void* k, const void* v, const void* o,
                               const void* dout, const float* lse, void* dq, void* dk, void* dv,
                               const int32_t* cu_seqlens, int32_t B, int64_t T,
                               int32_t max_seqlen, int32_t H, int32_t D, int32_t block,
                               const int32_t* q_rowptr, const int32_t* q_cols,
                               const int32_t* kv_colptr, const int32_t* kv_rows,
                               float softmax_scale, void* workspace, size_t workspace_bytes,
                               hipStream_t stream) {
  static const char* fn = "ut_bsattn_bwd_varlen";
  g_last_error[0] = 0;
  UT_TRY(check_attn_common(fn, B, max_seqlen, H, D, block, softmax_scale));
  UT_TRY(check_varlen(fn, cu_seqlens, B, T, max_seqlen, stream));
  if (T * H * D >= (int64_t)1 << 40) return fail(UT_ERR_INVALID_ARG, "%s: problem too large", fn);
  if (T == 0) return UT_OK;
  const struct { const char* n; const void* p; uintptr_t a; } ptrs[] = {
      {"q", q, 16},   {"k", k, 16},   {"v", v, 16},         {"o", o, 16},
      {"dout", dout, 16}, {"lse", lse, 4}, {"dq", dq, 16},   {"dk", dk, 16},
      {"dv", dv, 16}, {"q_rowptr", q_rowptr, 4}, {"q_cols", q_cols, 4},
      {"kv_colptr", kv_colptr, 4}, {"kv_rows", kv_rows, 4}};
  for (const auto& p : ptrs) UT_TRY(check_ptr(fn, p.n, p.p, p.a));
  const size_t need = ut_bsattn_bwd_varlen_workspace_size(T, H);
  if (!workspace || workspace_bytes < need)
    return fail(UT_ERR_WORKSPACE, "%s: workspace of %zu bytes required (got %zu)", fn, need,
                workspace ? workspace_bytes : (size_t)0);
  UT_TRY(check_ptr(fn, "workspace", workspace, 16));
  const AttnShape sh{B, max_seqlen, H, D, block, (max_seqlen + block - 1) / block,
                     softmax_scale, cu_seqlens, T};
  if (validate_mode()) {
    UT_TRY(validate_lists(fn, "row lists", q_rowptr, q_cols, (int64_t)B * H * sh.nblk, sh.nblk,
                          stream));
    UT_TRY(validate_lists(fn, "column lists", kv_colptr, kv_rows, (int64_t)B * H * sh.nblk,
                          sh.nblk, stream));
  }
  const DsTiles ds = ds_region(workspace, workspace_bytes, need, (int64_t)B * H * sh.nblk, block);
  return check_hip(launch_bsattn_bwd(q, k, v, o, dout, lse, dq, dk, dv, sh, q_rowptr, q_cols,
                                     kv_colptr, kv_rows, static_cast<float*>(workspace), ds,
                                     stream),
                   "backward launch");
}

size_t ut_topk_block_mask_workspace_size(int32_t B, int32_t N, int32_t H, int32_t D,
                                         int32_t block) {
  if (B < 1 || N < 1 || H < 1 || D < 1 || block < 1) return 0;
  const int64_t nblk = ((int64_t)N + block - 1) / block;
  return (size_t)2 * B * H * nblk * D * sizeof(float);   // pooled Q and K
}

ut_status ut_topk_block_mask(const void* q, const void* k, int32_t B, int32_t N, int32_t H,
                             int32_t D, int32_t block, int32_t k_keep, int32_t prefix_blocks,
                             uint8_t* block_mask, void* workspace, size_t workspace_bytes,
                             hipStream_t stream) {
  static const char* fn = "ut_topk_block_mask";
  g_last_error[0] = 0;
  if (B < 1 || N < 1 || H < 1 || block < 1)
    return fail(UT_ERR_INVALID_ARG, "%s: B, N, H, block must be >= 1 (got %d, %d, %d, %d)", fn,
                B, N, H, block);
  if (D < 8 || D > 512 || D % 8 != 0)
    return fail(UT_ERR_INVALID_ARG, "%s: head_dim must be a multiple of 8 in [8, 512] (got %d)",
                fn, D);
  if (B > 65535) return fail(UT_ERR_INVALID_ARG, "%s: B must be <= 65535 (got %d)", fn, B);
  if (k_keep < 1) return fail(UT_ERR_INVALID_ARG, "%s: k_keep must be >= 1 (got %d)", fn, k_keep);
  const int64_t nblk = ((int64_t)N + block - 1) / block;
  if ((int64_t)B * N * H * D >= (int64_t)1 << 40 || (int64_t)B * H * nblk >= (int64_t)1 << 31)
    return fail(UT_ERR_INVALID_ARG, "%s: problem too large", fn);
  if (prefix_blocks < 0 || prefix_blocks > nblk)
    return fail(UT_ERR_INVALID_ARG, "%s: prefix_blocks must be in [0, %lld] (got %d)", fn,
                (long long)nblk, prefix_blocks);
  if (topk_rows_per_group(D, (int)nblk) == 0)
    return fail(UT_ERR_UNSUPPORTED, "%s: %lld blocks per row do not fit one workgroup", fn,
                (long long)nblk);
  UT_TRY(check_ptr(fn, "q", q, 16));
  UT_TRY(check_ptr(fn, "k", k, 16));
  UT_TRY(check_ptr(fn, "block_mask", block_mask, 1));
  const size_t need = ut_topk_block_mask_workspace_size(B, N, H, D, block);
  if (!workspace || workspace_bytes < need)
    return fail(UT_ERR_WORKSPACE, "%s: workspace of %zu bytes required (got %zu)", fn, need,
                workspace ? workspace_bytes : (size_t)0);
  UT_TRY(check_ptr(fn, "workspace", workspace, 16));
  return check_hip(launch_topk_block_mask(q, k, B, N, H, D, block, k_keep, prefix_blocks,
                                          block_mask, static_cast<float*>(workspace), stream),
                   "top-k launch");
}

namespace {
ut_status check_fg_common(const char* fn, int64_t L, int64_t C, int64_t n, const void* v,
                          ut_dtype vt) {
  if (L < 1 || L >= ((int64_t)1 << 31))
    return fail(UT_ERR_INVALID_ARG, "%s: L must be in [1, 2^31) (got %lld)", fn, (long long)L);
  if (C < 4 || C % 4 != 0 || C > (1 << 20))
    return fail(UT_ERR_INVALID_ARG, "%s: C must be a positive multiple of 4 (got %lld)", fn,
                (long long)C);
  if (n < 0 || n > L)
    return fail(UT_ERR_INVALID_ARG, "%s: n_kept must be in [0, L] (got %lld)", fn, (long long)n);
  if (vt != UT_BF16 && vt != UT_F32)
    return fail(UT_ERR_INVALID_ARG, "%s: unknown dtype %d", fn, (int)vt);
  if (n > 0) UT_TRY(check_ptr(fn, "v", v, vt == UT_BF16 ? 8 : 16));
  return UT_OK;
}
}  // namespace

ut_status ut_euler_update_foreground(float* z, int64_t L, int64_t C, const void* v,
                                     ut_dtype v_dtype, const int32_t* kept_idx,
                                     int64_t n_kept, float dt, hipStream_t stream) {
  static const char* fn = "ut_euler_update_foreground";
  g_last_error[0] = 0;
  UT_TRY(check_fg_common(fn, L, C, n_kept, v, v_dtype));
  if (!std::isfinite(dt)) return fail(UT_ERR_INVALID_ARG, "%s: dt must be finite", fn);
  if (n_kept == 0) return UT_OK;
  UT_TRY(check_ptr(fn, "z", z, 16));
  UT_TRY(check_ptr(fn, "kept_idx", kept_idx, 4));
  return check_hip(launch_euler_fg(z, L, C, v, v_dtype == UT_BF16, kept_idx, n_kept, dt, stream),
                   "euler launch");
}

size_t ut_fg_flow_loss_workspace_size(void) { return (size_t)kLossParts * sizeof(double); }

ut_status ut_fg_flow_loss(const void* v, ut_dtype v_dtype, const void* eps, const void* z0,
                          ut_dtype x_dtype, int64_t L, int64_t C, const int32_t* kept_idx,
                          int64_t n_kept, float* loss, float* grad, void* workspace,
                          size_t workspace_bytes, hipStream_t stream) {
  static const char* fn = "ut_fg_flow_loss";
  g_last_error[0] = 0;
  UT_TRY(check_fg_common(fn, L, C, n_kept, v, v_dtype));
  if (x_dtype != UT_BF16 && x_dtype != UT_F32)
    return fail(UT_ERR_INVALID_ARG, "%s: unknown dtype %d", fn, (int)x_dtype);
  UT_TRY(check_ptr(fn, "loss", loss, 4));
  if (n_kept > 0) {
    const uintptr_t xa = x_dtype == UT_BF16 ? 8 : 16;
    UT_TRY(check_ptr(fn, "eps", eps, xa));
    UT_TRY(check_ptr(fn, "z0", z0, xa));
    UT_TRY(check_ptr(fn, "kept_idx", kept_idx, 4));
    if (grad) UT_TRY(check_ptr(fn, "grad", grad, 16));
  }
  const size_t need = ut_fg_flow_loss_workspace_size();
  if (!workspace || workspace_bytes < need)
    return fail(UT_ERR_WORKSPACE, "%s: workspace of %zu bytes required (got %zu)", fn, need,
                workspace ? workspace_bytes : (size_t)0);
  UT_TRY(check_ptr(fn, "workspace", workspace, 8));
  return check_hip(launch_fg_loss(v, v_dtype == UT_BF16, eps, z0, x_dtype == UT_BF16, L, C,
                                  kept_idx, n_kept, loss, grad, static_cast<double*>(workspace),
                                  stream),
                   "loss launch");
}

ut_status ut_composite_latent(const void* x_packed, int64_t n_kept, const int32_t* inv_idx,
                              int64_t L, const void* z_bg, int64_t bg_rows, int64_t row_bytes,
                              void* z_mix, hipStream_t stream) {
  static const char* fn = "ut_composite_latent";
  g_last_error[0] = 0;
  if (L < 1 || L >= ((int64_t)1 << 31))
    return fail(UT_ERR_INVALID_ARG, "%s: L must be in [1, 2^31) (got %lld)", fn, (long long)L);
  if (bg_rows < 1)
    return fail(UT_ERR_INVALID_ARG, "%s: bg_rows must be >= 1 (got %lld)", fn, (long long)bg_rows);
  if (n_kept < 0 || n_kept > L)
    return fail(UT_ERR_INVALID_ARG, "%s: n_kept must be in [0, L] (got %lld)", fn, (long long)n_kept);
  if (row_bytes <= 0 || row_bytes % 16 != 0)
    return fail(UT_ERR_INVALID_ARG, "%s: row_bytes must be a positive multiple of 16 (got %lld)",
                fn, (long long)row_bytes);
  if (n_kept > 0) UT_TRY(check_ptr(fn, "x_packed", x_packed, 16));
  UT_TRY(check_ptr(fn, "inv_idx", inv_idx, 4));
  UT_TRY(check_ptr(fn, "z_bg", z_bg, 16));
  UT_TRY(check_ptr(fn, "z_mix", z_mix, 16));
  return check_hip(launch_composite(x_packed, n_kept, inv_idx, L, z_bg, bg_rows, row_bytes, z_mix,
                                    stream),
                   "composite launch");
}

size_t ut_token_mask_workspace_size(int32_t V, int32_t Hp, int32_t Wp, int32_t patch) {
  if (V < 1 || Hp < 1 || Wp < 1 || patch < 1) return 0;
  return (size_t)V * (Hp / patch) * (Wp / patch);
}

ut_status ut_token_mask_from_alpha(const uint8_t* alpha, int32_t V, int32_t Hp, int32_t Wp,
                                   int32_t patch, int32_t threshold, int32_t radius,
                                   uint8_t* token_mask, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  static const char* fn = "ut_token_mask_from_alpha";
  g_last_error[0] = 0;
  if (V < 1 || Hp < 1 || Wp < 1)
    return fail(UT_ERR_INVALID_ARG, "%s: V, Hp, Wp must be >= 1", fn);
  if (patch < 16 || patch % 16 != 0 || Hp % patch != 0 || Wp % patch != 0)
    return fail(UT_ERR_INVALID_ARG,
                "%s: patch must be a positive multiple of 16 dividing Hp and Wp (got %d for %d x %d)",
                fn, patch, Hp, Wp);
  if (threshold < 0 || threshold > 255)
    return fail(UT_ERR_INVALID_ARG, "%s: threshold must be in [0, 255] (got %d)", fn, threshold);
  if (radius < 0 || radius > 16)
    return fail(UT_ERR_INVALID_ARG, "%s: radius must be in [0, 16] (got %d)", fn, radius);
  if ((int64_t)V * Hp * Wp >= ((int64_t)1 << 40))
    return fail(UT_ERR_INVALID_ARG, "%s: alpha too large", fn);
  UT_TRY(check_ptr(fn, "alpha", alpha, 16));
  UT_TRY(check_ptr(fn, "token_mask", token_mask, 1));
  if (radius > 0) {
    const size_t need = ut_token_mask_workspace_size(V, Hp, Wp, patch);
    if (!workspace || workspace_bytes < need)
      return fail(UT_ERR_WORKSPACE, "%s: workspace of %zu bytes required (got %zu)", fn, need,
                  workspace ? workspace_bytes : (size_t)0);
  }
  return check_hip(launch_token_mask(alpha, V, Hp, Wp, patch, threshold, radius, token_mask,
                                     static_cast<uint8_t*>(workspace), stream),
                   "token mask launch");
}

}  // extern "C"
