// Internal declarations shared by the HIP sources of libultratex.so.
#pragma once

// Host-side declarations only (api.cpp builds with a plain C++ compiler too);
// the kernel sources include hip_runtime.h themselves.
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "ultratex.h"

namespace ut {

// Records a message for ut_last_error() and returns `st`.
ut_status fail(ut_status st, const char* fmt, ...);
// Maps a HIP error (if any) to UT_ERR_HIP with context; UT_OK otherwise.
ut_status check_hip(hipError_t e, const char* what);

// Brackets the kernel launches of its lifetime with HIP events on `s` while
// tracing is on (ut_trace_enable); name base<a,b> (a, b < 0: omitted).
class TraceScope {
 public:
  TraceScope(hipStream_t s, const char* base, int a = -1, int b = -1);
  ~TraceScope();
  TraceScope(const TraceScope&) = delete;
  TraceScope& operator=(const TraceScope&) = delete;

 private:
  hipStream_t stream_;
  hipEvent_t start_ = nullptr;
  char name_[48] = "";
};

// Host checks of the validate mode, on host copies of the arguments.
// Compressed lists: ptr[0] = 0, ptr non-decreasing, ptr[rows] = n_idx, and
// every row strictly ascending within [0, limit). With idx = NULL only the
// first two properties are checked.
ut_status check_lists(const char* fn, const char* what, const int32_t* ptr, const int32_t* idx,
                      int64_t n_idx, int64_t rows, int32_t limit);
// Sample offsets: cu[0] = 0, cu[B] = T, non-decreasing, no sample > max_seqlen.
ut_status check_cu_seqlens(const char* fn, const int32_t* cu, int32_t B, int64_t T,
                           int32_t max_seqlen);

// ---- Background Token Dropping (btd.hip) ----
constexpr int kCompactTile = 4096;   // mask bytes per workgroup of the scan
int64_t compact_tiles(int64_t L);
hipError_t launch_compact(const uint8_t* mask, int64_t L, int64_t capacity, int32_t* kept_idx,
                          int32_t* inv_idx, int32_t* n_kept, int32_t* tile_scratch,
                          hipStream_t s);
hipError_t launch_gather(const void* x_full, int64_t row_bytes, void* x_packed, int64_t capacity,
                         const int32_t* kept_idx, const int32_t* n_kept, hipStream_t s);
hipError_t launch_scatter(const void* x_packed, const int32_t* kept_idx, int64_t n_kept,
                          int64_t row_bytes, void* x_full, hipStream_t s);

// ---- Block index (block_index.hip) ----
hipError_t launch_block_index(const uint8_t* mask, int B, int H, int Nq, int Nk,
                              int32_t* q_rowptr, int32_t* q_cols, int32_t* kv_colptr,
                              int32_t* kv_rows, int64_t cap, hipStream_t s);

// ---- Attention (bsattn_fwd.hip, bsattn_bwd.hip) ----
struct AttnShape {
  int B, N, H, D, block, nblk;   // N: tokens per sample (the longest, with cu)
  float scale;
  const int32_t* cu = nullptr;   // [B + 1] sample offsets, or null for a uniform batch
  int64_t T = 0;                 // packed tokens (B N when uniform)
};
hipError_t launch_bsattn_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
                             const AttnShape& sh, const int32_t* rowptr, const int32_t* cols,
                             hipStream_t s);
// Where the backward keeps stored dS tiles (max_pairs = 0: none; dQ is then
// recomputed for every query block).
struct DsTiles {
  int32_t* row_ok = nullptr;   // [B H Nq] query block takes dQ from the tiles
  int32_t* map = nullptr;      // [max_pairs] row-list entry -> tile (column-list position)
  char* tiles = nullptr;       // [max_pairs][2 block^2] bf16 dS
  int64_t max_pairs = 0;
};
// Backward. `aux` holds the two statistics planes (8 bytes per query row).
hipError_t launch_bsattn_bwd(const void* q, const void* k, const void* v, const void* o,
                             const void* dout, const float* lse, void* dq, void* dk, void* dv,
                             const AttnShape& sh, const int32_t* rowptr, const int32_t* cols,
                             const int32_t* colptr, const int32_t* rows, float* aux,
                             const DsTiles& ds, hipStream_t s);

// Scratch of ut_bsattn_bwd_noalloc: a file-scope device array in
// bsattn_bwd.hip, one copy per GPU, holding the backward's two statistics
// planes (8 bytes per query row).
constexpr size_t kNoallocScratchBytes = (size_t)32 << 20;
// Device address of that array on the device that `s` belongs to (the current
// device for the null stream), looked up once per device.
hipError_t noalloc_scratch(hipStream_t s, float** ptr);

// ---- Top-K block selection (topk_mask.hip) ----
constexpr int64_t kTopkMaxLds = 65536;   // LDS bytes of one selection workgroup
// Query blocks per selection workgroup (16, 4 or 1), 0 if one row does not fit.
int topk_rows_per_group(int D, int nblk);
hipError_t launch_topk_block_mask(const void* q, const void* k, int B, int N, int H, int D,
                                  int block, int k_keep, int prefix, uint8_t* mask, float* pooled,
                                  hipStream_t s);

// ---- Foreground Euler update and loss (fg_step.hip) ----
constexpr int kLossParts = 1024;   // partial sums of the loss (fixed order)
hipError_t launch_euler_fg(float* z, int64_t L, int64_t C, const void* v, bool v_bf16,
                           const int32_t* kept, int64_t n, float dt, hipStream_t s);
hipError_t launch_fg_loss(const void* v, bool v_bf16, const void* eps, const void* z0,
                          bool x_bf16, int64_t L, int64_t C, const int32_t* kept, int64_t n,
                          float* loss, float* grad, double* partial, hipStream_t s);

// ---- Composite latent and token masks (composite.hip) ----
hipError_t launch_composite(const void* packed, int64_t n_kept, const int32_t* inv, int64_t L,
                            const void* bg, int64_t bg_rows, int64_t row_bytes, void* out,
                            hipStream_t s);
hipError_t launch_token_mask(const uint8_t* alpha, int V, int Hp, int Wp, int patch, int thr,
                             int radius, uint8_t* out, uint8_t* pooled, hipStream_t s);

}  // namespace ut
