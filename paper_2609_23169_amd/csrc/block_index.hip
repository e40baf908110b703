// Block lists from a binary block mask on gfx950 (paper Sec. 3.3, Eq. 7 and
// the selected sets S_i of Eq. 8).
//
// Row lists (S_i, ascending j) feed the forward and the dQ pass; column lists
// (query blocks selecting key block j, ascending i) feed the dK/dV pass. Both
// are built without atomics, so the output is unique and deterministic:
//   1. counts: one wave per mask row (64-column ballots); one workgroup per
//      (b, h, 64-column slab) that walks 64x64 byte tiles through LDS and
//      counts each column with one ballot per tile;
//   2. an in-place scan of the counts into offsets (one workgroup per list);
//   3. fill: the same traversals, each lane writing its index at
//      offset + popcount of the set lanes below it.
#include <hip/hip_runtime.h>

#include "common.h"

namespace ut {
namespace {

constexpr int kThreads = 256;

__device__ inline uint64_t lanes_below_mask() {
  const int lane = threadIdx.x & 63;
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// One wave per row r in [0, rows): counts (fill == false) or writes (fill).
template <bool kFill>
__global__ __launch_bounds__(kThreads) void rows_pass(const uint8_t* __restrict__ mask, int64_t rows,
                                                      int Nk, int32_t* __restrict__ rowptr,
                                                      int32_t* __restrict__ cols, int64_t cap) {
  const int64_t r = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int lane = threadIdx.x & 63;
  const uint8_t* row = mask + r * Nk;
  int64_t pos = kFill ? rowptr[r] : 0;
  for (int j0 = 0; j0 < Nk; j0 += 64) {
    const int j = j0 + lane;
    const bool set = j < Nk && row[j] != 0;
    const uint64_t bal = __ballot(set);
    if (kFill && set) {
      const int64_t k = pos + __popcll(bal & lanes_below_mask());
      if (k < cap) cols[k] = j;
    }
    pos += __popcll(bal);
  }
  if (!kFill && lane == 0) rowptr[r + 1] = (int32_t)pos;
}

// One workgroup per (slab of 64 columns, b*h): walks the Nq rows in 64-row
// tiles staged in LDS; wave w owns columns 16w..16w+15 of the slab.
template <bool kFill>
__global__ __launch_bounds__(kThreads) void cols_pass(const uint8_t* __restrict__ mask, int Nq,
                                                      int Nk, int32_t* __restrict__ colptr,
                                                      int32_t* __restrict__ rows_out,
                                                      int64_t cap) {
  __shared__ uint8_t tile[64][64 + 4];
  const int64_t bh = blockIdx.y;
  const int j0 = blockIdx.x * 64;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint8_t* base = mask + bh * (int64_t)Nq * Nk;
  int64_t pos[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    const int j = j0 + 16 * w + c;
    pos[c] = (kFill && j < Nk) ? colptr[bh * Nk + j] : 0;
  }
  for (int i0 = 0; i0 < Nq; i0 += 64) {
    // 64 x 64 bytes: thread t loads row t/4, bytes 16*(t%4) .. +15
    const int tr = threadIdx.x >> 2, tc = 16 * (threadIdx.x & 3);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int i = i0 + tr, j = j0 + tc + e;
      tile[tr][tc + e] = (i < Nq && j < Nk) ? base[(int64_t)i * Nk + j] : 0;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const int jl = 16 * w + c;
      const bool set = tile[lane][jl] != 0;
      const uint64_t bal = __ballot(set);
      if (kFill && set) {
        const int64_t k = pos[c] + __popcll(bal & lanes_below_mask());
        if (k < cap) rows_out[k] = i0 + lane;
      }
      pos[c] += __popcll(bal);
    }
    __syncthreads();
  }
  if (!kFill && lane == 0) {
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const int j = j0 + 16 * w + c;
      if (j < Nk) colptr[bh * Nk + j + 1] = (int32_t)pos[c];
    }
  }
}

// In-place scan: ptr[1..n] holds counts -> ptr[0..n] holds offsets.
// blockIdx.x selects one of two arrays.
__global__ __launch_bounds__(1024) void scan_counts(int32_t* __restrict__ a, int64_t na,
                                                    int32_t* __restrict__ b, int64_t nb) {
  int32_t* p = blockIdx.x == 0 ? a : b;
  const int64_t n = blockIdx.x == 0 ? na : nb;
  __shared__ int wsum[16];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int carry = 0;
  if (threadIdx.x == 0) p[0] = 0;
  for (int64_t c0 = 1; c0 <= n; c0 += 1024) {
    const int64_t t = c0 + threadIdx.x;
    int x = t <= n ? p[t] : 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    int off = carry, tot = 0;
    for (int i = 0; i < 16; ++i) {
      off += (i < w) ? wsum[i] : 0;
      tot += wsum[i];
    }
    if (t <= n) p[t] = off + x;
    carry += tot;
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_block_index(const uint8_t* mask, int B, int H, int Nq, int Nk,
                              int32_t* q_rowptr, int32_t* q_cols, int32_t* kv_colptr,
                              int32_t* kv_rows, int64_t cap, hipStream_t s) {
  const int64_t rows = (int64_t)B * H * Nq;
  const unsigned row_blocks = (unsigned)((rows + 3) / 4);
  const dim3 col_grid((unsigned)((Nk + 63) / 64), (unsigned)(B * H));
  {
    TraceScope ts_(s, "rows_pass_count");
    hipLaunchKernelGGL(rows_pass<false>, dim3(row_blocks), dim3(kThreads), 0, s, mask, rows, Nk,
                     q_rowptr, q_cols, cap);
  }
  {
    TraceScope ts_(s, "cols_pass_count");
    hipLaunchKernelGGL(cols_pass<false>, col_grid, dim3(kThreads), 0, s, mask, Nq, Nk, kv_colptr,
                     kv_rows, cap);
  }
  {
    TraceScope ts_(s, "scan_counts");
    hipLaunchKernelGGL(scan_counts, dim3(2), dim3(1024), 0, s, q_rowptr, rows, kv_colptr,
                     (int64_t)B * H * Nk);
  }
  {
    TraceScope ts_(s, "rows_pass_fill");
    hipLaunchKernelGGL(rows_pass<true>, dim3(row_blocks), dim3(kThreads), 0, s, mask, rows, Nk,
                     q_rowptr, q_cols, cap);
  }
  {
    TraceScope ts_(s, "cols_pass_fill");
    hipLaunchKernelGGL(cols_pass<true>, col_grid, dim3(kThreads), 0, s, mask, Nq, Nk, kv_colptr,
                     kv_rows, cap);
  }
  return hipGetLastError();
}

}  // namespace ut
