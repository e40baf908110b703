// Background Token Dropping on gfx950 (paper Sec. 3.2): compaction of the
// per-view foreground mask into the ascending list of kept positions, and the
// row gather / scatter between the full token grid and the packed sequence.
//
// Compaction is three small launches over 4 KiB mask tiles (count, one-workgroup
// scan of the tile counts, fill), so any L up to 2^31 works and the result is
// deterministic. The row copies are HBM-bound: one 64-lane wave moves one row
// with 16-byte non-temporal loads and stores, all of a row's loads in flight
// before its stores.
#include <hip/hip_runtime.h>

#include "common.h"

namespace ut {
namespace {

constexpr int kThreads = 256;                       // 4 waves
constexpr int kBytesPerThread = kCompactTile / kThreads;  // 16
static_assert(kBytesPerThread == 16, "tile layout assumes 16 mask bytes per thread");

__device__ inline int wave_inclusive_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

// Exclusive prefix of x over a 256-thread block; *total receives the sum.
__device__ inline int block_exclusive_scan(int x, int* total) {
  __shared__ int wsum[kThreads / 64];
  const int inc = wave_inclusive_scan(x);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 63) wsum[w] = inc;
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kThreads / 64; ++i) {
    off += (i < w) ? wsum[i] : 0;
    tot += wsum[i];
  }
  *total = tot;
  return off + inc - x;
}

// The 16 mask bytes of this thread as a bit set (bit e = byte base+e nonzero).
__device__ inline uint32_t load_flags(const uint8_t* mask, int64_t L, int64_t base) {
  uint32_t bits = 0;
  if (base + 16 <= L && ((reinterpret_cast<uintptr_t>(mask + base) & 15) == 0)) {
    const uint4 v = *reinterpret_cast<const uint4*>(mask + base);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int b = 0; b < 4; ++b) bits |= (((w[q] >> (8 * b)) & 0xffu) != 0u) << (4 * q + b);
  } else {
    for (int e = 0; e < 16; ++e)
      if (base + e < L && mask[base + e] != 0) bits |= 1u << e;
  }
  return bits;
}

__global__ __launch_bounds__(kThreads) void compact_count(const uint8_t* __restrict__ mask,
                                                          int64_t L,
                                                          int32_t* __restrict__ tile_count) {
  const int64_t base = (int64_t)blockIdx.x * kCompactTile + threadIdx.x * kBytesPerThread;
  int total;
  block_exclusive_scan(__popc(load_flags(mask, L, base)), &total);
  if (threadIdx.x == 0) tile_count[blockIdx.x] = total;
}

// One workgroup: in-place exclusive scan of the tile counts; writes n_kept.
__global__ __launch_bounds__(kThreads) void compact_scan(int32_t* __restrict__ tile, int64_t ntiles,
                                                         int32_t* __restrict__ n_kept) {
  int carry = 0;
  for (int64_t c0 = 0; c0 < ntiles; c0 += kThreads) {
    const int64_t t = c0 + threadIdx.x;
    const int x = t < ntiles ? tile[t] : 0;
    int total;
    const int ex = block_exclusive_scan(x, &total);
    if (t < ntiles) tile[t] = carry + ex;
    carry += total;
    __syncthreads();  // wsum is reused by the next chunk
  }
  if (threadIdx.x == 0) *n_kept = carry;
}

__global__ __launch_bounds__(kThreads) void compact_fill(const uint8_t* __restrict__ mask, int64_t L,
                                                         const int32_t* __restrict__ tile_off,
                                                         int64_t capacity,
                                                         int32_t* __restrict__ kept_idx,
                                                         int32_t* __restrict__ inv_idx) {
  const int64_t base = (int64_t)blockIdx.x * kCompactTile + threadIdx.x * kBytesPerThread;
  const uint32_t bits = load_flags(mask, L, base);
  int total;
  int k = tile_off[blockIdx.x] + block_exclusive_scan(__popc(bits), &total);
  for (int e = 0; e < 16; ++e) {
    const int64_t p = base + e;
    if (p >= L) break;
    if (bits & (1u << e)) {
      if (k < capacity) kept_idx[k] = (int32_t)p;
      if (inv_idx) inv_idx[p] = k;
      ++k;
    } else if (inv_idx) {
      inv_idx[p] = -1;
    }
  }
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kRowsPerBlock = kThreads / 64;  // one wave per row
constexpr int kUnroll = 8;                    // 8 KiB of a row in flight per wave
constexpr int64_t kGatherRowsPerPass = 131072;  // rows of one gather pass (32768 workgroups)

__device__ inline void copy_row(const u32x4* __restrict__ s, u32x4* __restrict__ d, int64_t nvec) {
  const int lane = threadIdx.x & 63;
  for (int64_t c = lane; c < nvec; c += 64 * kUnroll) {
    u32x4 tmp[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (c + 64 * u < nvec) tmp[u] = __builtin_nontemporal_load(s + c + 64 * u);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (c + 64 * u < nvec) __builtin_nontemporal_store(tmp[u], d + c + 64 * u);
  }
}

// The kept count is only known on the device, so the grid is sized for
// min(capacity, kGatherRowsPerPass) rows and each wave strides over the kept
// rows: a capacity far above the kept count launches no idle workgroups
// beyond one pass.
__global__ __launch_bounds__(kThreads) void gather_rows(const u32x4* __restrict__ src, int64_t nvec,
                                                        u32x4* __restrict__ dst, int64_t capacity,
                                                        const int32_t* __restrict__ kept_idx,
                                                        const int32_t* __restrict__ n_kept) {
  const int64_t n = min((int64_t)*n_kept, capacity);
  const int64_t stride = (int64_t)gridDim.x * kRowsPerBlock;
  for (int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6); row < n;
       row += stride) {
    const int64_t srow = kept_idx[row];
    copy_row(src + srow * nvec, dst + row * nvec, nvec);
  }
}

__global__ __launch_bounds__(kThreads) void scatter_rows(const u32x4* __restrict__ src, int64_t nvec,
                                                         u32x4* __restrict__ dst, int64_t n,
                                                         const int32_t* __restrict__ kept_idx) {
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= n) return;
  const int64_t drow = kept_idx[row];
  copy_row(src + row * nvec, dst + drow * nvec, nvec);
}

}  // namespace

int64_t compact_tiles(int64_t L) { return (L + kCompactTile - 1) / kCompactTile; }

hipError_t launch_compact(const uint8_t* mask, int64_t L, int64_t capacity, int32_t* kept_idx,
                          int32_t* inv_idx, int32_t* n_kept, int32_t* tile_scratch,
                          hipStream_t s) {
  const int64_t nt = compact_tiles(L);
  {
    TraceScope ts_(s, "compact_count");
    hipLaunchKernelGGL(compact_count, dim3((unsigned)nt), dim3(kThreads), 0, s, mask, L, tile_scratch);
  }
  {
    TraceScope ts_(s, "compact_scan");
    hipLaunchKernelGGL(compact_scan, dim3(1), dim3(kThreads), 0, s, tile_scratch, nt, n_kept);
  }
  {
    TraceScope ts_(s, "compact_fill");
    hipLaunchKernelGGL(compact_fill, dim3((unsigned)nt), dim3(kThreads), 0, s, mask, L, tile_scratch,
                     capacity, kept_idx, inv_idx);
  }
  return hipGetLastError();
}

hipError_t launch_gather(const void* x_full, int64_t row_bytes, void* x_packed, int64_t capacity,
                         const int32_t* kept_idx, const int32_t* n_kept, hipStream_t s) {
  if (capacity == 0) return hipSuccess;
  const int64_t rows = min(capacity, kGatherRowsPerPass);
  const int64_t blocks = (rows + kRowsPerBlock - 1) / kRowsPerBlock;
  {
    TraceScope ts_(s, "gather_rows");
    hipLaunchKernelGGL(gather_rows, dim3((unsigned)blocks), dim3(kThreads), 0, s,
                     static_cast<const u32x4*>(x_full), row_bytes / 16,
                     static_cast<u32x4*>(x_packed), capacity, kept_idx, n_kept);
  }
  return hipGetLastError();
}

hipError_t launch_scatter(const void* x_packed, const int32_t* kept_idx, int64_t n_kept,
                          int64_t row_bytes, void* x_full, hipStream_t s) {
  if (n_kept == 0) return hipSuccess;
  const int64_t blocks = (n_kept + kRowsPerBlock - 1) / kRowsPerBlock;
  {
    TraceScope ts_(s, "scatter_rows");
    hipLaunchKernelGGL(scatter_rows, dim3((unsigned)blocks), dim3(kThreads), 0, s,
                     static_cast<const u32x4*>(x_packed), row_bytes / 16,
                     static_cast<u32x4*>(x_full), n_kept, kept_idx);
  }
  return hipGetLastError();
}

}  // namespace ut
