// Block lists from a binary block mask on gfx950 (paper Sec. 3.3, Eq. 7 and
// the selected sets S_i of Eq. 8).
//
// Row lists (S_i, ascending j) feed the forward and the dQ pass; column lists
// (query blocks selecting key block j, ascending i) feed the dK/dV pass. Both
// are built without atomics, so the output is unique and deterministic, in
// three launches:
//   1. the count of every row and every column;
//   2. an in-place scan of each count array into offsets (one workgroup per
//      array);
//   3. fill: the same traversals, each entry written at its list's offset
//      plus the number of set entries before it.
// Launches 1 and 3 each build both kinds of list: their first workgroups take
// a 64-column slab of one (b, h) each (column lists), the rest take 64 mask
// rows each (row lists).
#include <hip/hip_runtime.h>

#include "common.h"

namespace ut {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kRowChunks = 8;     // 64-column chunks of a row loaded before their ballots
constexpr int kRowsPerWave = 4;   // mask rows per wave in the row lists

__device__ inline uint64_t lanes_below_mask() {
  const int lane = threadIdx.x & 63;
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

__device__ inline uint64_t readlane64(uint64_t v, int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, lane);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

// Row lists: each wave takes kRowsPerWave consecutive mask rows (of B*H*Nq),
// 64 columns per ballot.
template <bool kFill>
__device__ void row_lists(const uint8_t* __restrict__ mask, int64_t rows, int Nk,
                          int32_t* __restrict__ rowptr, int32_t* __restrict__ cols, int64_t cap,
                          int64_t wg) {
  const int64_t r0 = (wg * kWaves + (threadIdx.x >> 6)) * kRowsPerWave;
  if (r0 >= rows) return;   // no barrier below
  const int lane = threadIdx.x & 63;
  int64_t pos[kRowsPerWave];
#pragma unroll
  for (int q = 0; q < kRowsPerWave; ++q) pos[q] = kFill && r0 + q < rows ? rowptr[r0 + q] : 0;
  for (int j0 = 0; j0 < Nk; j0 += 64 * kRowChunks) {
    // every load issued before any is tested (rows past the last and columns
    // past Nk re-read the last ones and are masked)
    uint32_t b[kRowsPerWave][kRowChunks];
#pragma unroll
    for (int q = 0; q < kRowsPerWave; ++q) {
      const uint8_t* row = mask + min(r0 + q, rows - 1) * Nk;
#pragma unroll
      for (int u = 0; u < kRowChunks; ++u) b[q][u] = row[min(j0 + 64 * u + lane, Nk - 1)];
    }
#pragma unroll
    for (int q = 0; q < kRowsPerWave; ++q) {
#pragma unroll
      for (int u = 0; u < kRowChunks; ++u) {
        const int j = j0 + 64 * u + lane;
        const bool set = r0 + q < rows && j < Nk && b[q][u] != 0;
        const uint64_t bal = __ballot(set);
        if (kFill && set) {
          const int64_t k = pos[q] + __popcll(bal & lanes_below_mask());
          if (k < cap) cols[k] = j;
        }
        pos[q] += __popcll(bal);
      }
    }
  }
  if (!kFill && lane == 0) {
#pragma unroll
    for (int q = 0; q < kRowsPerWave; ++q)
      if (r0 + q < rows) rowptr[r0 + q + 1] = (int32_t)pos[q];
  }
}

// Column lists: the workgroup owns columns j0..j0+63 of one (b, h); lane c is
// column j0 + c. Wave w walks a contiguous range of 64-row tiles; per tile
// each lane gathers its column's 64 bits with one coalesced 64-byte load per
// row. The waves' counts, added in wave order through LDS, place each wave's
// rows within its columns' lists; filling then takes the columns one at a
// time with the lanes as rows, so each column's new entries are written
// contiguously.
template <bool kFill>
__device__ void col_lists(const uint8_t* __restrict__ mask, int Nq, int Nk,
                          int32_t* __restrict__ colptr, int32_t* __restrict__ rows_out,
                          int64_t cap, int64_t wg, int slabs, int* __restrict__ part) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t bh = wg / slabs;
  const int j = (int)(wg % slabs) * 64 + lane;
  const bool col_ok = j < Nk;
  const int ntiles = (Nq + 63) / 64;
  const int per = (ntiles + kWaves - 1) / kWaves;
  const int t0 = min(ntiles, w * per), t1 = min(ntiles, t0 + per);
  const uint8_t* col = mask + bh * (int64_t)Nq * Nk + j;
  auto bits = [&](int t) __attribute__((always_inline)) {
    const int i0 = 64 * t;
    uint64_t m = 0;
    if (col_ok) {
      // 32 loads at a time, issued before any is tested (rows past Nq re-read
      // the last row and are masked): a guard per load would wait for each
      // one in turn
#pragma unroll
      for (int h = 0; h < 64; h += 32) {
        uint32_t b[32];
#pragma unroll
        for (int u = 0; u < 32; ++u) b[u] = col[(int64_t)min(i0 + h + u, Nq - 1) * Nk];
#pragma unroll
        for (int u = 0; u < 32; ++u)
          if (i0 + h + u < Nq && b[u] != 0) m |= 1ull << (h + u);
      }
    }
    return m;
  };
  // a wave with one tile (Nq <= 1024) keeps its mask for the fill
  const uint64_t one = t1 - t0 == 1 ? bits(t0) : 0;
  int cnt = __popcll(one);
  if (t1 - t0 > 1)
    for (int t = t0; t < t1; ++t) cnt += __popcll(bits(t));
  part[w * 64 + lane] = cnt;
  __syncthreads();
  if (!kFill) {
    if (w == 0 && col_ok) {
      int tot = 0;
      for (int x = 0; x < kWaves; ++x) tot += part[x * 64 + lane];
      colptr[bh * Nk + j + 1] = tot;
    }
    return;
  }
  // this wave's first entry of the lane's column: the column's offset plus
  // the entries of the earlier waves' (lower) rows
  int64_t pos = col_ok ? colptr[bh * Nk + j] : 0;
  for (int x = 0; x < w; ++x) pos += part[x * 64 + lane];
  for (int t = t0; t < t1; ++t) {
    const uint64_t m = t1 - t0 == 1 ? one : bits(t);
    // one column at a time, the lanes as the tile's rows: the column's set
    // rows go to consecutive entries
    for (int c = 0; c < 64; ++c) {
      const uint64_t mc = readlane64(m, c);   // column j0 + c, rows 64 t .. +63
      if (mc == 0) continue;
      const int64_t pc = (int64_t)readlane64((uint64_t)pos, c);
      if ((mc >> lane) & 1) {
        const int64_t k = pc + __popcll(mc & lanes_below_mask());
        if (k < cap) rows_out[k] = 64 * t + lane;
      }
    }
    pos += __popcll(m);
  }
}

// Launch 1 (counts) and 3 (fill): workgroups [0, col_wgs) build column lists,
// the rest row lists.
template <bool kFill>
__global__ __launch_bounds__(kThreads) void index_pass(const uint8_t* __restrict__ mask, int64_t rows,
                                                       int Nq, int Nk, int slabs, int64_t col_wgs,
                                                       int32_t* __restrict__ rowptr,
                                                       int32_t* __restrict__ cols,
                                                       int32_t* __restrict__ colptr,
                                                       int32_t* __restrict__ rows_out, int64_t cap) {
  __shared__ int part[kThreads];
  const int64_t wg = blockIdx.x;
  if (wg < col_wgs)
    col_lists<kFill>(mask, Nq, Nk, colptr, rows_out, cap, wg, slabs, part);
  else
    row_lists<kFill>(mask, rows, Nk, rowptr, cols, cap, wg - col_wgs);
}

// In-place scan: ptr[1..n] holds counts -> ptr[0..n] holds offsets.
// blockIdx.x selects one of two arrays. Each pass stages 16K counts in LDS
// with coalesced loads, scans 16 consecutive counts per thread, and writes
// the offsets back coalesced (one pass for the lists of a 2K canvas).
constexpr int kScanThreads = 1024;
constexpr int kScanPer = 16;
constexpr int kScanChunk = kScanThreads * kScanPer;

__global__ __launch_bounds__(kScanThreads) void scan_counts(int32_t* __restrict__ a, int64_t na,
                                                            int32_t* __restrict__ b, int64_t nb) {
  int32_t* p = blockIdx.x == 0 ? a : b;
  const int64_t n = blockIdx.x == 0 ? na : nb;
  // logical count L at buf[L + L / 16]: conflict-free both for the
  // coalesced order (consecutive L per lane) and for 16 consecutive counts
  // per thread (lane stride 17)
  __shared__ int buf[kScanChunk + kScanChunk / 16];
  auto at = [](int L) { return L + (L >> 4); };
  __shared__ int wsum[kScanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int carry = 0;
  if (tid == 0) p[0] = 0;
  for (int64_t c0 = 1; c0 <= n; c0 += kScanChunk) {
#pragma unroll
    for (int e = 0; e < kScanPer; ++e) {
      const int64_t i = c0 + e * kScanThreads + tid;
      buf[at(e * kScanThreads + tid)] = i <= n ? p[i] : 0;
    }
    __syncthreads();
    int x[kScanPer];
    int s = 0;
#pragma unroll
    for (int e = 0; e < kScanPer; ++e) {
      s += buf[at(tid * kScanPer + e)];
      x[e] = s;   // inclusive within the thread
    }
    int incl = s;   // inclusive over the wave's threads
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o, 64);
      if (lane >= o) incl += y;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    int off = carry + incl - s, tot = 0;
    for (int i = 0; i < kScanThreads / 64; ++i) {
      off += (i < w) ? wsum[i] : 0;
      tot += wsum[i];
    }
#pragma unroll
    for (int e = 0; e < kScanPer; ++e) buf[at(tid * kScanPer + e)] = off + x[e];
    __syncthreads();
#pragma unroll
    for (int e = 0; e < kScanPer; ++e) {
      const int64_t i = c0 + e * kScanThreads + tid;
      if (i <= n) p[i] = buf[at(e * kScanThreads + tid)];
    }
    carry += tot;
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_block_index(const uint8_t* mask, int B, int H, int Nq, int Nk,
                              int32_t* q_rowptr, int32_t* q_cols, int32_t* kv_colptr,
                              int32_t* kv_rows, int64_t cap, hipStream_t s) {
  const int64_t rows = (int64_t)B * H * Nq;
  const int slabs = (Nk + 63) / 64;
  const int64_t col_wgs = (int64_t)slabs * B * H;
  const int64_t row_wgs = (rows + kWaves * kRowsPerWave - 1) / (kWaves * kRowsPerWave);
  const dim3 grid((unsigned)(col_wgs + row_wgs));
  {
    TraceScope ts_(s, "index_count");
    hipLaunchKernelGGL(index_pass<false>, grid, dim3(kThreads), 0, s, mask, rows, Nq, Nk, slabs,
                       col_wgs, q_rowptr, q_cols, kv_colptr, kv_rows, cap);
  }
  {
    TraceScope ts_(s, "index_scan");
    hipLaunchKernelGGL(scan_counts, dim3(2), dim3(kScanThreads), 0, s, q_rowptr, rows, kv_colptr,
                       (int64_t)B * H * Nk);
  }
  {
    TraceScope ts_(s, "index_fill");
    hipLaunchKernelGGL(index_pass<true>, grid, dim3(kThreads), 0, s, mask, rows, Nq, Nk, slabs,
                       col_wgs, q_rowptr, q_cols, kv_colptr, kv_rows, cap);
  }
  return hipGetLastError();
}

}  // namespace ut
