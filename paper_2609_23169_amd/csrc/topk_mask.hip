// Top-K block selection on gfx950 (paper Sec. 3.3, Eq. 6 and Eq. 7): the
// block mask of block-sparse attention, chosen from mean-pooled query and key
// blocks. Two launches:
//
//   pool   : one workgroup per (block i, batch b, tensor Q or K). It streams
//            the block's token rows once, all heads together (each row is
//            H*D contiguous bf16, read in coalesced 16-byte chunks), sums
//            them in fp32 and divides by the block's real token count.
//            HBM-bound: Q and K are each read exactly once.
//   select : one workgroup per (b, h, 16 consecutive query blocks). It
//            first forms the 16 score rows S_c[i, j] = pool(Q)_i . pool(K)_j
//            in LDS as order-preserving integer keys (fp32 MFMA for head_dim
//            64 / 128 and rows of at most 1024 blocks; fp32 fused
//            multiply-adds otherwise, with fewer rows per workgroup when a
//            row is long), then each wave takes one row at a time: a 32-step
//            radix select (counts by ballot and scalar popcount) finds the
//            k-th largest key, and the row of the mask keeps every larger key
//            plus, of the keys equal to it, the lowest block indices up to k
//            in total. With P prefix blocks (always-kept text tokens), the
//            first P rows are dense, the first P columns are always kept, and
//            the k best blocks are chosen among the rest.
#include <algorithm>

#include <hip/hip_runtime.h>

#include "common.h"

namespace ut {
namespace {

constexpr int kPoolMaxThreads = 1024;
constexpr int kSelThreads = 256;       // generic selection workgroup
constexpr int kSelMfmaThreads = 512;   // MFMA-path selection workgroup

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;

// pool(x)[b, h, i, d] = (1 / r_i) sum_{t in block i} x[b, t, h, d], written to
// out[((b H + h) nblk + i) D + d] (pq for Q, pk for K). Thread (g, c) of the
// workgroup (blockDim.x = G * stride, stride >= chunks) sums 16-byte chunk c of
// the rows of part g of the block (G parts of consecutive rows, so G times the
// loads in flight); part 0 then adds the other parts' sums from LDS in the
// order g = 1 .. G-1, so the result does not depend on timing.
__global__ __launch_bounds__(kPoolMaxThreads) void pool_kernel(const __bf16* __restrict__ q,
                                                            const __bf16* __restrict__ k,
                                                            float* __restrict__ pq,
                                                            float* __restrict__ pk, int N, int H,
                                                            int D, int block, int nblk, int stride) {
  __shared__ float part[kPoolMaxThreads * 8];   // sums of parts 1 .. G-1: [g - 1][c][8]
  const int i = blockIdx.x, b = blockIdx.y;
  const __bf16* __restrict__ x = blockIdx.z ? k : q;
  float* __restrict__ out = blockIdx.z ? pk : pq;
  const int64_t row = (int64_t)H * D;              // elements per token
  const int t0 = i * block, r = min(N, t0 + block) - t0;
  const int chunks = H * D / 8, cpr = D / 8;       // 8-element chunks per token / per head
  const int G = blockDim.x / stride;               // 1 whenever chunks > stride
  const int g = threadIdx.x / stride;
  const int ta = r * g / G, tb = r * (g + 1) / G;  // this part's rows
  for (int c = threadIdx.x % stride; c - (int)(threadIdx.x % stride) < chunks; c += stride) {
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (c < chunks) {
      const __bf16* src = x + ((int64_t)b * N + t0) * row + 8 * c;
#pragma unroll 16
      for (int t = ta; t < tb; ++t) {
        const bf16x8_t v = __builtin_nontemporal_load(reinterpret_cast<const bf16x8_t*>(src + t * row));
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += (float)v[e];
      }
    }
    if (G > 1) {   // a single pass: stride >= chunks
      if (g > 0 && c < chunks) {
#pragma unroll
        for (int e = 0; e < 8; ++e) part[((g - 1) * stride + c) * 8 + e] = acc[e];
      }
      __syncthreads();
      if (g == 0 && c < chunks)
        for (int gg = 1; gg < G; ++gg)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[e] += part[((gg - 1) * stride + c) * 8 + e];
    }
    if (g > 0 || c >= chunks) continue;
    const int h = c / cpr, d0 = 8 * (c % cpr);
    // true division keeps the mean correctly rounded (one rounding after the sum)
    float* dst = out + (((int64_t)b * H + h) * nblk + i) * D + d0;
    float4 lo, hi;
    lo.x = acc[0] / (float)r; lo.y = acc[1] / (float)r; lo.z = acc[2] / (float)r; lo.w = acc[3] / (float)r;
    hi.x = acc[4] / (float)r; hi.y = acc[5] / (float)r; hi.z = acc[6] / (float)r; hi.w = acc[7] / (float)r;
    reinterpret_cast<float4*>(dst)[0] = lo;
    reinterpret_cast<float4*>(dst)[1] = hi;
  }
}

// Order-preserving map of a finite float to uint32 (larger float, larger key).
__device__ inline uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Keys of one row: in registers (M64 > 0: at most 64 * M64 blocks) or read
// from LDS each time (M64 == 0).
template <int M64>
struct RowKeys {
  uint32_t k[M64 > 0 ? M64 : 1];
  const uint32_t* lds;
  int nk, lane;
  __device__ RowKeys(const uint32_t* row, int nk_, int lane_) : lds(row), nk(nk_), lane(lane_) {
    if constexpr (M64 > 0) {
#pragma unroll
      for (int m = 0; m < M64; ++m) k[m] = 64 * m + lane < nk ? row[64 * m + lane] : 0u;
    }
  }
  // Number of keys of the row for which pred(key) holds (uniform). Slots
  // past nk hold key 0, which no predicate used here accepts (they compare
  // a key with >= T | bit or > T), so the register path needs no guard.
  template <typename Pred>
  __device__ int count(Pred pred) const {
    int n = 0;
    if constexpr (M64 > 0) {
#pragma unroll
      for (int m = 0; m < M64; ++m) n += __popcll(__ballot(pred(k[m])));
    } else {
      for (int base = 0; base < nk; base += 64)
        n += __popcll(__ballot(base + lane < nk && pred(lds[base + lane])));
    }
    return n;
  }
};

// One wave selects rows r0, r0 + step, ... of the workgroup's score rows in
// `keys` ([rows][nk] order keys) and writes their mask rows.
template <int M64>
__device__ void select_rows(uint32_t* keys, uint8_t* mask_rows, int i0, int rows, int r0,
                            int step, int nk, int k_keep, int prefix, int lane) {
  for (int r = r0; r < rows; r += step) {
    uint8_t* mrow = mask_rows + (int64_t)r * nk;
    if (i0 + r < prefix || k_keep >= nk - prefix) {   // a dense row
      for (int j = lane; j < nk; j += 64) mrow[j] = 1;
      continue;
    }
    // Prefix columns are always kept: give them key 0, which no threshold
    // accepts (every score maps to a key >= 1), and choose among the rest.
    for (int j = lane; j < prefix; j += 64) keys[r * nk + j] = 0u;
    const RowKeys<M64> rk(keys + r * nk, nk, lane);
    // T = the largest key with at least k_keep keys >= T, i.e. the k-th largest.
    uint32_t T = 0;
    for (int bit = 31; bit >= 0; --bit) {
      const uint32_t cand = T | (1u << bit);
      if (rk.count([cand](uint32_t x) { return x >= cand; }) >= k_keep) T = cand;
    }
    // scores equal to the k-th are taken lowest j first, up to k_keep in all
    int quota = k_keep - rk.count([T](uint32_t x) { return x > T; });
    auto emit = [&](int m, uint32_t key) __attribute__((always_inline)) {
      const int j = 64 * m + lane;
      const bool tie = j < nk && key == T;
      const uint64_t tm = __ballot(tie);
      const int before = __popcll(tm & ((1ull << lane) - 1ull));
      if (j < nk) mrow[j] = (j < prefix || key > T || (tie && before < quota)) ? 1 : 0;
      quota -= __popcll(tm);
    };
    if constexpr (M64 > 0) {
#pragma unroll
      for (int m = 0; m < M64; ++m)
        if (64 * m < nk) emit(m, rk.k[m]);
    } else {
      for (int m = 0; 64 * m < nk; ++m) emit(m, 64 * m + lane < nk ? rk.lds[64 * m + lane] : 0u);
    }
  }
}

// Fast path: 16 query blocks per workgroup, D in {64, 128}, and a score row
// short enough that the 16 rows of keys and the pooled rows fit 64 KiB of LDS.
// Scores with v_mfma_f32_16x16x4_f32: wave w takes key tiles of 16 blocks;
// k-step s of lane group g = lane / 16 covers d = 16 (s / 4) + 4 g + s % 4,
// so each lane reads whole float4s of a pooled row (a row's 4 groups read 64
// contiguous bytes). Every product is exact in fp32 and each sum is rounded
// in fp32, as in the generic path.
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

template <int D>
__global__ __launch_bounds__(kSelMfmaThreads) void select_mfma_kernel(const float* __restrict__ pq,
                                                                  const float* __restrict__ pk,
                                                                  uint8_t* __restrict__ mask,
                                                                  int nq, int nk, int k_keep,
                                                                  int prefix) {
  constexpr int QR = 16;
  __shared__ __attribute__((aligned(16))) float sq[QR * D];
  extern __shared__ uint32_t keys[];   // [QR][nk]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int groups = (nq + QR - 1) / QR;
  const int64_t bh = blockIdx.x / groups;
  const int i0 = (int)(blockIdx.x % groups) * QR;
  const int rows = min(QR, nq - i0);
  for (int x = tid; x < QR * D; x += kSelMfmaThreads)
    sq[x] = x / D < rows ? pq[(bh * nq + i0) * D + x] : 0.f;
  __syncthreads();

  const int l16 = lane & 15, g = lane >> 4;
  const float* const pkh = pk + bh * nk * (int64_t)D;
  for (int j0 = 16 * w; j0 < nk; j0 += 16 * (kSelMfmaThreads / 64)) {
    const int j = j0 + l16;
    const float* krow = pkh + (int64_t)min(j, nk - 1) * D;
    f32x4_t c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < D / 16; ++q) {
      const float4 kv = *reinterpret_cast<const float4*>(krow + 16 * q + 4 * g);
      const float4 qv = *reinterpret_cast<const float4*>(sq + l16 * D + 16 * q + 4 * g);
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(qv.x, kv.x, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(qv.y, kv.y, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(qv.z, kv.z, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(qv.w, kv.w, c, 0, 0, 0);
    }
    // c[e] = S_c[i0 + 4 g + e, j]
    if (j < nk) {
#pragma unroll
      for (int e = 0; e < 4; ++e) keys[(4 * g + e) * nk + j] = order_key(c[e] + 0.0f);   // -0 -> +0
    }
  }
  __syncthreads();
  select_rows<16>(keys, mask + (bh * nq + i0) * (int64_t)nk, i0, rows, w, kSelMfmaThreads / 64, nk,
                  k_keep, prefix, lane);
}

// Generic path: QR query blocks per workgroup, any D (multiple of 8).
template <int QR>
__global__ __launch_bounds__(kSelThreads) void select_kernel(const float* __restrict__ pq,
                                                             const float* __restrict__ pk,
                                                             uint8_t* __restrict__ mask, int D,
                                                             int nq, int nk, int k_keep,
                                                             int prefix) {
  extern __shared__ float smem[];   // [QR][D] pooled query rows, then [QR][nk] keys
  float* const sq = smem;
  uint32_t* const keys = reinterpret_cast<uint32_t*>(smem + QR * D);
  const int tid = threadIdx.x;
  const int groups = (nq + QR - 1) / QR;
  const int64_t bh = blockIdx.x / groups;
  const int i0 = (int)(blockIdx.x % groups) * QR;
  const int rows = min(QR, nq - i0);
  for (int x = tid; x < QR * D; x += kSelThreads)
    sq[x] = x / D < rows ? pq[(bh * nq + i0) * D + x] : 0.f;
  __syncthreads();

  // one lane per key block j, all QR rows at once, d in order
  for (int j = tid; j < nk; j += kSelThreads) {
    float acc[QR];
#pragma unroll
    for (int r = 0; r < QR; ++r) acc[r] = 0.f;
    const float4* kr = reinterpret_cast<const float4*>(pk + (bh * nk + j) * D);
    for (int d4 = 0; d4 < D / 4; ++d4) {
      const float4 kv = kr[d4];
#pragma unroll
      for (int r = 0; r < QR; ++r) {
        const float4 qv = reinterpret_cast<const float4*>(sq + r * D)[d4];
        acc[r] = __builtin_fmaf(qv.x, kv.x, acc[r]);
        acc[r] = __builtin_fmaf(qv.y, kv.y, acc[r]);
        acc[r] = __builtin_fmaf(qv.z, kv.z, acc[r]);
        acc[r] = __builtin_fmaf(qv.w, kv.w, acc[r]);
      }
    }
#pragma unroll
    for (int r = 0; r < QR; ++r) keys[r * nk + j] = order_key(acc[r] + 0.0f);   // -0 -> +0
  }
  __syncthreads();
  select_rows<0>(keys, mask + (bh * nq + i0) * (int64_t)nk, i0, rows, threadIdx.x >> 6,
                 kSelThreads / 64, nk, k_keep, prefix, threadIdx.x & 63);
}

template <int QR>
hipError_t launch_select(const float* pq, const float* pk, uint8_t* mask, int B, int H, int D,
                         int nq, int k_keep, int prefix, hipStream_t s) {
  const int groups = (nq + QR - 1) / QR;
  const size_t lds = (size_t)QR * (D + nq) * sizeof(float);
  {
    TraceScope ts_(s, "topk_select", QR);
    hipLaunchKernelGGL((select_kernel<QR>), dim3((unsigned)((int64_t)B * H * groups)),
                     dim3(kSelThreads), lds, s, pq, pk, mask, D, nq, nq, k_keep, prefix);
  }
  return hipGetLastError();
}

template <int D>
hipError_t launch_select_mfma(const float* pq, const float* pk, uint8_t* mask, int B, int H,
                              int nq, int k_keep, int prefix, hipStream_t s) {
  const int groups = (nq + 15) / 16;
  {
    TraceScope ts_(s, "topk_select_mfma", D);
    hipLaunchKernelGGL((select_mfma_kernel<D>), dim3((unsigned)((int64_t)B * H * groups)),
                     dim3(kSelMfmaThreads), (size_t)16 * nq * sizeof(uint32_t), s, pq, pk, mask, nq,
                     nq, k_keep, prefix);
  }
  return hipGetLastError();
}

}  // namespace

int topk_rows_per_group(int D, int nblk) {
  const int64_t per_row = (int64_t)(D + nblk) * sizeof(float);
  for (int qr : {16, 4, 1})
    if (qr * per_row <= kTopkMaxLds) return qr;
  return 0;
}

hipError_t launch_topk_block_mask(const void* q, const void* k, int B, int N, int H, int D,
                                  int block, int k_keep, int prefix, uint8_t* mask, float* pooled,
                                  hipStream_t s) {
  const int nblk = (N + block - 1) / block;
  float* pq = pooled;
  float* pk = pooled + (size_t)B * H * nblk * D;
  // one 16-byte chunk of a token row per thread, the block's rows in up to
  // four parts (at most 1024 threads); more chunks than that loop per thread
  const int chunks = H * D / 8;
  const int stride = (int)std::min<int64_t>(kPoolMaxThreads, (chunks + 63) / 64 * 64);
  const int parts = std::max(1, std::min(4, kPoolMaxThreads / stride));
  {
    TraceScope ts_(s, "topk_pool");
    hipLaunchKernelGGL(pool_kernel, dim3((unsigned)nblk, (unsigned)B, 2), dim3(stride * parts), 0, s,
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), pq, pk, N, H,
                     D, block, nblk, stride);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if ((D == 64 || D == 128) && 16 * (int64_t)(D + nblk) * 4 <= kTopkMaxLds)
    return D == 128 ? launch_select_mfma<128>(pq, pk, mask, B, H, nblk, k_keep, prefix, s)
                    : launch_select_mfma<64>(pq, pk, mask, B, H, nblk, k_keep, prefix, s);
  const int qr = topk_rows_per_group(D, nblk);
  if (qr == 16) return launch_select<16>(pq, pk, mask, B, H, D, nblk, k_keep, prefix, s);
  if (qr == 4) return launch_select<4>(pq, pk, mask, B, H, D, nblk, k_keep, prefix, s);
  return launch_select<1>(pq, pk, mask, B, H, D, nblk, k_keep, prefix, s);
}

}  // namespace ut
