// Foreground-aware decoding input and token masks on gfx950.
//
//   composite : Eq. 9 (paper Sec. 3.4). One pass over the full grid: row i of
//               the output is packed row inv_idx[i] where the position was
//               retained, otherwise row i mod P of the canonical background
//               latent (one view's token grid, tile-repeated over the views).
//               Reads through the inverse index map, so every output row is
//               written exactly once with coalesced 16-byte stores.
//   token mask: Sec. 3.2 mask construction. pool: one thread per token ORs
//               its patch x patch block of the alpha mask (16-byte loads,
//               alpha > threshold); dilate: one thread per token ORs the
//               (2 radius + 1)^2 square of pooled tokens around it, clipped
//               at the view border.
#include <hip/hip_runtime.h>

#include "common.h"

namespace ut {
namespace {

constexpr int kThreads = 256;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;

__global__ __launch_bounds__(kThreads) void composite_kernel(
    const u32x4_t* __restrict__ packed, int64_t n_kept, const int32_t* __restrict__ inv,
    int64_t L, const u32x4_t* __restrict__ bg, int64_t bg_rows, int64_t cpr,
    u32x4_t* __restrict__ out) {
  const int64_t total = L * cpr;
  for (int64_t x = (int64_t)blockIdx.x * kThreads + threadIdx.x; x < total;
       x += (int64_t)gridDim.x * kThreads) {
    const int64_t i = x / cpr, c = x % cpr;
    const int64_t k = inv[i];
    const u32x4_t* src = (k >= 0 && k < n_kept) ? packed + k * cpr : bg + (i % bg_rows) * cpr;
    out[x] = src[c];
  }
}

// Byte-wise "any byte > t" of a 16-byte segment.
__device__ inline bool any_above(u32x4_t w, uint32_t t) {
  if (t == 0) return (w[0] | w[1] | w[2] | w[3]) != 0u;
  bool a = false;
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int b = 0; b < 4; ++b) a |= ((w[e] >> (8 * b)) & 0xffu) > t;
  return a;
}

__global__ __launch_bounds__(kThreads) void mask_pool_kernel(const uint8_t* __restrict__ alpha,
                                                             int V, int Hp, int Wp, int patch,
                                                             uint32_t thr,
                                                             uint8_t* __restrict__ pooled) {
  const int gh = Hp / patch, gw = Wp / patch;
  const int64_t total = (int64_t)V * gh * gw;
  for (int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * kThreads) {
    const int x = (int)(t % gw), y = (int)((t / gw) % gh);
    const int64_t v = t / ((int64_t)gw * gh);
    const uint8_t* base = alpha + ((v * Hp + (int64_t)y * patch) * Wp + (int64_t)x * patch);
    bool any = false;
    for (int py = 0; py < patch && !any; ++py)
      for (int s = 0; s < patch / 16; ++s)
        any |= any_above(*reinterpret_cast<const u32x4_t*>(base + (int64_t)py * Wp + 16 * s), thr);
    pooled[t] = any ? 1 : 0;
  }
}

__global__ __launch_bounds__(kThreads) void mask_dilate_kernel(const uint8_t* __restrict__ pooled,
                                                               int V, int gh, int gw, int radius,
                                                               uint8_t* __restrict__ out) {
  const int64_t total = (int64_t)V * gh * gw;
  for (int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * kThreads) {
    const int x = (int)(t % gw), y = (int)((t / gw) % gh);
    const uint8_t* view = pooled + (t / ((int64_t)gw * gh)) * gh * gw;
    const int y0 = max(0, y - radius), y1 = min(gh, y + radius + 1);
    const int x0 = max(0, x - radius), x1 = min(gw, x + radius + 1);
    uint8_t any = 0;
    for (int yy = y0; yy < y1; ++yy)
      for (int xx = x0; xx < x1; ++xx) any |= view[yy * gw + xx];
    out[t] = any ? 1 : 0;
  }
}

unsigned grid_of(int64_t work) {
  const int64_t g = (work + kThreads - 1) / kThreads;
  return (unsigned)(g < 1 ? 1 : (g > 65536 ? 65536 : g));
}

}  // namespace

hipError_t launch_composite(const void* packed, int64_t n_kept, const int32_t* inv, int64_t L,
                            const void* bg, int64_t bg_rows, int64_t row_bytes, void* out,
                            hipStream_t s) {
  const int64_t cpr = row_bytes / 16;
  {
    TraceScope ts_(s, "composite");
    hipLaunchKernelGGL(composite_kernel, dim3(grid_of(L * cpr)), dim3(kThreads), 0, s,
                     static_cast<const u32x4_t*>(packed), n_kept, inv, L,
                     static_cast<const u32x4_t*>(bg), bg_rows, cpr, static_cast<u32x4_t*>(out));
  }
  return hipGetLastError();
}

hipError_t launch_token_mask(const uint8_t* alpha, int V, int Hp, int Wp, int patch, int thr,
                             int radius, uint8_t* out, uint8_t* pooled, hipStream_t s) {
  const int gh = Hp / patch, gw = Wp / patch;
  const int64_t tokens = (int64_t)V * gh * gw;
  {
    TraceScope ts_(s, "mask_pool");
    hipLaunchKernelGGL(mask_pool_kernel, dim3(grid_of(tokens)), dim3(kThreads), 0, s, alpha, V, Hp,
                     Wp, patch, (uint32_t)thr, radius > 0 ? pooled : out);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || radius == 0) return e;
  {
    TraceScope ts_(s, "mask_dilate");
    hipLaunchKernelGGL(mask_dilate_kernel, dim3(grid_of(tokens)), dim3(kThreads), 0, s, pooled, V,
                     gh, gw, radius, out);
  }
  return hipGetLastError();
}

}  // namespace ut
