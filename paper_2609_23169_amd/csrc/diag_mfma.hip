// Matrix-core rate probe (libutdiag.so, a measurement aid kept out of the
// product library): a grid of two 4-wave workgroups per CU issues only bf16
// MFMAs on operands read once from `in`, so its rate is the sustained
// matrix-core throughput of the board, under its power limit, for those
// operand values. Shape 0 issues v_mfma_f32_32x32x16_bf16, shape 1 issues
// v_mfma_f32_16x16x32_bf16 (two per 32x32x16, equal FLOPs).
// The call is declared and documented in include/ultratex_diag.h.
#include <hip/hip_runtime.h>

#include "ultratex_diag.h"

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace {

template <int SHAPE>
__global__ __launch_bounds__(256, 2) void mfma_rate_kernel(const bf16x8* __restrict__ in,
                                                           float* __restrict__ out, int iters,
                                                           unsigned long long* __restrict__ clk) {
  const int gid = blockIdx.x * 256 + threadIdx.x;
  bf16x8 a[8], b[8];
  for (int u = 0; u < 8; ++u) {
    a[u] = in[(size_t)gid * 16 + u];
    b[u] = in[(size_t)gid * 16 + 8 + u];
  }
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  float res = 0.f;
  if constexpr (SHAPE == 0) {
    f32x16 acc[4] = {};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int v = 0; v < 8; ++v)
          acc[(u * 8 + v) & 3] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[u], b[v], acc[(u * 8 + v) & 3], 0, 0, 0);
    }
    for (int i = 0; i < 4; ++i)
      for (int e = 0; e < 16; ++e) res += acc[i][e];
  } else {
    f32x4 acc[8] = {};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          acc[(u * 8 + v) & 7] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u], b[v], acc[(u * 8 + v) & 7], 0, 0, 0);
          acc[(u * 8 + v + 1) & 7] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[v], a[u], acc[(u * 8 + v + 1) & 7], 0, 0, 0);
        }
    }
    for (int i = 0; i < 8; ++i)
      for (int e = 0; e < 4; ++e) res += acc[i][e];
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  out[gid] = res;
  if (gid == 0) {
    clk[0] = t1 - t0;
    clk[1] = r1 - r0;
  }
}

}  // namespace

extern "C" int ut_diag_mfma_rate(int shape, int iters, int grid, const void* in, float* out,
                                 unsigned long long* clocks, hipStream_t s) {
  if ((shape != 0 && shape != 1) || iters < 1 || grid < 1 || !in || !out || !clocks) return -1;
  if (shape == 0)
    hipLaunchKernelGGL(mfma_rate_kernel<0>, dim3(grid), dim3(256), 0, s,
                       static_cast<const bf16x8*>(in), out, iters, clocks);
  else
    hipLaunchKernelGGL(mfma_rate_kernel<1>, dim3(grid), dim3(256), 0, s,
                       static_cast<const bf16x8*>(in), out, iters, clocks);
  return (int)hipGetLastError();
}
