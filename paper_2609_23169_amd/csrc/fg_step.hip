// Foreground-restricted sampling and training steps on gfx950 (paper
// Sec. 3.2): the Euler update applied only at the retained positions (Eq. 4)
// and the flow-matching loss over the gathered foreground target tokens
// (Eq. 3). Both are HBM-bound row gathers / scatters over the kept index list.
//
//   euler : z[kept[k], c] += dt * v[k, c], one fused multiply-add (a single
//           fp32 rounding) per element, four channels per thread; rows not
//           listed are never touched.
//   loss  : per element d = v[k, c] - (eps[i, c] - z0[i, c]), i = kept[k], in
//           fp64 (exact differences of the fp32 / bf16 inputs, then one
//           rounding each), d^2 summed in fp64 per thread and per workgroup
//           into a fixed number of partial sums, which one workgroup adds in
//           a fixed order: the loss is deterministic. The optional gradient
//           2 d / (n C) is written in fp32.
// Entries of kept outside [0, L) are skipped (they would address memory
// outside the grids).
#include <hip/hip_runtime.h>

#include "common.h"

namespace ut {
namespace {

constexpr int kThreads = 256;

template <typename T>
__device__ inline float4 load4(const T* p);
template <>
__device__ inline float4 load4<float>(const float* p) {
  return *reinterpret_cast<const float4*>(p);
}
template <>
__device__ inline float4 load4<__bf16>(const __bf16* p) {
  typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4_t;
  const bf16x4_t v = *reinterpret_cast<const bf16x4_t*>(p);
  return make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
}

template <typename VT>
__global__ __launch_bounds__(kThreads) void euler_kernel(float* __restrict__ z,
                                                         const VT* __restrict__ v,
                                                         const int32_t* __restrict__ kept,
                                                         int64_t n, int64_t L, int C, float dt) {
  const int c4n = C / 4;
  const int64_t total = n * c4n;
  for (int64_t x = (int64_t)blockIdx.x * kThreads + threadIdx.x; x < total;
       x += (int64_t)gridDim.x * kThreads) {
    const int64_t k = x / c4n;
    const int c = 4 * (int)(x % c4n);
    const int64_t i = kept[k];
    if (i < 0 || i >= L) continue;
    float* zp = z + i * C + c;
    const float4 vv = load4<VT>(v + k * C + c);
    float4 zz = *reinterpret_cast<float4*>(zp);
    zz.x = __builtin_fmaf(dt, vv.x, zz.x);
    zz.y = __builtin_fmaf(dt, vv.y, zz.y);
    zz.z = __builtin_fmaf(dt, vv.z, zz.z);
    zz.w = __builtin_fmaf(dt, vv.w, zz.w);
    *reinterpret_cast<float4*>(zp) = zz;
  }
}

template <typename VT, typename XT>
__global__ __launch_bounds__(kThreads) void loss_partial_kernel(
    const VT* __restrict__ v, const XT* __restrict__ eps, const XT* __restrict__ z0,
    const int32_t* __restrict__ kept, int64_t n, int64_t L, int C, float* __restrict__ grad,
    double* __restrict__ partial) {
  __shared__ double red[kThreads / 64];
  const int c4n = C / 4;
  const int64_t total = n * c4n;
  const double gscale = 2.0 / ((double)n * (double)C);
  double acc = 0.0;
  for (int64_t x = (int64_t)blockIdx.x * kThreads + threadIdx.x; x < total;
       x += (int64_t)gridDim.x * kThreads) {
    const int64_t k = x / c4n;
    const int c = 4 * (int)(x % c4n);
    const int64_t i = kept[k];
    if (i < 0 || i >= L) continue;
    const float4 vv = load4<VT>(v + k * C + c);
    const float4 ee = load4<XT>(eps + i * C + c);
    const float4 zz = load4<XT>(z0 + i * C + c);
    const double d0 = (double)vv.x - ((double)ee.x - (double)zz.x);
    const double d1 = (double)vv.y - ((double)ee.y - (double)zz.y);
    const double d2 = (double)vv.z - ((double)ee.z - (double)zz.z);
    const double d3 = (double)vv.w - ((double)ee.w - (double)zz.w);
    acc += d0 * d0 + d1 * d1 + d2 * d2 + d3 * d3;
    if (grad)
      *reinterpret_cast<float4*>(grad + k * C + c) =
          make_float4((float)(gscale * d0), (float)(gscale * d1), (float)(gscale * d2),
                      (float)(gscale * d3));
  }
  // fixed-order reduction: lanes by xor shuffles, then the waves in order
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int w = 0; w < kThreads / 64; ++w) s += red[w];
    partial[blockIdx.x] = s;
  }
}

__global__ __launch_bounds__(64) void loss_final_kernel(const double* __restrict__ partial,
                                                        int parts, int64_t n, int C,
                                                        float* __restrict__ loss) {
  double s = 0.0;
  for (int p = threadIdx.x; p < parts; p += 64) s += partial[p];
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
  if (threadIdx.x == 0) *loss = n > 0 ? (float)(s / ((double)n * (double)C)) : 0.f;
}

int grid_for(int64_t total4) {
  const int64_t g = (total4 + kThreads - 1) / kThreads;
  return (int)(g < 1 ? 1 : (g > kLossParts ? kLossParts : g));
}

}  // namespace

hipError_t launch_euler_fg(float* z, int64_t L, int64_t C, const void* v, bool v_bf16,
                           const int32_t* kept, int64_t n, float dt, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int grid = grid_for(n * (C / 4));
  TraceScope ts_(s, "euler");
  if (v_bf16)
    hipLaunchKernelGGL(euler_kernel<__bf16>, dim3(grid), dim3(kThreads), 0, s, z,
                       static_cast<const __bf16*>(v), kept, n, L, (int)C, dt);
  else
    hipLaunchKernelGGL(euler_kernel<float>, dim3(grid), dim3(kThreads), 0, s, z,
                       static_cast<const float*>(v), kept, n, L, (int)C, dt);
  return hipGetLastError();
}

hipError_t launch_fg_loss(const void* v, bool v_bf16, const void* eps, const void* z0,
                          bool x_bf16, int64_t L, int64_t C, const int32_t* kept, int64_t n,
                          float* loss, float* grad, double* partial, hipStream_t s) {
  const int grid = grid_for(n * (C / 4));
  const int c = (int)C;
#define UT_LOSS(VT, XT)                                                                      \
  hipLaunchKernelGGL((loss_partial_kernel<VT, XT>), dim3(grid), dim3(kThreads), 0, s,        \
                     static_cast<const VT*>(v), static_cast<const XT*>(eps),                 \
                     static_cast<const XT*>(z0), kept, n, L, c, grad, partial)
  {
    TraceScope ts_(s, "loss_partial");
    if (v_bf16 && x_bf16) UT_LOSS(__bf16, __bf16);
    else if (v_bf16) UT_LOSS(__bf16, float);
    else if (x_bf16) UT_LOSS(float, __bf16);
    else UT_LOSS(float, float);
  }
#undef UT_LOSS
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    TraceScope ts_(s, "loss_final");
    hipLaunchKernelGGL(loss_final_kernel, dim3(1), dim3(64), 0, s, partial, grid, n, c, loss);
  }
  return hipGetLastError();
}

}  // namespace ut
