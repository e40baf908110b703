// Block-sparse attention backward on gfx950: gradients of Eq. 8 (paper
// Sec. 3.3) with the block mask held constant. Three launches, no atomics:
//
//   delta  : delta_r = sum_d dO[r,d] * O[r,d]   (fp32, one pass over O and dO)
//   dK/dV  : one workgroup per (b, h, key block j), walking the query blocks
//            that select j (column lists). Each wave owns 32 keys and keeps
//            its K and V rows as MFMA operands in registers. Per 64-query
//            sub-tile staged in LDS: S = Q K^T and dP = dO V^T (lane = key
//            column), P = exp(S - LSE), dS = P (dP - delta), then
//            dV^T += dO^T P and dK^T += Q^T dS with transposing LDS reads.
//   dQ     : one workgroup per (b, h, query block i), walking S_i (row
//            lists). Each wave owns 32 queries (Q and dO rows in registers).
//            Per 64-key sub-tile: S^T = K Q^T, dP^T = V dO^T (lane = query
//            column), dS^T, then dQ^T += K^T dS^T.
//
// The dQ pass recomputes S and dP rather than accumulating dQ with atomics
// from the dK/dV pass: the result is deterministic.
#include "attn_util.h"
#include "common.h"

namespace ut {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// delta = rowsum(dO o O)
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_delta_kernel(const __bf16* __restrict__ O,
                                                        const __bf16* __restrict__ dO,
                                                        float* __restrict__ delta, int B, int N,
                                                        int H) {
  constexpr int CPR = D / 8;  // lanes per (token, head) row
  const int64_t rows = (int64_t)B * N * H;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = gid / CPR;  // (b, n, h) in memory order
  const int c = (int)(gid % CPR);
  float acc = 0.f;
  if (row < rows) {
    const bf16x8 o = *reinterpret_cast<const bf16x8*>(O + row * D + 8 * c);
    const bf16x8 d = *reinterpret_cast<const bf16x8*>(dO + row * D + 8 * c);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc += (float)o[e] * (float)d[e];
  }
#pragma unroll
  for (int m = CPR / 2; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
  if (row < rows && c == 0) {
    const int h = (int)(row % H);
    const int64_t bn = row / H;
    const int n = (int)(bn % N), b = (int)(bn / N);
    delta[((int64_t)b * H + h) * N + n] = acc;
  }
}

template <int D, int BLOCK>
struct BwdCfg {
  static constexpr int NW = BLOCK / 32;
  static constexpr int NT = 64 * NW;
  static constexpr int ST = 64;                  // rows per sub-tile
  static constexpr int SUBS = BLOCK / ST;
  static constexpr int CPR = D / 8;
  static constexpr int TILEB = ST * D * 2;       // one 64-row bf16 tile
  static constexpr int KS = D / 16;
  static constexpr int DT = D / 32;
  static constexpr int LPT = 2 * ST * CPR / NT;  // 16-byte loads per thread per stage
  static_assert(2 * ST * CPR % NT == 0, "stage must split evenly over threads");
};

// ---------------------------------------------------------------------------
// dK, dV: key-stationary over the column lists
// ---------------------------------------------------------------------------
template <int D, int BLOCK>
__global__ __launch_bounds__(64 * (BLOCK / 32), 1) void bwd_dkdv_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const __bf16* __restrict__ dO, const float* __restrict__ LSE, const float* __restrict__ delta,
    __bf16* __restrict__ dK, __bf16* __restrict__ dV, int B, int N, int H, int nblk, float scale,
    const int32_t* __restrict__ colptr, const int32_t* __restrict__ rows_list) {
  using C = BwdCfg<D, BLOCK>;
  constexpr int STAGEB = 2 * C::TILEB + 2 * C::ST * 4;   // Q, dO, lse2, delta
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGEB];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g = lane >> 5;
  const int64_t G = (int64_t)B * H * nblk;
  const int64_t lt = xcd_tile(blockIdx.x, G);
  const int j = (int)(lt % nblk);
  const int64_t bh = lt / nblk;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int64_t tok_stride = (int64_t)H * D;
  const int64_t base_bh = (int64_t)b * N * tok_stride + (int64_t)h * D;

  const int key = j * BLOCK + 32 * w + l32;  // this lane's key row (column of S)
  const int p0 = colptr[lt], p1 = colptr[lt + 1];
  const int T = (p1 - p0) * C::SUBS;

  f32x16 dkt[C::DT], dvt[C::DT];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) dkt[dt] = dvt[dt] = f32x16{};

  if (T > 0) {
    bf16x8 kop[C::KS], vop[C::KS];
    {
      const int64_t off = base_bh + (int64_t)min(key, N - 1) * tok_stride + 8 * g;
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        kop[ks] = *reinterpret_cast<const bf16x8*>(K + off + 16 * ks);
        vop[ks] = *reinterpret_cast<const bf16x8*>(V + off + 16 * ks);
      }
    }
    u32x4 stg[C::LPT];
    float stg_f = 0.f;
    auto load_stage = [&](int t) __attribute__((always_inline)) {
      const int i = rows_list[p0 + t / C::SUBS];
      const int r0 = i * BLOCK + (t % C::SUBS) * C::ST;
#pragma unroll
      for (int u = 0; u < C::LPT; ++u) {
        const int x = tid + C::NT * u;
        const int isdo = x / (C::ST * C::CPR);
        const int r = (x / C::CPR) % C::ST, c = x % C::CPR;
        const int qr = min(r0 + r, N - 1);
        stg[u] = *reinterpret_cast<const u32x4*>((isdo ? dO : Q) + base_bh + (int64_t)qr * tok_stride + 8 * c);
      }
      if (tid < 2 * C::ST) {
        const int r = tid % C::ST, qr = r0 + r;
        if (tid < C::ST)
          stg_f = qr < N ? LSE[bh * N + qr] * kLog2e : INFINITY;   // rows past N: P = 0
        else
          stg_f = qr < N ? delta[bh * N + qr] : 0.f;
      }
    };
    auto store_stage = [&](int s) __attribute__((always_inline)) {
      char* st = smem + s * STAGEB;
#pragma unroll
      for (int u = 0; u < C::LPT; ++u) {
        const int x = tid + C::NT * u;
        const int isdo = x / (C::ST * C::CPR);
        const int r = (x / C::CPR) % C::ST, c = x % C::CPR;
        *reinterpret_cast<u32x4*>(st + isdo * C::TILEB + lds_off<C::CPR>(r, c)) = stg[u];
      }
      if (tid < 2 * C::ST) reinterpret_cast<float*>(st + 2 * C::TILEB)[tid] = stg_f;
    };

    const float c2 = scale * kLog2e;
    const int jr = lane & 15;
    const int dsub = 16 * ((lane >> 4) & 1) + 4 * (jr & 3);

    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int t = 0; t < T; ++t) {
      const int cur = t & 1;
      if (t + 1 < T) load_stage(t + 1);
      const char* q_lds = smem + cur * STAGEB;
      const char* do_lds = q_lds + C::TILEB;
      const float* lse_lds = reinterpret_cast<const float*>(q_lds + 2 * C::TILEB);
      const float* dl_lds = lse_lds + C::ST;

      // S = Q K^T and dP = dO V^T, two 32-query tiles; lane column = key
      f32x16 s[2] = {f32x16{}, f32x16{}}, dp[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks)
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
          const int off = lds_off<C::CPR>(32 * qt + l32, 2 * ks + g);
          s[qt] = mfma32(*reinterpret_cast<const bf16x8*>(q_lds + off), kop[ks], s[qt]);
          dp[qt] = mfma32(*reinterpret_cast<const bf16x8*>(do_lds + off), vop[ks], dp[qt]);
        }

      bf16x8 pb[2][2], dsb[2][2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const int r = 32 * qt + 8 * a + 4 * g;
          const f32x4 l4 = *reinterpret_cast<const f32x4*>(lse_lds + r);
          const f32x4 d4 = *reinterpret_cast<const f32x4*>(dl_lds + r);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int idx = 4 * a + e;
            const float p = fast_exp2(__builtin_fmaf(s[qt][idx], c2, -l4[e]));
            const float ds = p * (dp[qt][idx] - d4[e]);
            pb[qt][idx >> 3][idx & 7] = (__bf16)p;
            dsb[qt][idx >> 3][idx & 7] = (__bf16)ds;
          }
        }

      // dV^T += dO^T P and dK^T += Q^T dS (contraction over the 64 queries)
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int r0 = 32 * qt + 16 * hh + 4 * g + (jr >> 2);
            const int d = 32 * dt + dsub;
            const int o_lo = lds_off<C::CPR>(r0, d >> 3) + 2 * (d & 7);
            const int o_hi = lds_off<C::CPR>(r0 + 8, d >> 3) + 2 * (d & 7);
            const s16x4 dlo = lds_read_tr16(do_lds + o_lo), dhi = lds_read_tr16(do_lds + o_hi);
            const s16x4 qlo = lds_read_tr16(q_lds + o_lo), qhi = lds_read_tr16(q_lds + o_hi);
            const s16x8 d8 = {dlo[0], dlo[1], dlo[2], dlo[3], dhi[0], dhi[1], dhi[2], dhi[3]};
            const s16x8 q8 = {qlo[0], qlo[1], qlo[2], qlo[3], qhi[0], qhi[1], qhi[2], qhi[3]};
            dvt[dt] = mfma32(__builtin_bit_cast(bf16x8, d8), pb[qt][hh], dvt[dt]);
            dkt[dt] = mfma32(__builtin_bit_cast(bf16x8, q8), dsb[qt][hh], dkt[dt]);
          }

      if (t + 1 < T) store_stage(cur ^ 1);
      __syncthreads();
    }
  }

  if (key < N) {
    const int64_t off = base_bh + (int64_t)key * tok_stride;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        bf16x4 k4, v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          k4[e] = (__bf16)(dkt[dt][4 * a + e] * scale);
          v4[e] = (__bf16)dvt[dt][4 * a + e];
        }
        *reinterpret_cast<bf16x4*>(dK + off + 32 * dt + 8 * a + 4 * g) = k4;
        *reinterpret_cast<bf16x4*>(dV + off + 32 * dt + 8 * a + 4 * g) = v4;
      }
  }
}

// ---------------------------------------------------------------------------
// dQ: query-stationary over the row lists
// ---------------------------------------------------------------------------
template <int D, int BLOCK>
__global__ __launch_bounds__(64 * (BLOCK / 32), 1) void bwd_dq_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const __bf16* __restrict__ dO, const float* __restrict__ LSE, const float* __restrict__ delta,
    __bf16* __restrict__ dQ, int B, int N, int H, int nblk, float scale,
    const int32_t* __restrict__ rowptr, const int32_t* __restrict__ cols) {
  using C = BwdCfg<D, BLOCK>;
  constexpr int STAGEB = 2 * C::TILEB;   // K, V
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGEB];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g = lane >> 5;
  const int64_t G = (int64_t)B * H * nblk;
  const int64_t lt = xcd_tile(blockIdx.x, G);
  const int i = (int)(lt % nblk);
  const int64_t bh = lt / nblk;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int64_t tok_stride = (int64_t)H * D;
  const int64_t base_bh = (int64_t)b * N * tok_stride + (int64_t)h * D;

  const int q = i * BLOCK + 32 * w + l32;
  const int p0 = rowptr[lt], p1 = rowptr[lt + 1];
  const int T = (p1 - p0) * C::SUBS;

  f32x16 dqt[C::DT];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) dqt[dt] = f32x16{};

  if (T > 0) {
    bf16x8 qop[C::KS], doop[C::KS];
    {
      const int64_t off = base_bh + (int64_t)min(q, N - 1) * tok_stride + 8 * g;
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        qop[ks] = *reinterpret_cast<const bf16x8*>(Q + off + 16 * ks);
        doop[ks] = *reinterpret_cast<const bf16x8*>(dO + off + 16 * ks);
      }
    }
    const float lse2 = q < N ? LSE[bh * N + q] * kLog2e : INFINITY;
    const float dl = q < N ? delta[bh * N + q] : 0.f;

    u32x4 stg[C::LPT];
    auto load_stage = [&](int t) __attribute__((always_inline)) {
      const int j = cols[p0 + t / C::SUBS];
      const int k0 = j * BLOCK + (t % C::SUBS) * C::ST;
#pragma unroll
      for (int u = 0; u < C::LPT; ++u) {
        const int x = tid + C::NT * u;
        const int isv = x / (C::ST * C::CPR);
        const int r = (x / C::CPR) % C::ST, c = x % C::CPR;
        const int kr = min(k0 + r, N - 1);
        stg[u] = *reinterpret_cast<const u32x4*>((isv ? V : K) + base_bh + (int64_t)kr * tok_stride + 8 * c);
      }
    };
    auto store_stage = [&](int s) __attribute__((always_inline)) {
      char* st = smem + s * STAGEB;
#pragma unroll
      for (int u = 0; u < C::LPT; ++u) {
        const int x = tid + C::NT * u;
        const int isv = x / (C::ST * C::CPR);
        const int r = (x / C::CPR) % C::ST, c = x % C::CPR;
        *reinterpret_cast<u32x4*>(st + isv * C::TILEB + lds_off<C::CPR>(r, c)) = stg[u];
      }
    };

    const float c2 = scale * kLog2e;
    const int jr = lane & 15;
    const int dsub = 16 * ((lane >> 4) & 1) + 4 * (jr & 3);

    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int t = 0; t < T; ++t) {
      const int cur = t & 1;
      if (t + 1 < T) load_stage(t + 1);
      const char* k_lds = smem + cur * STAGEB;
      const char* v_lds = k_lds + C::TILEB;

      f32x16 s[2] = {f32x16{}, f32x16{}}, dp[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          const int off = lds_off<C::CPR>(32 * kt + l32, 2 * ks + g);
          s[kt] = mfma32(*reinterpret_cast<const bf16x8*>(k_lds + off), qop[ks], s[kt]);
          dp[kt] = mfma32(*reinterpret_cast<const bf16x8*>(v_lds + off), doop[ks], dp[kt]);
        }

      const int j = cols[p0 + t / C::SUBS];
      const int k0 = j * BLOCK + (t % C::SUBS) * C::ST;
      const bool tail = k0 + C::ST > N;
      bf16x8 dsb[2][2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          float p = fast_exp2(__builtin_fmaf(s[kt][e], c2, -lse2));
          if (tail && k0 + 32 * kt + 8 * (e >> 2) + 4 * g + (e & 3) >= N) p = 0.f;
          dsb[kt][e >> 3][e & 7] = (__bf16)(p * (dp[kt][e] - dl));
        }

      // dQ^T += K^T dS^T (contraction over the 64 keys)
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int r0 = 32 * kt + 16 * hh + 4 * g + (jr >> 2);
            const int d = 32 * dt + dsub;
            const s16x4 lo = lds_read_tr16(k_lds + lds_off<C::CPR>(r0, d >> 3) + 2 * (d & 7));
            const s16x4 hi = lds_read_tr16(k_lds + lds_off<C::CPR>(r0 + 8, d >> 3) + 2 * (d & 7));
            const s16x8 k8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            dqt[dt] = mfma32(__builtin_bit_cast(bf16x8, k8), dsb[kt][hh], dqt[dt]);
          }

      if (t + 1 < T) store_stage(cur ^ 1);
      __syncthreads();
    }
  }

  if (q < N) {
    const int64_t off = base_bh + (int64_t)q * tok_stride;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        bf16x4 v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = (__bf16)(dqt[dt][4 * a + e] * scale);
        *reinterpret_cast<bf16x4*>(dQ + off + 32 * dt + 8 * a + 4 * g) = v4;
      }
  }
}

template <int D, int BLOCK>
hipError_t launch_bwd_t(const void* q, const void* k, const void* v, const void* o,
                        const void* dout, const float* lse, void* dq, void* dk, void* dv,
                        const AttnShape& sh, const int32_t* rowptr, const int32_t* cols,
                        const int32_t* colptr, const int32_t* rows, float* delta, hipStream_t s) {
  auto bf = [](const void* p) { return static_cast<const __bf16*>(p); };
  const int64_t rows_total = (int64_t)sh.B * sh.N * sh.H * (D / 8);
  hipLaunchKernelGGL((bwd_delta_kernel<D>), dim3((unsigned)((rows_total + 255) / 256)), dim3(256), 0,
                     s, bf(o), bf(dout), delta, sh.B, sh.N, sh.H);
  const int64_t G = (int64_t)sh.B * sh.H * sh.nblk;
  constexpr int NT = BwdCfg<D, BLOCK>::NT;
  hipLaunchKernelGGL((bwd_dkdv_kernel<D, BLOCK>), dim3((unsigned)G), dim3(NT), 0, s, bf(q), bf(k),
                     bf(v), bf(dout), lse, delta, static_cast<__bf16*>(dk),
                     static_cast<__bf16*>(dv), sh.B, sh.N, sh.H, sh.nblk, sh.scale, colptr, rows);
  hipLaunchKernelGGL((bwd_dq_kernel<D, BLOCK>), dim3((unsigned)G), dim3(NT), 0, s, bf(q), bf(k),
                     bf(v), bf(dout), lse, delta, static_cast<__bf16*>(dq), sh.B, sh.N, sh.H,
                     sh.nblk, sh.scale, rowptr, cols);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bsattn_bwd(const void* q, const void* k, const void* v, const void* o,
                             const void* dout, const float* lse, void* dq, void* dk, void* dv,
                             const AttnShape& sh, const int32_t* rowptr, const int32_t* cols,
                             const int32_t* colptr, const int32_t* rows, float* delta,
                             hipStream_t s) {
#define UT_BWD(DD, BB)                                                                        \
  if (sh.D == DD && sh.block == BB)                                                           \
    return launch_bwd_t<DD, BB>(q, k, v, o, dout, lse, dq, dk, dv, sh, rowptr, cols, colptr, \
                                rows, delta, s);
  UT_BWD(128, 128)
  UT_BWD(128, 64)
  UT_BWD(64, 128)
  UT_BWD(64, 64)
#undef UT_BWD
  return hipErrorInvalidValue;
}

}  // namespace ut
