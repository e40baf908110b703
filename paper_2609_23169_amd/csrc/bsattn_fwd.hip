// Block-sparse attention forward on gfx950 (paper Sec. 3.3, Eq. 8): for each
// (batch, head, query block i), O_i = softmax(Q_i K_{S_i}^T * scale) V_{S_i}
// with an online softmax over the listed key blocks only; key blocks outside
// S_i are never read.
//
// One workgroup per (b, h, i); BLOCK/32 waves, each owning 32 query rows.
// Scores are formed transposed, S^T = K Q^T, with 32x32x16 bf16 MFMA: each
// lane then holds one query column (16 keys per 32x32 tile), so row max and
// row sum are in-lane plus one permlane32 swap, and the probabilities feed the
// second product O^T += V^T P^T straight from registers as the B operand.
// V^T operands come from LDS with the transposing ds_read_b64_tr_b16.
// Keys stream through LDS in 64-key sub-tiles, double buffered: the global
// loads of sub-tile t+1 are in flight (in registers) while sub-tile t is
// computed, then written to the other LDS stage before one barrier.
#include "attn_util.h"
#include "common.h"

namespace ut {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <int D, int BLOCK>
struct FwdCfg {
  static constexpr int NW = BLOCK / 32;          // waves per workgroup
  static constexpr int NT = 64 * NW;             // threads
  static constexpr int KT = 64;                  // keys per sub-tile
  static constexpr int SUBS = BLOCK / KT;        // sub-tiles per key block
  static constexpr int ROWB = D * 2;             // bytes per LDS row
  static constexpr int CPR = D / 8;              // 16-byte chunks per row
  static constexpr int TILEB = KT * ROWB;        // one K or V sub-tile
  static constexpr int STAGEB = 2 * TILEB;       // K + V
  static constexpr int LDSB = 2 * STAGEB;        // two stages
  static constexpr int LPT = 2 * KT * CPR / NT;  // 16-byte loads per thread per stage
  static constexpr int KS = D / 16;              // k-steps of the score product
  static constexpr int DT = D / 32;              // 32-wide d tiles of O
  static_assert(2 * KT * CPR % NT == 0, "stage must split evenly over threads");
};

template <int D, int BLOCK>
__global__ __launch_bounds__(64 * (BLOCK / 32), (BLOCK == 128 || D == 64) ? 2 : 1) void bsattn_fwd_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    __bf16* __restrict__ O, float* __restrict__ LSE, int B, int N, int H, int nblk, float scale,
    const int32_t* __restrict__ rowptr, const int32_t* __restrict__ cols) {
  using C = FwdCfg<D, BLOCK>;
  __shared__ __attribute__((aligned(16))) char smem[C::LDSB];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g = lane >> 5;
  const int64_t G = (int64_t)B * H * nblk;
  const int64_t lt = xcd_tile(blockIdx.x, G);
  const int i = (int)(lt % nblk);
  const int64_t bh = lt / nblk;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int64_t tok_stride = (int64_t)H * D;     // elements between tokens
  const int64_t base_bh = (int64_t)b * N * tok_stride + (int64_t)h * D;

  const int q = i * BLOCK + 32 * w + l32;       // this lane's query row
  const int p0 = rowptr[lt], p1 = rowptr[lt + 1];
  const int T = (p1 - p0) * C::SUBS;            // sub-tiles to visit (uniform)

  if (T == 0) {  // empty S_i: O = 0, LSE = -inf
    if (q < N) {
      uint2 z = make_uint2(0, 0);
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
        for (int a = 0; a < 4; ++a)
          *reinterpret_cast<uint2*>(O + base_bh + q * tok_stride + 32 * dt + 8 * a + 4 * g) = z;
      if (g == 0) LSE[bh * N + q] = -INFINITY;
    }
    return;
  }

  // Q operand (B of S^T = K Q^T): lane holds Q[q][16 ks + 8 g .. +7].
  bf16x8 qop[C::KS];
  {
    const __bf16* qp = Q + base_bh + (int64_t)min(q, N - 1) * tok_stride + 8 * g;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) qop[ks] = *reinterpret_cast<const bf16x8*>(qp + 16 * ks);
  }

  // Staging: chunk x = tid + NT*u of the stage; tensor (K/V), row, chunk.
  u32x4 stg[C::LPT];
  auto load_stage = [&](int t) __attribute__((always_inline)) {
    const int j = cols[p0 + t / C::SUBS];
    const int key0 = j * BLOCK + (t % C::SUBS) * C::KT;
#pragma unroll
    for (int u = 0; u < C::LPT; ++u) {
      const int x = tid + C::NT * u;
      const int isv = x / (C::KT * C::CPR);
      const int r = (x / C::CPR) % C::KT, c = x % C::CPR;
      const int key = min(key0 + r, N - 1);
      const __bf16* src = (isv ? V : K) + base_bh + (int64_t)key * tok_stride + 8 * c;
      stg[u] = *reinterpret_cast<const u32x4*>(src);
    }
  };
  auto store_stage = [&](int s) __attribute__((always_inline)) {
    char* st = smem + s * C::STAGEB;
#pragma unroll
    for (int u = 0; u < C::LPT; ++u) {
      const int x = tid + C::NT * u;
      const int isv = x / (C::KT * C::CPR);
      const int r = (x / C::CPR) % C::KT, c = x % C::CPR;
      const int off = isv ? C::TILEB + lds_off<C::CPR>(r, c) : lds_off<C::CPR>(r, c);
      *reinterpret_cast<u32x4*>(st + off) = stg[u];
    }
  };

  const float c2 = scale * kLog2e;   // scores in log2 units
  f32x16 oacc[C::DT];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) oacc[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  load_stage(0);
  store_stage(0);
  __syncthreads();

  for (int t = 0; t < T; ++t) {
    const int cur = t & 1;
    if (t + 1 < T) load_stage(t + 1);
    const char* kt_lds = smem + cur * C::STAGEB;
    const char* vt_lds = kt_lds + C::TILEB;

    // ---- S^T = K Q^T over the 64 keys: two 32-key tiles
    f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(
            kt_lds + lds_off<C::CPR>(32 * kt + l32, 2 * ks + g));
        s[kt] = mfma32(a, qop[ks], s[kt]);
      }

    // ---- keys past N (only in a short last block) never count
    const int j = cols[p0 + t / C::SUBS];
    const int key0 = j * BLOCK + (t % C::SUBS) * C::KT;
    if (key0 + C::KT > N) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = key0 + 32 * kt + 8 * (e >> 2) + 4 * g + (e & 3);
          if (key >= N) s[kt][e] = -INFINITY;
        }
    }

    // ---- online softmax (lane owns query l32; its partner lane l^32 the other 16 keys)
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt][e]);
    mx = pair_max(mx);
    const float m_new = fmaxf(m_run, mx * c2);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);
    m_run = m_new;
    float lsum = 0.f;
    bf16x8 pb[2][2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = fast_exp2(__builtin_fmaf(s[kt][e], c2, -m_use));
        lsum += p;
        pb[kt][e >> 3][e & 7] = (__bf16)p;
      }
    l_run = l_run * alpha + lsum;
    if (__ballot(alpha != 1.f)) {
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt) oacc[dt] *= alpha;
    }

    // ---- O^T += V^T P^T: P^T tile kt, half hh covers keys 32kt + 16hh + {4g+0..3, 8+4g+0..3}
    {
      const int jr = lane & 15;                       // lane within a 16-lane group
      const int dsub = 16 * ((lane >> 4) & 1) + 4 * (jr & 3);
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int r0 = 32 * kt + 16 * hh + 4 * g + (jr >> 2);
            const int d = 32 * dt + dsub;
            const s16x4 lo = lds_read_tr16(vt_lds + lds_off<C::CPR>(r0, d >> 3) + 2 * (d & 7));
            const s16x4 hi = lds_read_tr16(vt_lds + lds_off<C::CPR>(r0 + 8, d >> 3) + 2 * (d & 7));
            const s16x8 v8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            oacc[dt] = mfma32(__builtin_bit_cast(bf16x8, v8), pb[kt][hh], oacc[dt]);
          }
    }

    if (t + 1 < T) store_stage(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: O = O^T / l, LSE = ln(sum) + max
  const float l_tot = pair_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (q < N) {
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        bf16x4 v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = (__bf16)(oacc[dt][4 * a + e] * inv);
        *reinterpret_cast<bf16x4*>(O + base_bh + q * tok_stride + 32 * dt + 8 * a + 4 * g) = v4;
      }
    if (g == 0) LSE[bh * N + q] = l_tot > 0.f ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

template <int D, int BLOCK>
hipError_t launch_fwd_t(const void* q, const void* k, const void* v, void* o, float* lse,
                        const AttnShape& sh, const int32_t* rowptr, const int32_t* cols,
                        hipStream_t s) {
  const int64_t G = (int64_t)sh.B * sh.H * sh.nblk;
  hipLaunchKernelGGL((bsattn_fwd_kernel<D, BLOCK>), dim3((unsigned)G), dim3(FwdCfg<D, BLOCK>::NT), 0,
                     s, static_cast<const __bf16*>(q), static_cast<const __bf16*>(k),
                     static_cast<const __bf16*>(v), static_cast<__bf16*>(o), lse, sh.B, sh.N, sh.H,
                     sh.nblk, sh.scale, rowptr, cols);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bsattn_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
                             const AttnShape& sh, const int32_t* rowptr, const int32_t* cols,
                             hipStream_t s) {
  if (sh.D == 128 && sh.block == 128) return launch_fwd_t<128, 128>(q, k, v, o, lse, sh, rowptr, cols, s);
  if (sh.D == 128 && sh.block == 64) return launch_fwd_t<128, 64>(q, k, v, o, lse, sh, rowptr, cols, s);
  if (sh.D == 64 && sh.block == 128) return launch_fwd_t<64, 128>(q, k, v, o, lse, sh, rowptr, cols, s);
  if (sh.D == 64 && sh.block == 64) return launch_fwd_t<64, 64>(q, k, v, o, lse, sh, rowptr, cols, s);
  return hipErrorInvalidValue;
}

}  // namespace ut
