// Block-sparse attention forward on gfx950 (paper Sec. 3.3, Eq. 8): for each
// (batch, head, query block i), O_i = softmax(Q_i K_{S_i}^T * scale) V_{S_i}
// with an online softmax over the listed key blocks only; key blocks outside
// S_i are never read.
//
// One workgroup per (b, h, i); BLOCK/32 waves, each owning 32 query rows;
// two workgroups share a CU, so each SIMD runs two independent waves.
// Scores are formed transposed, S^T = K Q^T, with 32x32x16 bf16 MFMA: each
// lane holds one query column (16 keys per 32x32 tile), so row max and row
// sum are in-lane plus one permlane32 swap, and the probabilities feed the
// second product O^T += V^T P^T straight from registers as the B operand.
// V^T operands come from LDS with the transposing ds_read_b64_tr_b16.
//
// The loop is built to spend as few vector instructions per MFMA as
// possible, since the vector ALU (softmax) and not the matrix core is the
// scarce resource at head_dim 128:
//  * K and V tiles (64 keys) go from global memory straight into LDS with
//    buffer loads; the tile base lives in the scalar buffer descriptor, so
//    the per-lane offsets are loop invariant, and rows past N fall outside
//    the descriptor's range and read as zeros;
//  * the loop is unrolled by two so that both LDS stages are at constant
//    offsets: every LDS read address is a precomputed lane offset plus an
//    immediate;
//  * no row max per tile: the exponentials use the running max set on the
//    first tile, and a new max is taken (O and the row sum rescaled, the tile
//    recomputed) only when a lane's tile sum exceeds 2^64 or is not finite,
//    which keeps every value far inside fp32 range. O and the row sum always
//    use the same max, so the result is exact in real arithmetic;
//  * only the sub-tiles of a short last key block run the masking code.
#include <type_traits>

#include "attn_util.h"
#include "common.h"

namespace ut {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kSumGuard = 18446744073709551616.0f;   // 2^64: per-lane tile sum bound

template <int D, int BLOCK>
struct FwdCfg {
  static constexpr int NW = BLOCK / 32;          // waves per workgroup
  static constexpr int NT = 64 * NW;             // threads
  static constexpr int KT = 64;                  // keys per sub-tile
  static constexpr int SUBS = BLOCK / KT;        // sub-tiles per key block
  static constexpr int ROWB = D * 2;             // bytes per LDS row
  static constexpr int CPR = D / 8;              // 16-byte chunks per row
  static constexpr int TILEB = KT * ROWB;        // one K or V sub-tile
  static constexpr int RPI = 1024 / ROWB;        // rows per direct-load instruction
  static constexpr int IPW = TILEB / 1024 / NW;  // direct-load instructions per wave per tile
  static constexpr int KS = D / 16;              // k-steps of the score product
  static constexpr int DT = D / 32;              // 32-wide d tiles of O
  static_assert(TILEB % (1024 * NW) == 0, "tile must split evenly over the waves");
};

template <int D, int BLOCK>
__global__ __launch_bounds__(64 * (BLOCK / 32), (BLOCK == 128 || D == 64) ? 2 : 1) void bsattn_fwd_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    __bf16* __restrict__ O, float* __restrict__ LSE, int B, int N_all, int H, int nblk, float scale,
    const int32_t* __restrict__ rowptr, const int32_t* __restrict__ cols,
    const int32_t* __restrict__ cu_seqlens, int64_t T_tok) {
  using C = FwdCfg<D, BLOCK>;
  // Four LDS objects (K and V, two stages each): distinct objects let the
  // compiler see that a load into one never aliases reads of another.
  __shared__ __attribute__((aligned(1024))) char k_lds0[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char k_lds1[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char v_lds0[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char v_lds1[C::TILEB];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index, uniform
  const int l32 = lane & 31, g = lane >> 5;
  const int64_t lt = blockIdx.x;   // tile order: see the launcher
  const int i = (int)(lt % nblk);
  const int64_t bh = lt / nblk;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int64_t tok_stride = (int64_t)H * D;     // elements between tokens
  const SampleRows sr = sample_rows(cu_seqlens, T_tok, b, h, H, N_all);
  const int N = sr.n;                            // this sample's tokens
  if (N <= 0 || i * BLOCK >= N) return;         // no query rows of this sample here
  const int64_t base_bh = sr.tok0 * tok_stride + (int64_t)h * D;

  const int q = i * BLOCK + 32 * w + l32;       // this lane's query row
  const int p0 = rowptr[lt];
  int p1 = rowptr[lt + 1];
  // entries past the sample's last key block (possible only with variable
  // lengths, where the block grid is sized for the longest) are ignored
  while (p1 > p0 && cols[p1 - 1] >= (N + BLOCK - 1) / BLOCK) --p1;
  const int T = (p1 - p0) * C::SUBS;            // sub-tiles to visit (uniform)

  if (T == 0) {  // empty S_i: O = 0, LSE = -inf
    if (q < N) {
      const bf16x4 z = {};
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
        for (int a = 0; a < 4; ++a)
          *reinterpret_cast<bf16x4*>(O + base_bh + q * tok_stride + 32 * dt + 8 * a + 4 * g) = z;
      if (g == 0) LSE[sr.stat0 + q] = -INFINITY;
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

  // Loop-invariant lane offsets. Direct loads: lane L of instruction u writes
  // 16 bytes at dst + 1024 (w IPW + u) + 16 L, i.e. row r, physical chunk
  // p = L mod CPR, which holds logical chunk p ^ swizzle(r); it reads that
  // chunk of key row r of the tile.
  int dma_off[C::IPW];
#pragma unroll
  for (int u = 0; u < C::IPW; ++u) {
    const int r = (w * C::IPW + u) * C::RPI + lane / C::CPR, p = lane % C::CPR;
    const int c = (lds_off<C::CPR>(r, p) >> 4) & (C::CPR - 1);
    dma_off[u] = r * (int)(tok_stride * 2) + 16 * c;
  }
  // Tile t of X (K or V) into `dst`: descriptor base at the tile's first key,
  // range ending after the last valid key row (rows past N read zeros).
  auto load_tile = [&](const __bf16* X, int t, char* dst) __attribute__((always_inline)) {
    const int j = cols[p0 + t / C::SUBS];
    const int key0 = j * BLOCK + (t % C::SUBS) * C::KT;
    const __bf16* tile = X + base_bh + (int64_t)key0 * tok_stride;
    // a sub-tile wholly past N (second half of a short last block) gets an
    // empty range: every load reads zeros and nothing past the tensor is touched
    const int nrec = key0 < N ? (N - key0 - 1) * (int)(tok_stride * 2) + 2 * D : 0;
    const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(tile, nrec);
#pragma unroll
    for (int u = 0; u < C::IPW; ++u)
      buffer_load_lds16(rs, dst + (w * C::IPW + u) * 1024, dma_off[u]);
  };

  // LDS lane offsets of the two products (immediates add kt, hh and stage).
  int koff[C::KS];
#pragma unroll
  for (int ks = 0; ks < C::KS; ++ks) koff[ks] = lds_off<C::CPR>(l32, 2 * ks + g);
  const int jr = lane & 15;
  const int dsub = 16 * ((lane >> 4) & 1) + 4 * (jr & 3);
  int voff[C::DT][2];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
    for (int lh = 0; lh < 2; ++lh) {
      const int r0 = 4 * g + (jr >> 2) + 8 * lh;
      const int d = 32 * dt + dsub;
      voff[dt][lh] = lds_off<C::CPR>(r0, d >> 3) + 2 * (d & 7);
    }

  const float c2 = scale * kLog2e;   // scores in log2 units
  f32x16 oacc[C::DT];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) oacc[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  // One sub-tile: S^T = K Q^T, online softmax, O^T += V^T P^T. Rows 32 kt + l32
  // and 32 kt + 16 hh + r of a tile share the swizzle of rows l32 and r (the
  // swizzle depends on the row mod 16), so kt and hh are pure immediates.
  auto step = [&](int t, const char* kt_lds, const char* vt_lds, auto masked)
      __attribute__((always_inline)) {
    f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const bf16x8 av = *reinterpret_cast<const bf16x8*>(kt_lds + koff[ks] + kt * 32 * C::ROWB);
        s[kt] = mfma32(av, qop[ks], s[kt]);
      }
    if constexpr (decltype(masked)::value) {   // keys past N in a short last block
      const int j = cols[p0 + t / C::SUBS];
      const int lim = N - (j * BLOCK + (t % C::SUBS) * C::KT);
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          s[kt][e] = 32 * kt + 8 * (e >> 2) + 4 * g + (e & 3) >= lim ? -INFINITY : s[kt][e];
    }
    // Exponentials against the running max; the max itself is taken only on
    // the first tile or when a tile's sum leaves the guard (rare).
    bf16x8 pb[2][2];
    float lsum = 0.f;
    auto expo = [&]() __attribute__((always_inline)) {
      const float m_use = m_run == -INFINITY ? 0.f : m_run;
      lsum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = fast_exp2(__builtin_fmaf(s[kt][e], c2, -m_use));
          lsum += p;
          pb[kt][e >> 3][e & 7] = (__bf16)p;
        }
    };
    bool redo = __ballot(m_run == -INFINITY) != 0;
    if (!redo) {
      expo();
      redo = __ballot(!(lsum <= kSumGuard)) != 0;   // also catches inf and NaN
    }
    if (redo) {
      float mx = s[0][0];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = (kt == 0 ? 1 : 0); e < 16; ++e) mx = fmaxf(mx, s[kt][e]);
      mx = pair_max(mx) * c2;
      if (mx > m_run) {
        const float alpha = fast_exp2(m_run - mx);   // 0 on the first tile
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt) oacc[dt] *= alpha;
        m_run = mx;
      }
      expo();
    }
    l_run += lsum;
    // O^T += V^T P^T: P^T tile kt, half hh covers keys 32kt + 16hh + {4g+0..3, 8+4g+0..3}
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const char* vb = vt_lds + (32 * kt + 16 * hh) * C::ROWB;
          const s16x4 lo = lds_read_tr16(vb + voff[dt][0]);
          const s16x4 hi = lds_read_tr16(vb + voff[dt][1]);
          const s16x8 v8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          oacc[dt] = mfma32(__builtin_bit_cast(bf16x8, v8), pb[kt][hh], oacc[dt]);
        }
  };

  // Iteration t: issue the loads of tile t+1 into the other stage (read in
  // iteration t-1, before the last barrier), compute tile t, wait for the
  // new tile and barrier.
  auto iter = [&](int t, auto par, auto masked) __attribute__((always_inline)) {
    constexpr int P = decltype(par)::value;
    char* const kc = P ? k_lds1 : k_lds0;
    char* const vc = P ? v_lds1 : v_lds0;
    char* const kn = P ? k_lds0 : k_lds1;
    char* const vn = P ? v_lds0 : v_lds1;
    if (t + 1 < T) {
      load_tile(K, t + 1, kn);
      load_tile(V, t + 1, vn);
    }
    step(t, kc, vc, masked);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };

  load_tile(K, 0, k_lds0);
  load_tile(V, 0, v_lds0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // The sub-tiles of a short last key block (always the end of the ascending
  // list) take the masked path.
  const bool tail = (N % BLOCK != 0) && cols[p1 - 1] == (N + BLOCK - 1) / BLOCK - 1;
  const int Tm = tail ? T - C::SUBS : T;
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using F = std::false_type;
  using Tt = std::true_type;
  int t = 0;
  for (; t + 1 < Tm; t += 2) {
    iter(t, I0{}, F{});
    iter(t + 1, I1{}, F{});
  }
  if (t < Tm) {   // one unmasked step left at parity 0; masked steps continue at parity 1
    iter(t, I0{}, F{});
    for (++t; t < T; t += 2) {
      iter(t, I1{}, Tt{});
      if (t + 1 < T) iter(t + 1, I0{}, Tt{});
    }
  } else {        // masked steps from parity 0
    for (; t < T; t += 2) {
      iter(t, I0{}, Tt{});
      if (t + 1 < T) iter(t + 1, I1{}, Tt{});
    }
  }

  // ---- epilogue: O = O^T / l, LSE = (m + log2 l) ln 2
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
    if (g == 0) LSE[sr.stat0 + q] = l_tot > 0.f ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

template <int D, int BLOCK>
hipError_t launch_fwd_t(const void* q, const void* k, const void* v, void* o, float* lse,
                        const AttnShape& sh, const int32_t* rowptr, const int32_t* cols,
                        hipStream_t s) {
  // One workgroup per (b, h, block) in plain order. Workgroups go round-robin
  // to the 8 XCDs, so all XCDs work on the same few heads at once (their K and
  // V stay in the shared last-level cache) and a run of heavy blocks is spread
  // over every XCD.
  const dim3 grid((unsigned)((int64_t)sh.B * sh.H * sh.nblk));
  hipLaunchKernelGGL((bsattn_fwd_kernel<D, BLOCK>), grid, dim3(FwdCfg<D, BLOCK>::NT), 0,
                     s, static_cast<const __bf16*>(q), static_cast<const __bf16*>(k),
                     static_cast<const __bf16*>(v), static_cast<__bf16*>(o), lse, sh.B, sh.N, sh.H,
                     sh.nblk, sh.scale, rowptr, cols, sh.cu, sh.T);
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
