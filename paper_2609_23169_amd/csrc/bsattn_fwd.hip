// Block-sparse attention forward on gfx950 (paper Sec. 3.3, Eq. 8): for each
// (batch, head, query block i), O_i = softmax(Q_i K_{S_i}^T * scale) V_{S_i}
// with an online softmax over the listed key blocks only; key blocks outside
// S_i are never read.
//
// One workgroup per (b, h, i); BLOCK/32 waves, each owning 32 query rows;
// two workgroups share a CU, so each SIMD runs two independent waves.
// Scores are formed transposed, S^T = K Q^T, with 32x32x16 bf16 MFMA: each
// lane holds one query column (16 keys per 32x32 tile), so row max and row
// sum are in-lane plus one permlane32 swap. The second product
// O^T += V^T P^T runs on 16x16x32 bf16 MFMA, the shape that draws less power
// per FLOP (under the board's power limit it holds a higher clock): one
// v_permlane16_swap per register moves the probabilities from the score
// layout (lane = one query, 16 keys) to the B-operand layout of two 16-query
// groups (lane = one query of each group, 8 keys), with the keys in an
// order whose V^T operand the transposing ds_read_b64_tr_b16 reads without
// bank conflicts. (The score product stays on 32x32x16: a forward with both
// products on 16x16x32, K in a conflict-free layout, held a higher clock but
// kept the matrix cores busy a smaller share of the time, and was slower.)
//
// The loop is built to spend as few vector instructions per MFMA as
// possible: at head_dim 128 the softmax's vector work per score once set the
// kernel's pace, and under the board's power limit every instruction costs
// clock:
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
  static constexpr int DT = D / 16;              // 16-wide d tiles of O
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
      const bf16x8 z = {};
#pragma unroll
      for (int dc = 0; dc < D / 16; ++dc)   // this lane: 8 columns of 16 per half
        *reinterpret_cast<bf16x8*>(O + base_bh + q * tok_stride + 16 * dc + 8 * g) = z;
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
  // V^T operand of the 16x16x32 product for d tile dt, key step kc (32
  // keys): lane group gq = lane / 16 reads rows 32 kc + base(gq) + (c16 >> 2)
  // (slots 0..3) and the same + 16 (slots 4..7), columns 16 dt + 4 (c16 & 3)
  // .. +3, base(gq) = 8 (gq & 1) + 4 (gq >> 1): the keys the P exchange
  // below leaves in that lane group. Rows 16 apart share the swizzle, so kc and
  // the +16 are immediates.
  const int c16 = lane & 15, gq = lane >> 4;
  int voff[C::DT];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) {
    const int d = 16 * dt + 4 * (c16 & 3);
    voff[dt] = lds_off<C::CPR>(8 * (gq & 1) + 4 * (gq >> 1) + (c16 >> 2), d >> 3) + 2 * (d & 7);
  }

  const float c2 = scale * kLog2e;   // scores in log2 units
  // O^T in the 16x16 layout: oacc[dt][qg] lane holds
  // O^T[16 dt + 4 gq + (0..3)][query 32 w + 16 qg + c16]
  f32x4 oacc[C::DT][2];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) oacc[dt][0] = oacc[dt][1] = f32x4{};
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
    // pq[kt][0]: elements 0-3, 8-11 (keys 32 kt + 4 g + {0..3, 16..19}),
    // pq[kt][1]: elements 4-7, 12-15 (keys 32 kt + 4 g + {8..11, 24..27}),
    // as bf16 pairs (elements e, e + 1 in one register)
    u32x4 pq[2][2];
    float lsum = 0.f;
    auto expo = [&]() __attribute__((always_inline)) {
      const float m_use = m_run == -INFINITY ? 0.f : m_run;
      lsum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
          const float p0 = fast_exp2(__builtin_fmaf(s[kt][e], c2, -m_use));
          const float p1 = fast_exp2(__builtin_fmaf(s[kt][e + 1], c2, -m_use));
          lsum += p0;
          lsum += p1;
          pq[kt][(e >> 2) & 1][((e & 3) >> 1) + 2 * (e >> 3)] = pack_bf16x2(p0, p1);
        }
    };
    // V^T operands of the second product, pair pp = (dt, kc) = (pp / 2,
    // pp % 2): the first kPre pairs are read here, so that their latency hides
    // behind the softmax; the rest are read kPre pairs ahead of their use.
    constexpr int kPairs = 2 * C::DT, kPre = 4;
    bf16x8 vop[kPre];
    auto read_v = [&](int pp) __attribute__((always_inline)) {
      const char* vb = vt_lds + 32 * (pp & 1) * C::ROWB + voff[pp >> 1];
      const s16x4 lo = lds_read_tr16(vb);
      const s16x4 hi = lds_read_tr16(vb + 16 * C::ROWB);
      const s16x8 v8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      return __builtin_bit_cast(bf16x8, v8);
    };
#pragma unroll
    for (int pp = 0; pp < kPre; ++pp) vop[pp] = read_v(pp);
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
      float alpha = 1.f;
      if (mx > m_run) {
        alpha = fast_exp2(m_run - mx);   // 0 on the first tile
        l_run *= alpha;
        m_run = mx;
      }
      // O^T columns are queries c16 (qg 0, held in the even 16-lane row of
      // each pair in the score layout) and 16 + c16 (qg 1, the odd row)
      const auto ar = __builtin_amdgcn_permlane16_swap(__float_as_uint(alpha),
                                                       __float_as_uint(alpha), false, false);
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt) {
        oacc[dt][0] *= __uint_as_float(ar[0]);
        oacc[dt][1] *= __uint_as_float(ar[1]);
      }
      expo();
    }
    l_run += lsum;
    // P^T to the B-operand layout of two 16-query groups: the swap leaves in
    // register 0 (qg 0) and 1 (qg 1) of 16-lane row gq the keys
    // 32 kt + base(gq) + {0..3, 16..19} of queries c16 and 16 + c16.
    bf16x8 pop[2][2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const u32x4 a = pq[kt][0], b = pq[kt][1];
      u32x4 na, nb;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const auto r = __builtin_amdgcn_permlane16_swap(a[v], b[v], false, false);
        na[v] = r[0];
        nb[v] = r[1];
      }
      pop[kt][0] = __builtin_bit_cast(bf16x8, na);
      pop[kt][1] = __builtin_bit_cast(bf16x8, nb);
    }
    // O^T += V^T P^T over the two 32-key steps, operands kPre pairs ahead
#pragma unroll
    for (int pp = 0; pp < kPairs; ++pp) {
      const bf16x8 av = vop[pp % kPre];
      if (pp + kPre < kPairs) vop[pp % kPre] = read_v(pp + kPre);
      oacc[pp >> 1][0] = mfma16(av, pop[pp & 1][0], oacc[pp >> 1][0]);
      oacc[pp >> 1][1] = mfma16(av, pop[pp & 1][1], oacc[pp >> 1][1]);
    }
    // keep that order: two products, then the two reads of a later pair
#pragma unroll
    for (int pp = 0; pp + kPre < kPairs; ++pp) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);   // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // DS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2 * kPre, 0);
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
  if (q < N && g == 0) LSE[sr.stat0 + q] = l_tot > 0.f ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
  // 1/l of queries c16 (qg 0) and 16 + c16 (qg 1) for the 16x16 layout
  const auto ir = __builtin_amdgcn_permlane16_swap(__float_as_uint(inv), __float_as_uint(inv),
                                                   false, false);
#pragma unroll
  for (int qg = 0; qg < 2; ++qg) {
    const int qo = i * BLOCK + 32 * w + 16 * qg + c16;
    const float iv = __uint_as_float(ir[qg]);
    if (qo < N) {
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt) {
        bf16x4 v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = (__bf16)(oacc[dt][qg][e] * iv);
        *reinterpret_cast<bf16x4*>(O + base_bh + qo * tok_stride + 16 * dt + 4 * gq) = v4;
      }
    }
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
  {
    TraceScope ts_(s, "bsattn_fwd", D, BLOCK);
    hipLaunchKernelGGL((bsattn_fwd_kernel<D, BLOCK>), grid, dim3(FwdCfg<D, BLOCK>::NT), 0,
                     s, static_cast<const __bf16*>(q), static_cast<const __bf16*>(k),
                     static_cast<const __bf16*>(v), static_cast<__bf16*>(o), lse, sh.B, sh.N, sh.H,
                     sh.nblk, sh.scale, rowptr, cols, sh.cu, sh.T);
  }
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
