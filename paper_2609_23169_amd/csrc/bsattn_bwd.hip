// Block-sparse attention backward on gfx950: gradients of Eq. 8 (paper
// Sec. 3.3) with the block mask held constant. No atomics, deterministic.
// Three launches with the minimum workspace (five when it holds dS tiles,
// below):
//
//   prep  : per query row, LSE log2(e) and -delta = -sum_d dO[r,d] O[r,d]
//           (fp32, two planes of the workspace);
//   dQ    : one workgroup per (b, h, query block i), walking S_i (row lists).
//           Each wave owns 32 queries, with its Q and dO rows as MFMA operands
//           in registers. Per 64-key tile streamed through LDS:
//           S^T = K Q^T and dP^T = V dO^T (lane = query column, 32x32x16),
//           P = exp(S - LSE), dS^T = P^T o (dP^T - delta), then
//           dQ^T += K^T dS^T on 16x16x32 MFMA after one v_permlane16_swap per
//           register moves dS^T to the B-operand layout (as the forward does
//           for P; the smaller shape draws less power per FLOP);
//   dK/dV : one workgroup per (b, h, key block j), walking the query blocks
//           that select j (column lists) in 32-row query tiles. One wave per
//           32 keys (K rows in registers, the key block's V rows in LDS):
//           S = Q K^T and dP = dO V^T (lane = key column, 32x32x16; the dP
//           accumulator starts at -delta, so it ends as dP - delta), then
//           dV^T += dO^T P and dK^T += Q^T dS on 16x16x32 after a
//           v_permlane16_swap exchange of P and dS, with transposing LDS
//           reads. Two workgroups share a
//           CU, so the two waves on each SIMD belong to different workgroups
//           and never wait at the same barrier.
//
//   dQ from stored dS (when the workspace holds the tiles): the dK/dV pass
//           also writes each retained pair's bf16 dS tile, at the pair's
//           column-list position, and this pass takes dQ^T += K^T dS^T from
//           it: one product per pair instead of three. A map pass, first,
//           gives each row-list entry its tile and flags the query blocks whose
//           tiles all fit in the workspace; the others keep the recompute pass
//           above.
//
// Without stored tiles the dQ pass recomputes S and dP instead of accumulating
// dQ with atomics from the dK/dV pass. Tiles go from global memory straight into LDS with
// buffer loads; rows past N are outside the descriptor range and read as
// zeros. For query rows past N that makes every contribution exactly zero
// (zero Q and dO rows give dP = 0 and delta = 0, hence dS = 0 and P dO = 0).
// Keys past N are masked explicitly in the dQ pass (their P would not be 0).
#include <mutex>
#include <type_traits>

#include "attn_util.h"
#include "common.h"

namespace ut {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// prep: two planes over the statistics rows, in the layout of LSE ([B, H, N]
// for a uniform batch, [H, T] over packed tokens otherwise):
//   A[r] = LSE log2 e,   Dn[r] = -delta = -rowsum(dO o O)
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_prep_kernel(const __bf16* __restrict__ O,
                                                       const __bf16* __restrict__ dO,
                                                       const float* __restrict__ LSE,
                                                       float* __restrict__ aux, int64_t T_tok,
                                                       int N, int H, bool packed) {
  constexpr int CPR = D / 8;  // lanes per (token, head) row
  const int64_t rows = T_tok * H;
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
    const int64_t tok = row / H;
    const int64_t r = packed ? (int64_t)h * T_tok + tok
                             : ((tok / N) * H + h) * N + tok % N;
    aux[r] = LSE[r] * kLog2e;
    aux[rows + r] = -acc;
  }
}

template <int D, int BLOCK, int NWAVES, int ST_ = 64>
struct BwdCfg {
  static constexpr int NT = 64 * NWAVES;
  static constexpr int ST = ST_;                 // rows per streamed tile
  static constexpr int SUBS = BLOCK / ST;        // tiles per block
  static constexpr int ROWB = D * 2;
  static constexpr int CPR = D / 8;
  static constexpr int TILEB = ST * ROWB;        // one ST-row bf16 tile
  static constexpr int RPI = 1024 / ROWB;        // rows per direct-load instruction
  static constexpr int IPW = TILEB / 1024 / NWAVES;
  static constexpr int KS = D / 16;
  static constexpr int DT = D / 32;
  static_assert(TILEB % (1024 * NWAVES) == 0, "tile must split evenly over the waves");
};

// Loop-invariant lane offsets shared by both passes.
template <class C>
struct LaneOffsets {
  int dma[C::IPW];      // global byte offset of this lane's 16-byte chunk within a tile
  int row[C::KS];       // LDS: b128 read of row l32, chunk 2 ks + g
  int tr[C::DT][2];     // LDS: transposing read, rows 4g + (jr >> 2) (+8), columns of d tile
  __device__ inline LaneOffsets(int w, int lane, int64_t tok_stride) {
    const int l32 = lane & 31, g = lane >> 5, jr = lane & 15;
#pragma unroll
    for (int u = 0; u < C::IPW; ++u) {
      const int r = (w * C::IPW + u) * C::RPI + lane / C::CPR, p = lane % C::CPR;
      const int c = (lds_off<C::CPR>(r, p) >> 4) & (C::CPR - 1);
      dma[u] = r * (int)(tok_stride * 2) + 16 * c;
    }
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) row[ks] = lds_off<C::CPR>(l32, 2 * ks + g);
    const int dsub = 16 * ((lane >> 4) & 1) + 4 * (jr & 3);
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
      for (int lh = 0; lh < 2; ++lh) {
        const int d = 32 * dt + dsub;
        tr[dt][lh] = lds_off<C::CPR>(4 * g + (jr >> 2) + 8 * lh, d >> 3) + 2 * (d & 7);
      }
  }
};

// ---------------------------------------------------------------------------
// map: for row-list entry p (pair (i, j) of query block row r) the column-list
// position e of the same pair, which indexes its dS tile, by a binary search
// of column j's ascending list for i; and row_ok[r] = 1 when every tile of the
// row lies below max_pairs (its dQ then comes from the tiles). One wave per
// query block row; entries at or past max_pairs get no map entry.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void bwd_ds_map_kernel(
    const int32_t* __restrict__ rowptr, const int32_t* __restrict__ cols,
    const int32_t* __restrict__ colptr, const int32_t* __restrict__ rows_list, int nblk,
    int64_t max_pairs, int32_t* __restrict__ map, int32_t* __restrict__ row_ok) {
  const int64_t r = blockIdx.x;
  const int i = (int)(r % nblk);
  const int64_t cbase = r - i;   // (b, h) * nblk
  const int p0 = rowptr[r], p1 = rowptr[r + 1];
  bool ok = (int64_t)p1 <= max_pairs;
  for (int p = p0 + (int)threadIdx.x; p < p1 && (int64_t)p < max_pairs; p += 64) {
    const int j = cols[p];
    int e = -1;
    if (j >= 0 && j < nblk) {
      const int lo0 = colptr[cbase + j], hi0 = colptr[cbase + j + 1];
      int lo = lo0, hi = hi0;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (rows_list[mid] < i) lo = mid + 1;
        else hi = mid;
      }
      if (lo < hi0 && rows_list[lo] == i) e = lo;
    }
    map[p] = e;
    ok = ok && e >= 0 && (int64_t)e < max_pairs;
  }
  ok = __all(ok);
  if (threadIdx.x == 0) row_ok[r] = ok ? 1 : 0;
}

// ---------------------------------------------------------------------------
// dQ: query-stationary over the row lists
// ---------------------------------------------------------------------------
template <int D, int BLOCK>
__global__ __launch_bounds__(64 * (BLOCK / 32), (BLOCK == 128 || D == 64) ? 2 : 1) void bwd_dq_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const __bf16* __restrict__ dO, const float* __restrict__ aux, __bf16* __restrict__ dQ, int B,
    int N_all, int H, int nblk, float scale, const int32_t* __restrict__ rowptr,
    const int32_t* __restrict__ cols, const int32_t* __restrict__ cu_seqlens, int64_t T_tok,
    const int32_t* __restrict__ row_ok) {
  using C = BwdCfg<D, BLOCK, BLOCK / 32>;
  __shared__ __attribute__((aligned(1024))) char k_lds0[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char k_lds1[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char v_lds0[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char v_lds1[C::TILEB];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  const int64_t lt = blockIdx.x;   // tile order: see the launcher
  if (row_ok && row_ok[lt]) return;   // dQ comes from the stored dS tiles
  const int i = (int)(lt % nblk);
  const int64_t bh = lt / nblk;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int64_t tok_stride = (int64_t)H * D;
  const SampleRows sr = sample_rows(cu_seqlens, T_tok, b, h, H, N_all);
  const int N = sr.n;
  if (N <= 0 || i * BLOCK >= N) return;
  const int64_t base_bh = sr.tok0 * tok_stride + (int64_t)h * D;
  const int q = i * BLOCK + 32 * w + l32;
  const int p0 = rowptr[lt];
  int p1 = rowptr[lt + 1];
  while (p1 > p0 && cols[p1 - 1] >= (N + BLOCK - 1) / BLOCK) --p1;   // past the sample
  const int T = (p1 - p0) * C::SUBS;

  // dQ^T in the 16x16 layout: dq16[dt][qg] lane holds
  // dQ^T[16 dt + 4 gq + (0..3)][query 32 w + 16 qg + c16]
  constexpr int DT16 = D / 16;
  const int c16 = lane & 15, gq = lane >> 4;
  f32x4 dq16[DT16][2];
#pragma unroll
  for (int dt = 0; dt < DT16; ++dt) dq16[dt][0] = dq16[dt][1] = f32x4{};

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
    const int64_t ar = sr.stat0 + min(q, N - 1);
    const float lse2 = aux[ar], ndl = aux[(int64_t)H * T_tok + ar];   // LSE log2 e, -delta
    const LaneOffsets<C> lo(w, lane, tok_stride);
    // K^T operand of the 16x16x32 dQ product for d tile dt, key step kc:
    // lane group gq reads key rows 32 kc + base(gq) + (c16 >> 2) (slots
    // 0..3) and the same + 16 (slots 4..7), columns 16 dt + 4 (c16 & 3) .. +3,
    // base(gq) = 8 (gq & 1) + 4 (gq >> 1): the keys the dS exchange leaves in
    // that lane group.
    int ktr[DT16];
#pragma unroll
    for (int dt = 0; dt < DT16; ++dt) {
      const int d = 16 * dt + 4 * (c16 & 3);
      ktr[dt] = lds_off<C::CPR>(8 * (gq & 1) + 4 * (gq >> 1) + (c16 >> 2), d >> 3) + 2 * (d & 7);
    }

    auto load_tile = [&](const __bf16* X, int t, char* dst) __attribute__((always_inline)) {
      const int j = cols[p0 + t / C::SUBS];
      const int key0 = j * BLOCK + (t % C::SUBS) * C::ST;
      const int nrec = key0 < N ? (N - key0 - 1) * (int)(tok_stride * 2) + 2 * D : 0;
      const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(X + base_bh + (int64_t)key0 * tok_stride, nrec);
#pragma unroll
      for (int u = 0; u < C::IPW; ++u) buffer_load_lds16(rs, dst + (w * C::IPW + u) * 1024, lo.dma[u]);
    };
    const float c2 = scale * kLog2e;

    // One 64-key tile as two 32-key halves kt: S^T and dP^T (32x32x16), dS^T,
    // its exchange to the 16x16 B-operand layout, and the dQ product of that
    // half (16x16x32); only one half's score accumulators are live at a time.
    auto step = [&](int t, const char* kt_lds, const char* vt_lds, auto masked)
        __attribute__((always_inline)) {
      int lim = 2 * C::ST;
      if constexpr (decltype(masked)::value) {   // keys past N in a short last block
        const int j = cols[p0 + t / C::SUBS];
        lim = N - (j * BLOCK + (t % C::SUBS) * C::ST);
      }
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) {
          const int off = lo.row[ks] + kt * 32 * C::ROWB;
          s = mfma32(*reinterpret_cast<const bf16x8*>(kt_lds + off), qop[ks], s);
          dp = mfma32(*reinterpret_cast<const bf16x8*>(vt_lds + off), doop[ks], dp);
        }
        // dS^T as bf16 pairs: pq[0] holds elements 0-3, 8-11 (keys
        // 32 kt + 4 g + {0..3, 16..19}), pq[1] elements 4-7, 12-15
        u32x4 pq[2];
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
          float p0 = fast_exp2(__builtin_fmaf(s[e], c2, -lse2));
          float p1 = fast_exp2(__builtin_fmaf(s[e + 1], c2, -lse2));
          if constexpr (decltype(masked)::value) {
            const int key = 32 * kt + 8 * (e >> 2) + 4 * g + (e & 3);
            p0 = key >= lim ? 0.f : p0;
            p1 = key + 1 >= lim ? 0.f : p1;
          }
          pq[(e >> 2) & 1][((e & 3) >> 1) + 2 * (e >> 3)] =
              pack_bf16x2(p0 * (dp[e] + ndl), p1 * (dp[e + 1] + ndl));
        }
        // to the B-operand layout of two 16-query groups (as the forward
        // does for P): register 0 serves queries c16, register 1 16 + c16
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const auto r = __builtin_amdgcn_permlane16_swap(pq[0][v], pq[1][v], false, false);
          pq[0][v] = r[0];
          pq[1][v] = r[1];
        }
        // dQ^T += K^T dS^T over this half's 32 keys
#pragma unroll
        for (int dt = 0; dt < DT16; ++dt) {
          const char* kb = kt_lds + 32 * kt * C::ROWB + ktr[dt];
          const s16x4 l4 = lds_read_tr16(kb);
          const s16x4 h4 = lds_read_tr16(kb + 16 * C::ROWB);
          const s16x8 k8 = {l4[0], l4[1], l4[2], l4[3], h4[0], h4[1], h4[2], h4[3]};
          const bf16x8 av = __builtin_bit_cast(bf16x8, k8);
          dq16[dt][0] = mfma16(av, __builtin_bit_cast(bf16x8, pq[0]), dq16[dt][0]);
          dq16[dt][1] = mfma16(av, __builtin_bit_cast(bf16x8, pq[1]), dq16[dt][1]);
        }
      }
    };
    auto iter = [&](int t, auto par, auto masked) __attribute__((always_inline)) {
      constexpr int P = decltype(par)::value;
      if (t + 1 < T) {
        load_tile(K, t + 1, P ? k_lds0 : k_lds1);
        load_tile(V, t + 1, P ? v_lds0 : v_lds1);
      }
      step(t, P ? k_lds1 : k_lds0, P ? v_lds1 : v_lds0, masked);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
    };

    load_tile(K, 0, k_lds0);
    load_tile(V, 0, v_lds0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
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
    if (t < Tm) {
      iter(t, I0{}, F{});
      for (++t; t < T; t += 2) {
        iter(t, I1{}, Tt{});
        if (t + 1 < T) iter(t + 1, I0{}, Tt{});
      }
    } else {
      for (; t < T; t += 2) {
        iter(t, I0{}, Tt{});
        if (t + 1 < T) iter(t + 1, I1{}, Tt{});
      }
    }
  }

#pragma unroll
  for (int qg = 0; qg < 2; ++qg) {
    const int qo = i * BLOCK + 32 * w + 16 * qg + c16;
    if (qo >= N) continue;
    const int64_t off = base_bh + (int64_t)qo * tok_stride;
#pragma unroll
    for (int dt = 0; dt < DT16; ++dt) {
      bf16x4 v4;
#pragma unroll
      for (int e = 0; e < 4; ++e) v4[e] = (__bf16)(dq16[dt][qg][e] * scale);
      *reinterpret_cast<bf16x4*>(dQ + off + 16 * dt + 4 * gq) = v4;
    }
  }
}

// ---------------------------------------------------------------------------
// dQ from the stored dS tiles: query-stationary over the row lists like the
// recompute pass, one product per pair. Wave w owns queries 32 w .. 32 w + 31
// of block i; per 64-key tile it takes the tile's K rows (shared, in LDS) and
// its own two 2 KB dS chunks (32 queries x 32 keys each, streamed into LDS by
// each wave for itself), and accumulates dQ^T += K^T dS^T on 16x16x32 with
// both operands from transposing LDS reads. Query blocks without row_ok are
// left to the recompute pass; for the others map[p] < max_pairs is the tile of
// every entry p.
// ---------------------------------------------------------------------------
template <int D, int BLOCK>
__global__ __launch_bounds__(64 * (BLOCK / 32), 2) void bwd_dq_stored_kernel(
    const __bf16* __restrict__ K, const char* __restrict__ ds, __bf16* __restrict__ dQ,
    int N_all, int H, int nblk, float scale, const int32_t* __restrict__ rowptr,
    const int32_t* __restrict__ cols, const int32_t* __restrict__ cu_seqlens, int64_t T_tok,
    const int32_t* __restrict__ map, const int32_t* __restrict__ row_ok) {
  constexpr int NW = BLOCK / 32;
  using C = BwdCfg<D, BLOCK, NW>;
  constexpr int PAIRB = 2 * BLOCK * BLOCK;   // one pair's dS tile
  constexpr int WSB = 2 * 2048;              // one wave's dS chunks of one 64-key tile
  __shared__ __attribute__((aligned(1024))) char k_lds0[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char k_lds1[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char s_lds0[NW * WSB];
  __shared__ __attribute__((aligned(1024))) char s_lds1[NW * WSB];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t lt = blockIdx.x;
  if (!row_ok[lt]) return;   // not all stored: the recompute pass takes it
  const int p0 = rowptr[lt], pe = rowptr[lt + 1];
  const int i = (int)(lt % nblk);
  const int64_t bh = lt / nblk;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int64_t tok_stride = (int64_t)H * D;
  const SampleRows sr = sample_rows(cu_seqlens, T_tok, b, h, H, N_all);
  const int N = sr.n;
  if (N <= 0 || i * BLOCK >= N) return;
  const int64_t base_bh = sr.tok0 * tok_stride + (int64_t)h * D;
  int p1 = pe;
  while (p1 > p0 && cols[p1 - 1] >= (N + BLOCK - 1) / BLOCK) --p1;   // past the sample
  const int T = (p1 - p0) * C::SUBS;

  constexpr int DT16 = D / 16;
  const int c16 = lane & 15, gq = lane >> 4;
  f32x4 dq16[DT16][2];
#pragma unroll
  for (int dt = 0; dt < DT16; ++dt) dq16[dt][0] = dq16[dt][1] = f32x4{};

  if (T > 0) {
    const LaneOffsets<C> lo(w, lane, tok_stride);
    // K^T operand for d tile dt: key rows base(gq) + (c16 >> 2) (slots 0..3)
    // and the same + 16 (slots 4..7), base(gq) = 8 (gq & 1) + 4 (gq >> 1).
    int ktr[DT16];
#pragma unroll
    for (int dt = 0; dt < DT16; ++dt) {
      const int d = 16 * dt + 4 * (c16 & 3);
      ktr[dt] = lds_off<C::CPR>(8 * (gq & 1) + 4 * (gq >> 1) + (c16 >> 2), d >> 3) + 2 * (d & 7);
    }
    // dS^T operand with the same key slots: lane c16 of group gq reads key
    // base(gq) + (c16 >> 2) (+16 for slots 4..7) at queries 16 qg + 4 u .. +3,
    // u = c16 & 3, which the storing lane (gs, cs) holds: base(gs) = 4 u,
    // cs = the key within its 16.
    const int u = c16 & 3;
    const int gs = ((u & 1) << 1) | (u >> 1);
    const int cs = 8 * (gq & 1) + 4 * (gq >> 1) + (c16 >> 2);
    const int sb = w * WSB + 16 * (16 * gs + (cs ^ (4 * (gs & 1))));

    auto load_k = [&](int t, char* kdst) __attribute__((always_inline)) {
      const int p = p0 + t / C::SUBS, hh = t % C::SUBS;
      const int key0 = cols[p] * BLOCK + hh * C::ST;
      const int nrec = key0 < N ? (N - key0 - 1) * (int)(tok_stride * 2) + 2 * D : 0;
      const __amdgpu_buffer_rsrc_t rk = buffer_rsrc(K + base_bh + (int64_t)key0 * tok_stride, nrec);
#pragma unroll
      for (int v = 0; v < C::IPW; ++v) buffer_load_lds16(rk, kdst + (w * C::IPW + v) * 1024, lo.dma[v]);
    };
    // this wave's two dS chunks of tile t, into its own part of the buffer
    auto load_s = [&](int t, char* sdst) __attribute__((always_inline)) {
      const int p = p0 + t / C::SUBS, hh = t % C::SUBS;
      const __amdgpu_buffer_rsrc_t rs =
          buffer_rsrc(ds + (int64_t)map[p] * PAIRB + (w * NW + 2 * hh) * 2048, WSB);
#pragma unroll
      for (int v = 0; v < WSB / 1024; ++v)
        buffer_load_lds16(rs, sdst + w * WSB + v * 1024, v * 1024 + 16 * lane);
    };

    auto step = [&](const char* kt_lds, const char* st_lds) __attribute__((always_inline)) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {   // 32-key halves: one dS chunk each
        bf16x8 bq[2];
#pragma unroll
        for (int qg = 0; qg < 2; ++qg) {
          const char* sp = st_lds + sb + kt * 2048 + qg * 1024;
          const s16x4 l4 = lds_read_tr16(sp);
          const s16x4 h4 = lds_read_tr16(sp + 8);
          const s16x8 s8 = {l4[0], l4[1], l4[2], l4[3], h4[0], h4[1], h4[2], h4[3]};
          bq[qg] = __builtin_bit_cast(bf16x8, s8);
        }
#pragma unroll
        for (int dt = 0; dt < DT16; ++dt) {
          const char* kb = kt_lds + 32 * kt * C::ROWB + ktr[dt];
          const s16x4 l4 = lds_read_tr16(kb);
          const s16x4 h4 = lds_read_tr16(kb + 16 * C::ROWB);
          const s16x8 k8 = {l4[0], l4[1], l4[2], l4[3], h4[0], h4[1], h4[2], h4[3]};
          const bf16x8 av = __builtin_bit_cast(bf16x8, k8);
          dq16[dt][0] = mfma16(av, bq[0], dq16[dt][0]);
          dq16[dt][1] = mfma16(av, bq[1], dq16[dt][1]);
        }
      }
    };
    auto iter = [&](int t, auto par) __attribute__((always_inline)) {
      constexpr int P = decltype(par)::value;
      if (t + 1 < T) {
        load_k(t + 1, P ? k_lds0 : k_lds1);
        load_s(t + 1, P ? s_lds0 : s_lds1);
      }
      // keep the loads ahead of this tile's work (the scheduler would sink them
      // to the wait at its end, exposing their latency)
      __builtin_amdgcn_sched_barrier(0);
      step(P ? k_lds1 : k_lds0, P ? s_lds1 : s_lds0);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
    };

    load_k(0, k_lds0);
    load_s(0, s_lds0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    int t = 0;
    for (; t + 1 < T; t += 2) {
      iter(t, I0{});
      iter(t + 1, I1{});
    }
    if (t < T) iter(t, I0{});
  }

#pragma unroll
  for (int qg = 0; qg < 2; ++qg) {
    const int qo = i * BLOCK + 32 * w + 16 * qg + c16;
    if (qo >= N) continue;
    const int64_t off = base_bh + (int64_t)qo * tok_stride;
#pragma unroll
    for (int dt = 0; dt < DT16; ++dt) {
      bf16x4 v4;
#pragma unroll
      for (int e = 0; e < 4; ++e) v4[e] = (__bf16)(dq16[dt][qg][e] * scale);
      *reinterpret_cast<bf16x4*>(dQ + off + 16 * dt + 4 * gq) = v4;
    }
  }
}

// ---------------------------------------------------------------------------
// dK, dV: key-stationary over the column lists, one wave per 32 keys
// ---------------------------------------------------------------------------
// With STORE, the pass also writes each pair's dS as bf16 into `ds` at the
// pair's column-list position e (tiles of pairs e >= max_pairs are not written):
// 2 BLOCK^2 bytes per pair, as (BLOCK/32)^2 chunks of 2 KB, chunk
// (query tile, key group) holding dS for 32 queries x 32 keys. Within a
// chunk, the lane (gq, c16) that holds keys c16 and 16 + c16 after the
// exchange stores, at 16-byte unit 16 gq + (c16 ^ 4 (gq & 1)) of half x, its
// four queries base(gq) + 16 x + (0..3) for key c16 and then for key
// 16 + c16. Each store instruction writes 1 KB contiguously; the dQ pass
// reads the chunk back with transposing LDS reads.
// At every block size the kernel is built for two waves per SIMD (the launch
// bound's second argument): up to 256 VGPRs per wave.
template <int D, int BLOCK, bool STORE>
__global__ __launch_bounds__(64 * (BLOCK / 32), 2) void bwd_dkdv_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const __bf16* __restrict__ dO, const float* __restrict__ aux, __bf16* __restrict__ dK,
    __bf16* __restrict__ dV, int B, int N_all, int H, int nblk, float scale,
    const int32_t* __restrict__ colptr, const int32_t* __restrict__ rows_list,
    const int32_t* __restrict__ cu_seqlens, int64_t T_tok, char* __restrict__ ds,
    int64_t max_pairs) {
  constexpr int NK = BLOCK / 32;        // key groups (one wave each)
  using C = BwdCfg<D, BLOCK, NK, 32>;
  constexpr int AUXB = 2048;            // 32 rows of each plane, one 1 KB load each
  // 68 KB at head_dim 128, block 128: two workgroups fit one CU's LDS
  __shared__ __attribute__((aligned(1024))) char q_lds0[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char q_lds1[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char o_lds0[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char o_lds1[C::TILEB];
  __shared__ __attribute__((aligned(1024))) char a_lds0[AUXB];
  __shared__ __attribute__((aligned(1024))) char a_lds1[AUXB];
  // V rows of this key block (the B operand of dP = dO V^T), loaded once
  __shared__ __attribute__((aligned(1024))) char vblk_lds[BLOCK * C::ROWB];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kw = w;   // 32-key group
  const int l32 = lane & 31, g = lane >> 5;
  const int64_t lt = blockIdx.x;   // tile order: see the launcher
  const int j = (int)(lt % nblk);
  const int64_t bh = lt / nblk;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int64_t tok_stride = (int64_t)H * D;
  const SampleRows sr = sample_rows(cu_seqlens, T_tok, b, h, H, N_all);
  const int N = sr.n;
  if (N <= 0 || j * BLOCK >= N) return;   // uniform over the workgroup
  const int64_t base_bh = sr.tok0 * tok_stride + (int64_t)h * D;
  const int key = j * BLOCK + 32 * kw + l32;
  const int p0 = colptr[lt];
  int p1 = colptr[lt + 1];
  while (p1 > p0 && rows_list[p1 - 1] >= (N + BLOCK - 1) / BLOCK) --p1;   // past the sample
  const int T = (p1 - p0) * C::SUBS;

  // dK^T and dV^T in the 16x16 layout: [dt][kg] lane holds
  // X^T[16 dt + 4 gq + (0..3)][key 32 kw + 16 kg + c16]
  constexpr int DT16 = D / 16;
  const int c16 = lane & 15, gq = lane >> 4;
  f32x4 dk16[DT16][2], dv16[DT16][2];
#pragma unroll
  for (int dt = 0; dt < DT16; ++dt) dk16[dt][0] = dk16[dt][1] = dv16[dt][0] = dv16[dt][1] = f32x4{};

  if (T > 0) {
    bf16x8 kop[C::KS];
    {
      const int64_t off = base_bh + (int64_t)min(key, N - 1) * tok_stride + 8 * g;
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) kop[ks] = *reinterpret_cast<const bf16x8*>(K + off + 16 * ks);
    }
    const LaneOffsets<C> lo(w, lane, tok_stride);
    {   // V block: BLOCK rows in the swizzled row layout (rows past N read zeros)
      const int k0 = j * BLOCK;
      const int nrec = (N - k0 - 1) * (int)(tok_stride * 2) + 2 * D;
      const __amdgpu_buffer_rsrc_t rv = buffer_rsrc(V + base_bh + (int64_t)k0 * tok_stride, nrec);
#pragma unroll
      for (int half = 0; half < C::SUBS; ++half)
#pragma unroll
        for (int u = 0; u < C::IPW; ++u)
          buffer_load_lds16(rv, vblk_lds + half * C::TILEB + (w * C::IPW + u) * 1024,
                            lo.dma[u] + half * C::ST * (int)(tok_stride * 2));
    }
    const char* const vrow = vblk_lds + 32 * kw * C::ROWB;   // this wave's 32 keys
    // dO^T and Q^T operands of the 16x16x32 products for d tile dt: lane group
    // gq reads query rows base(gq) + (c16 >> 2) (slots 0..3) and the same + 16
    // (slots 4..7), columns 16 dt + 4 (c16 & 3) .. +3, base(gq) =
    // 8 (gq & 1) + 4 (gq >> 1): the rows the P / dS exchange leaves there.
    int rtr[DT16];
#pragma unroll
    for (int dt = 0; dt < DT16; ++dt) {
      const int d = 16 * dt + 4 * (c16 & 3);
      rtr[dt] = lds_off<C::CPR>(8 * (gq & 1) + 4 * (gq >> 1) + (c16 >> 2), d >> 3) + 2 * (d & 7);
    }

    // Tile t: 32 query rows of Q and dO, and their {LSE log2 e, -delta}.
    auto load_tile = [&](int t, char* qd, char* od, char* ad) __attribute__((always_inline)) {
      const int i = rows_list[p0 + t / C::SUBS];
      const int r0 = i * BLOCK + (t % C::SUBS) * C::ST;
      const int nrec = r0 < N ? (N - r0 - 1) * (int)(tok_stride * 2) + 2 * D : 0;
      const __amdgpu_buffer_rsrc_t rq = buffer_rsrc(Q + base_bh + (int64_t)r0 * tok_stride, nrec);
      const __amdgpu_buffer_rsrc_t ro = buffer_rsrc(dO + base_bh + (int64_t)r0 * tok_stride, nrec);
#pragma unroll
      for (int u = 0; u < C::IPW; ++u) {
        buffer_load_lds16(rq, qd + (w * C::IPW + u) * 1024, lo.dma[u]);
        buffer_load_lds16(ro, od + (w * C::IPW + u) * 1024, lo.dma[u]);
      }
      if (w == 0) {   // rows past N (and lanes past the tile's rows) read zeros
        const int nb = r0 < N ? min(N - r0, C::ST) * 4 : 0;
        buffer_load_lds16(buffer_rsrc(aux + sr.stat0 + r0, nb), ad, 16 * lane);
        buffer_load_lds16(buffer_rsrc(aux + (int64_t)H * T_tok + sr.stat0 + r0, nb), ad + 1024,
                          16 * lane);
      }
    };
    const float c2 = scale * kLog2e;

    // dS of the last computed tile, not yet stored (pos -1: nothing to store)
    struct {
      u32x4 u0, u1;
      int pos = -1, sub = 0;
    } pend;
    auto store_pending = [&]() __attribute__((always_inline)) {
      if (pend.pos < 0) return;
      u32x4 u0 = pend.u0, u1 = pend.u1;
      if ((j + 1) * BLOCK > N) {   // keys past N store zeros (their P is not 0)
        const int k0 = j * BLOCK + 32 * kw + c16;
        if (k0 >= N) u0[0] = u0[1] = u1[0] = u1[1] = 0u;
        if (k0 + 16 >= N) u0[2] = u0[3] = u1[2] = u1[3] = 0u;
      }
      char* dst = ds + (int64_t)pend.pos * (2 * BLOCK * BLOCK) + (pend.sub * NK + kw) * 2048 +
                  16 * (16 * gq + (c16 ^ (4 * (gq & 1))));
      __builtin_nontemporal_store(u0, reinterpret_cast<u32x4*>(dst));
      __builtin_nontemporal_store(u1, reinterpret_cast<u32x4*>(dst + 1024));
    };
    auto step = [&](int t, int pos, const char* qt_lds, const char* ot_lds, const char* at_lds)
        __attribute__((always_inline)) {
      // S = Q K^T and dP = dO V^T for the tile's 32 query rows
      const float* const a_pl = reinterpret_cast<const float*>(at_lds) + 4 * g;
      f32x16 s = f32x16{}, dp;
#pragma unroll
      for (int a = 0; a < 4; ++a) {   // dP - delta directly: start at -delta
        const f32x4 x = *reinterpret_cast<const f32x4*>(a_pl + 256 + 8 * a);
#pragma unroll
        for (int e = 0; e < 4; ++e) dp[4 * a + e] = x[e];
      }
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        const int off = lo.row[ks];
        s = mfma32(*reinterpret_cast<const bf16x8*>(qt_lds + off), kop[ks], s);
        const bf16x8 vop = *reinterpret_cast<const bf16x8*>(vrow + lo.row[ks]);
        dp = mfma32(*reinterpret_cast<const bf16x8*>(ot_lds + off), vop, dp);
      }
      // P and dS (query rows 8 a + 4 g + (0..3) of key column l32) as bf16
      // pairs: [0] holds elements 0-3, 8-11 (rows 4 g + {0..3, 16..19}),
      // [1] elements 4-7, 12-15 (rows 4 g + {8..11, 24..27})
      u32x4 pp[2], pd[2];
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const f32x4 ls = *reinterpret_cast<const f32x4*>(a_pl + 8 * a);
#pragma unroll
        for (int e = 0; e < 4; e += 2) {
          const int idx = 4 * a + e;
          const float p0 = fast_exp2(__builtin_fmaf(s[idx], c2, -ls[e]));
          const float p1 = fast_exp2(__builtin_fmaf(s[idx + 1], c2, -ls[e + 1]));
          const int r = (idx >> 2) & 1, c = ((idx & 3) >> 1) + 2 * (idx >> 3);
          pp[r][c] = pack_bf16x2(p0, p1);
          pd[r][c] = pack_bf16x2(p0 * dp[idx], p1 * dp[idx + 1]);
        }
      }
      // to the B-operand layout of two 16-key groups: register 0 serves keys
      // c16 of this wave's 32, register 1 keys 16 + c16
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const auto r0 = __builtin_amdgcn_permlane16_swap(pp[0][v], pp[1][v], false, false);
        pp[0][v] = r0[0];
        pp[1][v] = r0[1];
        const auto r1 = __builtin_amdgcn_permlane16_swap(pd[0][v], pd[1][v], false, false);
        pd[0][v] = r1[0];
        pd[1][v] = r1[1];
      }
      if constexpr (STORE) {
        // this tile's dS, stored by the next iteration (or after the loop)
        pend.u0 = u32x4{pd[0][0], pd[0][1], pd[1][0], pd[1][1]};   // queries base(gq) + 0..3
        pend.u1 = u32x4{pd[0][2], pd[0][3], pd[1][2], pd[1][3]};   // queries base(gq) + 16..19
        pend.pos = pos;
        pend.sub = t % C::SUBS;
      }
      // dV^T += dO^T P and dK^T += Q^T dS over the tile's 32 query rows
#pragma unroll
      for (int dt = 0; dt < DT16; ++dt) {
        const s16x4 o_lo = lds_read_tr16(ot_lds + rtr[dt]);
        const s16x4 o_hi = lds_read_tr16(ot_lds + rtr[dt] + 16 * C::ROWB);
        const s16x4 q_lo = lds_read_tr16(qt_lds + rtr[dt]);
        const s16x4 q_hi = lds_read_tr16(qt_lds + rtr[dt] + 16 * C::ROWB);
        const s16x8 o8 = {o_lo[0], o_lo[1], o_lo[2], o_lo[3], o_hi[0], o_hi[1], o_hi[2], o_hi[3]};
        const s16x8 q8 = {q_lo[0], q_lo[1], q_lo[2], q_lo[3], q_hi[0], q_hi[1], q_hi[2], q_hi[3]};
        const bf16x8 ao = __builtin_bit_cast(bf16x8, o8), aq = __builtin_bit_cast(bf16x8, q8);
#pragma unroll
        for (int kg = 0; kg < 2; ++kg) {
          dv16[dt][kg] = mfma16(ao, __builtin_bit_cast(bf16x8, pp[kg]), dv16[dt][kg]);
          dk16[dt][kg] = mfma16(aq, __builtin_bit_cast(bf16x8, pd[kg]), dk16[dt][kg]);
        }
      }
    };
    auto iter = [&](int t, auto par) __attribute__((always_inline)) {
      constexpr int P = decltype(par)::value;
      // column-list position of this tile's pair, or -1 (no dS store)
      int pos = -1;
      if constexpr (STORE) {
        const int e = p0 + t / C::SUBS;
        pos = (int64_t)e < max_pairs ? e : -1;
        // the previous tile's dS: a whole iteration to reach L2 before the
        // wait at this iteration's end
        store_pending();
      }
      if (t + 1 < T) load_tile(t + 1, P ? q_lds0 : q_lds1, P ? o_lds0 : o_lds1, P ? a_lds0 : a_lds1);
      step(t, pos, P ? q_lds1 : q_lds0, P ? o_lds1 : o_lds0, P ? a_lds1 : a_lds0);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
    };

    load_tile(0, q_lds0, o_lds0, a_lds0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    int t = 0;
    for (; t + 1 < T; t += 2) {
      iter(t, I0{});
      iter(t + 1, I1{});
    }
    if (t < T) iter(t, I0{});
    if constexpr (STORE) store_pending();
  }

  // lane stores columns 16 dt + 4 gq .. +3 of keys 32 kw + 16 kg + c16
  auto store_out = [&](__bf16* X, const f32x4 (&acc)[DT16][2], float mul) __attribute__((always_inline)) {
#pragma unroll
    for (int kg = 0; kg < 2; ++kg) {
      const int ko = j * BLOCK + 32 * kw + 16 * kg + c16;
      if (ko >= N) continue;
      const int64_t off = base_bh + (int64_t)ko * tok_stride;
#pragma unroll
      for (int dt = 0; dt < DT16; ++dt) {
        bf16x4 v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = (__bf16)(acc[dt][kg][e] * mul);
        *reinterpret_cast<bf16x4*>(X + off + 16 * dt + 4 * gq) = v4;
      }
    }
  };
  store_out(dK, dk16, scale);
  store_out(dV, dv16, 1.f);
}

template <int D, int BLOCK>
hipError_t launch_bwd_t(const void* q, const void* k, const void* v, const void* o,
                        const void* dout, const float* lse, void* dq, void* dk, void* dv,
                        const AttnShape& sh, const int32_t* rowptr, const int32_t* cols,
                        const int32_t* colptr, const int32_t* rows, float* aux, const DsTiles& ds,
                        hipStream_t s) {
  auto bf = [](const void* p) { return static_cast<const __bf16*>(p); };
  const int64_t rows_total = sh.T * sh.H * (D / 8);
  // One workgroup per (b, h, block) in plain order. Workgroups go round-robin
  // to the 8 XCDs, so all XCDs work on the same few heads at once (their K and
  // V stay in the shared last-level cache) and a run of heavy blocks is spread
  // over every XCD.
  const int64_t nrow = (int64_t)sh.B * sh.H * sh.nblk;
  const dim3 grid((unsigned)nrow);
  const bool store = ds.max_pairs > 0 && ds.tiles && ds.map && ds.row_ok;
  if (store) {
    TraceScope ts_(s, "bwd_ds_map");
    hipLaunchKernelGGL(bwd_ds_map_kernel, grid, dim3(64), 0, s, rowptr, cols, colptr, rows, sh.nblk,
                       ds.max_pairs, ds.map, ds.row_ok);
  }
  {
    TraceScope ts_(s, "bwd_prep", D);
    hipLaunchKernelGGL((bwd_prep_kernel<D>), dim3((unsigned)((rows_total + 255) / 256)), dim3(256), 0,
                     s, bf(o), bf(dout), lse, aux, sh.T, sh.N, sh.H, sh.cu != nullptr);
  }
  if (store) {
    TraceScope ts_(s, "bwd_dkdv_store", D, BLOCK);
    hipLaunchKernelGGL((bwd_dkdv_kernel<D, BLOCK, true>), grid, dim3(64 * (BLOCK / 32)), 0, s,
                     bf(q), bf(k), bf(v), bf(dout), aux, static_cast<__bf16*>(dk),
                     static_cast<__bf16*>(dv), sh.B, sh.N, sh.H, sh.nblk, sh.scale, colptr, rows,
                     sh.cu, sh.T, ds.tiles, ds.max_pairs);
  } else {
    TraceScope ts_(s, "bwd_dkdv", D, BLOCK);
    hipLaunchKernelGGL((bwd_dkdv_kernel<D, BLOCK, false>), grid, dim3(64 * (BLOCK / 32)), 0, s,
                     bf(q), bf(k), bf(v), bf(dout), aux, static_cast<__bf16*>(dk),
                     static_cast<__bf16*>(dv), sh.B, sh.N, sh.H, sh.nblk, sh.scale, colptr, rows,
                     sh.cu, sh.T, static_cast<char*>(nullptr), (int64_t)0);
  }
  if (store) {
    TraceScope ts_(s, "bwd_dq_stored", D, BLOCK);
    hipLaunchKernelGGL((bwd_dq_stored_kernel<D, BLOCK>), grid, dim3(64 * (BLOCK / 32)), 0, s,
                     bf(k), static_cast<const char*>(ds.tiles), static_cast<__bf16*>(dq), sh.N, sh.H,
                     sh.nblk, sh.scale, rowptr, cols, sh.cu, sh.T, ds.map, ds.row_ok);
  }
  {
    // every query block without row_ok (all of them without stored tiles)
    TraceScope ts_(s, "bwd_dq", D, BLOCK);
    hipLaunchKernelGGL((bwd_dq_kernel<D, BLOCK>), grid, dim3(64 * (BLOCK / 32)), 0, s,
                     bf(q), bf(k), bf(v), bf(dout), aux, static_cast<__bf16*>(dq), sh.B, sh.N, sh.H,
                     sh.nblk, sh.scale, rowptr, cols, sh.cu, sh.T,
                     store ? static_cast<const int32_t*>(ds.row_ok) : nullptr);
  }
  return hipGetLastError();
}

// The allocation-free entry point's scratch: a file-scope device array, one
// copy per GPU, allocated by the loader with the code object and held until
// the process ends. Its name is a host-side stand-in in host code; only the
// address hipGetSymbolAddress returns is ever passed to a kernel.
__device__ __align__(256) float scratch[kNoallocScratchBytes / sizeof(float)];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

hipError_t noalloc_scratch(hipStream_t s, float** ptr) {
  int dev = 0;
  hipError_t e = s ? hipStreamGetDevice(s, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    // once per device, with that device current
    int cur = 0;
    if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    const hipError_t e2 = cur != dev ? hipSetDevice(cur) : hipSuccess;
    if (e != hipSuccess) return e;
    if (e2 != hipSuccess) return e2;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = static_cast<float*>(p);
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_bsattn_bwd(const void* q, const void* k, const void* v, const void* o,
                             const void* dout, const float* lse, void* dq, void* dk, void* dv,
                             const AttnShape& sh, const int32_t* rowptr, const int32_t* cols,
                             const int32_t* colptr, const int32_t* rows, float* aux,
                             const DsTiles& ds, hipStream_t s) {
#define UT_BWD(DD, BB)                                                                        \
  if (sh.D == DD && sh.block == BB)                                                           \
    return launch_bwd_t<DD, BB>(q, k, v, o, dout, lse, dq, dk, dv, sh, rowptr, cols, colptr, \
                                rows, aux, ds, s);
  UT_BWD(128, 128)
  UT_BWD(128, 64)
  UT_BWD(64, 128)
  UT_BWD(64, 64)
#undef UT_BWD
  return hipErrorInvalidValue;
}

}  // namespace ut
