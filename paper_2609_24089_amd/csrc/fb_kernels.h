// Attention forward, first backward and the two BoB passes as gfx950 kernels.
//
// Notation follows the paper: tau = softmax scale, U_Q/U_K/U_V are the
// cotangents on (dQ, dK, dV), and the BoB outputs are Qt, Kt, Vt, dOt
// (the paper's tilde-Q, tilde-K, tilde-V, tilde-dO).  All matrices are
// [B*H, N, D] row-major; row scalars L, D, alpha, E are fp32 [B*H, N].
// Softmax probabilities are recomputed from L as exp2(S*tau*log2e - L*log2e).
//
// Every kernel takes `causal`: without it every key is valid for every query;
// with it the mask M_mask of eq. 1 is -inf where key > query, masked entries
// get P = 0, tiles above the diagonal are skipped and diagonal tiles are
// masked per element.  Rows past N are masked the same way.
//
// Every kernel also takes `grp`, the number of query heads that share one
// key/value head (grouped-query attention, the extension the paper names in
// its limitations; grp = 1 is multi-head attention).  Query-side tensors
// (Q, dO, U_Q, O, dQ, Qt, dOt and the row scalars) have B*H heads and
// key-side tensors (K, V, U_K, U_V, dK, dV, Kt, Vt) B*H/grp; query head bh
// reads key/value head bh / grp.  Row kernels run one workgroup per query
// head row block; column kernels one per key/value head column block, and
// stream the grp query heads of that key/value head one after another, so
// their key-side outputs sum over the group with no atomics.  On grids with
// no more workgroups than CUs a column workgroup holds two wave sets that
// split those streamed tiles and add their partial sums through LDS.  The
// kParts forms split a column block over several workgroups instead, each
// storing fp32 partial sums to a caller's workspace that
// bob_column_parts_reduce_kernel adds (small or causal grids).
#pragma once
#include "fb_common.h"

namespace fb {

// ===========================================================================
// Forward: O = softmax(tau Q K^T + M) V and L = logsumexp(tau Q K^T + M)
// (eq. 1 and the log-normalizer of Sec. 2).  Stationary: query rows.
// Streamed: K, V.  Online softmax against a reference row maximum that
// moves only when a row has grown past it by more than 2^8.
// ===========================================================================
template <typename T, int D, int MR, int NW, int OCC, int NSTAGE>
__global__ __launch_bounds__(NW * 64, OCC) void attn_fwd_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    T* __restrict__ O, float* __restrict__ L, int N, int nRB, int total, float scale, int causal, int grp) {
  using E = Elt<T>;
  using G = Geo<T, D>;
  constexpr int BR = 16 * MR * NW;
  __shared__ __attribute__((aligned(16))) T lds[NSTAGE][2 * G::kTileElems];

  int bh, rb;
  map_block(nRB, total, bh, rb, causal != 0);
  const int64_t hoff = (int64_t)bh * N * D;
  const int64_t kvoff = (int64_t)(bh / grp) * N * D;  // key/value head of this query head
  const int l = lane_id(), g = l >> 4, j = l & 15;
  const int row0 = rb * BR + wave_id() * 16 * MR;

  u32x4 qf[MR][G::kChunks];
#pragma unroll
  for (int mb = 0; mb < MR; ++mb) load_stationary<T, D>(qf[mb], Q + hoff, row0 + 16 * mb + j, N);

  floatx4 acc[G::kNB][MR];
#pragma unroll
  for (int nb = 0; nb < G::kNB; ++nb)
#pragma unroll
    for (int mb = 0; mb < MR; ++mb) acc[nb][mb] = floatx4{0.f, 0.f, 0.f, 0.f};
  float mrun[MR], lsum[MR];
#pragma unroll
  for (int mb = 0; mb < MR; ++mb) { mrun[mb] = -1e30f; lsum[mb] = 0.f; }
  const float c = scale * kLog2e;
  floatx4 s[2][MR];
  typename E::TFrag pf[MR];

  // Online softmax against a lazily moved reference row maximum mrun (log2
  // domain).  The fast path forms p = exp2(s c - mrun) directly and checks
  // that no lane's eight p exceed 2^8 in sum (so every exponent is <= 8 and
  // p <= 256: exact in fp32 and fine in bf16; a NaN sum fails the check as
  // well); the stale reference cancels in
  // O = sum(P v) / sum(P) and in L = mrun + log2 sum(P).  Only when some lane
  // fails (a row grew by about 2^8 or more, or the first tile) does the slow
  // path find the tile's row maxima, move the reference of rows that grew by
  // more than 2^8, rescale their output accumulators and row sums, and form
  // p again.  `mode` 2 masks invalid entries (exponent -inf, p = 0).
  auto softmax_step = [&](int s0, int mode) {
#pragma unroll
    for (int mb = 0; mb < MR; ++mb) {
      floatx4 e[2];
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 4; ++r) e[sb][r] = __builtin_fmaf(s[sb][mb][r], c, -mrun[mb]);
      if (mode == 2) mask_tile1<true>(e, s0, row0 + 16 * mb + j, N, causal != 0);
      float p[8], ls = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        p[i] = fast_exp2(e[i >> 2][i & 3]);
        ls += p[i];
      }
      if (__builtin_amdgcn_ballot_w64(!(ls <= kRescaleP)) != 0) {
        // some row grew: tile maxima of the valid entries (in log2 units)
        floatx4 x[2];
#pragma unroll
        for (int sb = 0; sb < 2; ++sb) x[sb] = s[sb][mb] * c;
        if (mode == 2) mask_tile1<true>(x, s0, row0 + 16 * mb + j, N, causal != 0);
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 8; ++i) mx = fmaxf(mx, x[i >> 2][i & 3]);
        mx = group_max(mx);
        if (__builtin_amdgcn_ballot_w64(mx > mrun[mb] + kRescaleLog2) != 0) {
          const float mnew = fmaxf(mrun[mb], mx);
          const float corr = fast_exp2(mrun[mb] - mnew);
          mrun[mb] = mnew;
          lsum[mb] *= corr;
#pragma unroll
          for (int nb = 0; nb < G::kNB; ++nb) acc[nb][mb] *= corr;
        }
        ls = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          p[i] = fast_exp2(x[i >> 2][i & 3] - mrun[mb]);
          ls += p[i];
        }
      }
      lsum[mb] += ls;
#pragma unroll
      for (int i = 0; i < 8; ++i) pf[mb].set(i, p[i]);
    }
  };

  const T* const src[2] = {K + kvoff, V + kvoff};
  const int nT = (N + kBS - 1) / kBS;
  const int it_end = causal ? min(nT, (min(rb * BR + BR, N) - 1) / kBS + 1) : nT;
  const TileCopy<T, D, NW, 2> copy(wave_id());
  stream_loop<NSTAGE, tile_loads<T, D, NW, 2>()>(
      0, it_end,
      [&](int it, int st) { copy.issue(src, (T FB_LDS*)lds[st], it * kBS, N); },
      [&](int it, int st) {
        const int s0 = it * kBS;
        const int mode = tile_mode_rowmajor(s0, row0, row0 + 16 * MR - 1, N, causal != 0);
        if (mode == 0) return;
        const T FB_LDS* Ks = (const T FB_LDS*)lds[st];
        const T FB_LDS* Vs = Ks + G::kTileElems;
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int mb = 0; mb < MR; ++mb) s[sb][mb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int kk = 0; kk < G::kChunks; ++kk) {
            const u32x4 a = *(const u32x4 FB_LDS*)(Ks + G::chunk_off(16 * sb + j, 4 * kk + g));
#pragma unroll
            for (int mb = 0; mb < MR; ++mb) s[sb][mb] = E::mma_chunk(a, qf[mb][kk], s[sb][mb]);
          }
        softmax_step(s0, mode);
#pragma unroll
        for (int nb = 0; nb < G::kNB; ++nb) {
          const typename E::AFrag a = G::load_afrag(Vs, 16 * nb);
#pragma unroll
          for (int mb = 0; mb < MR; ++mb) acc[nb][mb] = E::mma_acc(a, pf[mb], acc[nb][mb]);
        }
      });
#pragma unroll
  for (int mb = 0; mb < MR; ++mb) {
    const int row = row0 + 16 * mb + j;
    const float lt = group_sum(lsum[mb]);
    const float inv = 1.f / lt;
    if (row < N) {
#pragma unroll
      for (int nb = 0; nb < G::kNB; ++nb) E::store4(O + hoff + (int64_t)row * D + 16 * nb + 4 * g, acc[nb][mb] * inv);
      if (g == 0) L[(int64_t)bh * N + row] = (mrun[mb] + __log2f(lt)) * kLn2;
    }
  }
}

// ===========================================================================
// First backward, row side: D_i = do_i . o_i and dQ = tau dS K with
// dS = P (dP - D), dP = dO V^T (eqs. 2-3).  Stationary: Q, dO rows.
// Streamed: K, V.  Writes D and dQ once per row; no atomics.
// ===========================================================================
template <typename T, int D, int MR, int NW, int OCC, int NSTAGE>
__global__ __launch_bounds__(NW * 64, OCC) void attn_bwd_rows_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    const T* __restrict__ O, const T* __restrict__ dO, const float* __restrict__ L,
    T* __restrict__ dQ, float* __restrict__ Dout, int N, int nRB, int total, float scale, int causal, int grp) {
  using E = Elt<T>;
  using G = Geo<T, D>;
  constexpr int BR = 16 * MR * NW;
  __shared__ __attribute__((aligned(16))) T lds[NSTAGE][2 * G::kTileElems];

  int bh, rb;
  map_block(nRB, total, bh, rb, causal != 0);
  const int64_t hoff = (int64_t)bh * N * D;
  const int64_t kvoff = (int64_t)(bh / grp) * N * D;  // key/value head of this query head
  const int l = lane_id(), g = l >> 4, j = l & 15;
  const int row0 = rb * BR + wave_id() * 16 * MR;

  u32x4 qf[MR][G::kChunks], dof[MR][G::kChunks];
  float lb[MR], drow[MR];
#pragma unroll
  for (int mb = 0; mb < MR; ++mb) {
    const int row = row0 + 16 * mb + j;
    load_stationary<T, D>(qf[mb], Q + hoff, row, N);
    load_stationary<T, D>(dof[mb], dO + hoff, row, N);
    u32x4 of[G::kChunks];
    load_stationary<T, D>(of, O + hoff, row, N);
    float part = 0.f;
#pragma unroll
    for (int kk = 0; kk < G::kChunks; ++kk) part += E::dot_chunk(dof[mb][kk], of[kk]);
    drow[mb] = group_sum(part);
    lb[mb] = row < N ? L[(int64_t)bh * N + row] * kLog2e : 0.f;
    if (g == 0 && row < N) Dout[(int64_t)bh * N + row] = drow[mb];
  }

  floatx4 acc[G::kNB][MR];
#pragma unroll
  for (int nb = 0; nb < G::kNB; ++nb)
#pragma unroll
    for (int mb = 0; mb < MR; ++mb) acc[nb][mb] = floatx4{0.f, 0.f, 0.f, 0.f};
  const float c = scale * kLog2e;
  floatx4 s[2][MR], dp[2][MR];
  typename E::TFrag dsf[MR];

  // s holds exponents s*tau*log2e - L*log2e (masked entries -inf); dp holds
  // dP - D (the MFMA started from -D)
  auto elementwise = [&]() {
#pragma unroll
    for (int mb = 0; mb < MR; ++mb)
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = fast_exp2(s[sb][mb][r]);
          dsf[mb].set(4 * sb + r, p * dp[sb][mb][r]);
        }
  };

  const T* const src[2] = {K + kvoff, V + kvoff};
  const int nT = (N + kBS - 1) / kBS;
  const int it_end = causal ? min(nT, (min(rb * BR + BR, N) - 1) / kBS + 1) : nT;
  const TileCopy<T, D, NW, 2> copy(wave_id());
  stream_loop<NSTAGE, tile_loads<T, D, NW, 2>()>(
      0, it_end,
      [&](int it, int st) { copy.issue(src, (T FB_LDS*)lds[st], it * kBS, N); },
      [&](int it, int st) {
        const int s0 = it * kBS;
        const int mode = tile_mode_rowmajor(s0, row0, row0 + 16 * MR - 1, N, causal != 0);
        if (mode == 0) return;
        const T FB_LDS* Ks = (const T FB_LDS*)lds[st];
        const T FB_LDS* Vs = Ks + G::kTileElems;
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int mb = 0; mb < MR; ++mb) {
            s[sb][mb] = floatx4{0.f, 0.f, 0.f, 0.f};
            dp[sb][mb] = floatx4{-drow[mb], -drow[mb], -drow[mb], -drow[mb]};
          }
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int kk = 0; kk < G::kChunks; ++kk) {
            const int off = G::chunk_off(16 * sb + j, 4 * kk + g);
            const u32x4 ak = *(const u32x4 FB_LDS*)(Ks + off);
            const u32x4 av = *(const u32x4 FB_LDS*)(Vs + off);
#pragma unroll
            for (int mb = 0; mb < MR; ++mb) {
              s[sb][mb] = E::mma_chunk(ak, qf[mb][kk], s[sb][mb]);
              dp[sb][mb] = E::mma_chunk(av, dof[mb][kk], dp[sb][mb]);
            }
          }
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int mb = 0; mb < MR; ++mb)
#pragma unroll
            for (int r = 0; r < 4; ++r) s[sb][mb][r] = __builtin_fmaf(s[sb][mb][r], c, -lb[mb]);
        if (mode == 2) mask_tile<true>(s, s0, row0 + j, N, causal != 0);
        elementwise();
#pragma unroll
        for (int nb = 0; nb < G::kNB; ++nb) {
          const typename E::AFrag a = G::load_afrag(Ks, 16 * nb);
#pragma unroll
          for (int mb = 0; mb < MR; ++mb) acc[nb][mb] = E::mma_acc(a, dsf[mb], acc[nb][mb]);
        }
      });
#pragma unroll
  for (int mb = 0; mb < MR; ++mb) {
    const int row = row0 + 16 * mb + j;
    if (row < N) {
#pragma unroll
      for (int nb = 0; nb < G::kNB; ++nb) E::store4(dQ + hoff + (int64_t)row * D + 16 * nb + 4 * g, acc[nb][mb] * scale);
    }
  }
}

// ===========================================================================
// First backward, column side: dV = P^T dO and dK = tau dS^T Q (eqs. 2-3).
// Stationary: K, V rows.  Streamed: Q, dO tiles with their L and D.
// KS wave sets of NW waves share the workgroup's column block and take the
// streamed tiles round-robin, each with its own LDS ring; their partial sums
// are added through LDS at the end (KS = 2 fills a CU when the grid has no
// more workgroups than CUs).
// ===========================================================================
template <typename T, int D, int MC, int NW, int OCC, int NSTAGE, bool kGQA, int KS, bool kParts = false,
          bool kFlush = false, bool kKL = false>
__global__ __launch_bounds__(KS * NW * 64, OCC) void attn_bwd_cols_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    const T* __restrict__ dO, const float* __restrict__ L, const float* __restrict__ Dv,
    T* __restrict__ dK, T* __restrict__ dV, int N, int nRB, int total, float scale, int causal, int grp,
    float* __restrict__ parts_out = nullptr, int nparts = 1, int flush_tiles = 0) {
  static_assert(KS == 1 || KS == 2, "wave sets");
  using E = Elt<T>;
  using G = Geo<T, D>;
  constexpr int BC = 16 * MC * NW;
  // The tile ring, and the raw L, D of NSTAGE tiles with two slots of
  // transformed ones: T0 = -L log2e (the exponent offset), T1 = -D (the dP
  // tile's start value).  One LDS variable, for the reason given at Pass 2's Smem2.
  // With kKL the stationary K rows sit in LDS instead of registers, in
  // 32-row tiles of the streamed tiles' layout: one per wave at 32 key rows
  // per wave (MC = 2), one per pair of consecutive waves at 16 (MC = 1),
  // shared by the waves of the same index in each wave set.  At d <= 128 the
  // freed registers let a wave own 32 key rows at two waves per SIMD, which
  // halves the LDS bytes per MFMA of the streamed tiles for 8 more b128 reads
  // per tile; at d = 256 they let 16 rows per wave run at two waves per SIMD.
  struct Smem {
    T lds[KS][NSTAGE][2 * G::kTileElems];
    float rawsc[KS][NSTAGE][2 * kBS];
    float tsc[KS][2][2 * kBS];
  };
  constexpr int kWPT = kBS / (16 * MC);  // waves per stationary K tile
  static_assert(!kKL || (kBS % (16 * MC) == 0 && NW % kWPT == 0), "stationary K in LDS: 32-row tiles");
  struct SmemK : Smem {
    T kst[NW / kWPT][G::kTileElems];
  };
  __shared__ __attribute__((aligned(16))) std::conditional_t<kKL, SmemK, Smem> sm;
  auto& lds = sm.lds;
  auto& rawsc = sm.rawsc;
  auto& tsc = sm.tsc;

  int bh, rb, part = 0;
  if constexpr (kParts)
    map_column_job(nRB, total, nparts, bh, rb, part);
  else
    map_block(nRB, total, bh, rb);
  const int64_t hoff = (int64_t)bh * N * D;
  const int l = lane_id(), g = l >> 4, j = l & 15;
  const int ks = KS == 1 ? 0 : wave_id() / NW;       // wave set
  const int wl = KS == 1 ? wave_id() : wave_id() % NW;  // wave within its set
  const int col0 = rb * BC + wl * 16 * MC;

  u32x4 kf[kKL ? 1 : MC][G::kChunks], vf[MC][G::kChunks];
#pragma unroll
  for (int mc = 0; mc < MC; ++mc) {
    if constexpr (!kKL) load_stationary<T, D>(kf[mc], K + hoff, col0 + 16 * mc + j, N);
    load_stationary<T, D>(vf[mc], V + hoff, col0 + 16 * mc + j, N);
  }
  if constexpr (kKL) {
    // rows past N read as zeros; a wave whose rows all lie past N stores
    // nothing, so its tile stays unwritten.  The first wave set copies; the
    // loop's first wait_vm<0>() and barrier publish the tile to both.
    if (ks == 0 && wl % kWPT == 0 && col0 < N) {
      const TileCopy<T, D, 1, 1> kc(0);
      const T* const ksrc[1] = {K + hoff};
      kc.issue(ksrc, (T FB_LDS*)sm.kst[wl / kWPT], col0, N);
    }
  }
  floatx4 dk[G::kNB][MC], dv[G::kNB][MC];
#pragma unroll
  for (int nb = 0; nb < G::kNB; ++nb)
#pragma unroll
    for (int mc = 0; mc < MC; ++mc) dk[nb][mc] = dv[nb][mc] = floatx4{0.f, 0.f, 0.f, 0.f};
  SectionSums<kFlush, G::kNB, MC> sect;
  sect.init();
  const float c = scale * kLog2e;
  floatx4 s[2][MC], dp[2][MC];
  typename E::TFrag pf[MC], dsf[MC];

  // s holds exponents s*tau*log2e - L*log2e (masked entries -inf); dp holds
  // dP - D (the MFMA started from -D)
  auto elementwise = [&]() {
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) {
          const float p = fast_exp2(s[sb][mc][r]);
          pf[mc].set(4 * sb + r, p);
          dsf[mc].set(4 * sb + r, p * dp[sb][mc][r]);
        }
  };

  const int nT = (N + kBS - 1) / kBS;
  const int it_begin = causal ? (rb * BC) / kBS : 0;
  const int nTh = nT - it_begin;
  const StreamSplit<kGQA, KS, kParts> sp{it_begin, nTh, kGQA ? grp * nTh : nTh, ks, bh, grp, part, nparts};
  const TileCopy<T, D, NW, 2> copy(wl);
  stream_loop_rs<NSTAGE, tile_loads<T, D, NW, 2>(), 1>(
      sp.begin(), sp.end(nT), __builtin_amdgcn_readfirstlane(wl) == 0,
      [&](int it, int rs) {
        const int64_t qs = (int64_t)sp.qhead(it) * N;
        issue_scalar_pair((float FB_LDS*)rawsc[ks][rs], L + qs, Dv + qs, sp.tile(it) * kBS, N);
      },
      [&](int it, int st) {
        const int64_t qo = (int64_t)sp.qhead(it) * N * D;
        const T* const src[2] = {Q + qo, dO + qo};
        copy.issue(src, (T FB_LDS*)lds[ks][st], sp.tile(it) * kBS, N);
      },
      [&](int it, int rs, int ts) {
        (void)it;
        if (l < kBS) {
          const float FB_LDS* raw = (const float FB_LDS*)rawsc[ks][rs];
          float FB_LDS* t = (float FB_LDS*)tsc[ks][ts];
          t[l] = -raw[l] * kLog2e;
          t[kBS + l] = -raw[kBS + l];
        }
      },
      [&](int it, int st, int ts, auto&& prep_next) {
        const int s0 = sp.tile(it) * kBS;
        const int mode = sp.live(it) ? tile_mode_colmajor(s0, col0, col0 + 16 * MC - 1, N, causal != 0) : 0;
        if (mode == 0) {
          prep_next();
          return;
        }
        const T FB_LDS* Qs = (const T FB_LDS*)lds[ks][st];
        const T FB_LDS* dOs = Qs + G::kTileElems;
        const float FB_LDS* Ts = (const float FB_LDS*)tsc[ks][ts];
#pragma unroll
        for (int sb = 0; sb < 2; ++sb) {
          const floatx4 t1 = *(const floatx4 FB_LDS*)(Ts + kBS + 16 * sb + 4 * g);
#pragma unroll
          for (int mc = 0; mc < MC; ++mc) {
            s[sb][mc] = floatx4{0.f, 0.f, 0.f, 0.f};
            dp[sb][mc] = t1;
          }
        }
        // the score MFMAs run at raised wave priority, so that a wave that
        // reaches them issues them ahead of the other waves' exponentials
        __builtin_amdgcn_s_setprio(1);
        if constexpr (kKL) {
          // each K chunk is read once per tile and serves both sub-blocks
          const T FB_LDS* Ks = (const T FB_LDS*)sm.kst[wl / kWPT];
          const int r0 = 16 * MC * (wl % kWPT);  // the wave's first row in the tile
#pragma unroll
          for (int kk = 0; kk < G::kChunks; ++kk) {
            u32x4 kfr[MC];
#pragma unroll
            for (int mc = 0; mc < MC; ++mc)
              kfr[mc] = *(const u32x4 FB_LDS*)(Ks + G::chunk_off(r0 + 16 * mc + j, 4 * kk + g));
#pragma unroll
            for (int sb = 0; sb < 2; ++sb) {
              const int off = G::chunk_off(16 * sb + j, 4 * kk + g);
              const u32x4 aq = *(const u32x4 FB_LDS*)(Qs + off);
              const u32x4 ado = *(const u32x4 FB_LDS*)(dOs + off);
#pragma unroll
              for (int mc = 0; mc < MC; ++mc) {
                s[sb][mc] = E::mma_chunk(aq, kfr[mc], s[sb][mc]);
                dp[sb][mc] = E::mma_chunk(ado, vf[mc][kk], dp[sb][mc]);
              }
            }
          }
        } else {
#pragma unroll
          for (int sb = 0; sb < 2; ++sb)
#pragma unroll
            for (int kk = 0; kk < G::kChunks; ++kk) {
              const int off = G::chunk_off(16 * sb + j, 4 * kk + g);
              const u32x4 aq = *(const u32x4 FB_LDS*)(Qs + off);
              const u32x4 ado = *(const u32x4 FB_LDS*)(dOs + off);
#pragma unroll
              for (int mc = 0; mc < MC; ++mc) {
                s[sb][mc] = E::mma_chunk(aq, kf[mc][kk], s[sb][mc]);
                dp[sb][mc] = E::mma_chunk(ado, vf[mc][kk], dp[sb][mc]);
              }
            }
        }
        __builtin_amdgcn_s_setprio(0);
#pragma unroll
        for (int sb = 0; sb < 2; ++sb) {
          const floatx4 t0 = *(const floatx4 FB_LDS*)(Ts + 16 * sb + 4 * g);
#pragma unroll
          for (int mc = 0; mc < MC; ++mc)
#pragma unroll
            for (int r = 0; r < 4; ++r) s[sb][mc][r] = __builtin_fmaf(s[sb][mc][r], c, t0[r]);
        }
        if (mode == 2) mask_tile<false>(s, s0, col0 + j, N, causal != 0);
        elementwise();
#pragma unroll
        for (int nb = 0; nb < G::kNB; ++nb) {
          const typename E::AFrag ado = G::load_afrag(dOs, 16 * nb);
          const typename E::AFrag aq = G::load_afrag(Qs, 16 * nb);
#pragma unroll
          for (int mc = 0; mc < MC; ++mc) {
            dv[nb][mc] = E::mma_acc(ado, pf[mc], dv[nb][mc]);
            dk[nb][mc] = E::mma_acc(aq, dsf[mc], dk[nb][mc]);
          }
        }
        sect.step(dk, dv, flush_tiles);
        prep_next();
      });
  sect.finish(dk, dv);
  if constexpr (KS == 2) {
    static_assert(sizeof(lds) >= (size_t)NW * G::kNB * MC * 1024, "set merge buffer");
    merge_wave_sets(dk, dv, ks, wl, (floatx4 FB_LDS*)&lds[0][0][0]);
    if (ks != 0) return;
  }
  if constexpr (kParts) {
    store_column_part<D>(parts_out, (int64_t)(total / nRB) * N * D, part, hoff, col0, N, dk, dv);
    return;
  }
#pragma unroll
  for (int mc = 0; mc < MC; ++mc) {
    const int col = col0 + 16 * mc + j;
    if (col < N) {
#pragma unroll
      for (int nb = 0; nb < G::kNB; ++nb) {
        E::store4(dK + hoff + (int64_t)col * D + 16 * nb + 4 * g, dk[nb][mc] * scale);
        E::store4(dV + hoff + (int64_t)col * D + 16 * nb + 4 * g, dv[nb][mc]);
      }
    }
  }
}

// ===========================================================================
// BoB Pass 1 (row-major; Alg. 1/2 Pass 1 with the affine fusion of Prop. 3.1).
// Stationary: Q, U_Q, dO rows (+ L, D).  Streamed: K, V, U_K, U_V.
// Per tile it recomputes S, P, dP, F, C (as transposed tiles), forms
// Pt0 = C + F (dP - D), and accumulates the row accumulators
//   alpha += rowsum(P F),  E0 += rowsum(P Pt0),
//   dOt0 += P U_V + (P F) V,  Omega += (P Pt0) K + (P (dP - D)) U_K,
//   Bacc += P K,  R += (P dP) K.
// Epilogue (eq. 8): E = E0 - alpha D, dOt = dOt0 - alpha O,
// Qt = tau (Omega - alpha R - E Bacc).  Writes alpha, E, Qt, dOt once.
//
// kWithDQ form: when the first-backward dQ is supplied, R is not accumulated.
// Since dQ / tau = sum_j P (dP - D) k_j = R - D Bacc, eq. 8 becomes
// Qt = tau (Omega - E0 Bacc) - alpha dQ with E0 = E + alpha D.  This drops one
// B_r x d accumulator and one tile contraction per tile, which is what lets
// the d = 128 kernel run two waves per SIMD.
//
// kAlphaGiven form: the second sweep of the three-pass control schedule
// (App. "Three-pass versus two-pass").  alpha comes in from a first sweep, so
// Pt = C + F (dP - D) - alpha dP and h = F - alpha are formed directly; the
// kernel accumulates E += rowsum(P Pt), Omega' += (P Pt) K + (P (dP - D)) U_K,
// Bacc += P K, dOt += P U_V + (P h) V and finishes Qt = tau (Omega' - E Bacc)
// (the one delayed correction).  Writes E, Qt, dOt.
// ===========================================================================
enum Pass1Form : int { kSixAcc = 0, kWithDQ = 1, kAlphaGiven = 2 };

template <typename T, int D, int MR, int NW, int OCC, int NSTAGE, int kForm, int DSPLIT, int kPF>
__global__ __launch_bounds__(NW * 64, OCC) void bob_pass1_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    const T* __restrict__ O, const T* __restrict__ dO, const T* __restrict__ UQ,
    const T* __restrict__ UK, const T* __restrict__ UV, const float* __restrict__ L,
    const float* __restrict__ Dv, const T* __restrict__ dQ, const float* __restrict__ alpha_in,
    T* __restrict__ Qt, T* __restrict__ dOt, float* __restrict__ alpha_out, float* __restrict__ E_out,
    int N, int nRB, int total, float scale, int causal, int grp) {
  using E = Elt<T>;
  using G = Geo<T, D>;
  constexpr bool kDQ = kForm == kWithDQ;
  constexpr bool kThree = kForm == kAlphaGiven;
  constexpr int BR = 16 * MR * NW;
  __shared__ __attribute__((aligned(16))) T lds[NSTAGE][4 * G::kTileElems];

  int bh, rb;
  map_block(nRB, total, bh, rb, causal != 0);
  const int64_t hoff = (int64_t)bh * N * D;
  const int64_t soff = (int64_t)bh * N;
  const int64_t kvoff = (int64_t)(bh / grp) * N * D;  // key/value head of this query head
  const int l = lane_id(), g = l >> 4, j = l & 15;
  const int row0 = rb * BR + wave_id() * 16 * MR;

  u32x4 qf[MR][G::kChunks], uqf[MR][G::kChunks], dof[MR][G::kChunks];
  float lb[MR], drow[MR], arow[MR];
#pragma unroll
  for (int mb = 0; mb < MR; ++mb) {
    const int row = row0 + 16 * mb + j;
    load_stationary<T, D>(qf[mb], Q + hoff, row, N);
    load_stationary<T, D>(uqf[mb], UQ + hoff, row, N);
    load_stationary<T, D>(dof[mb], dO + hoff, row, N);
    lb[mb] = row < N ? L[soff + row] * kLog2e : 0.f;
    drow[mb] = row < N ? Dv[soff + row] : 0.f;
    arow[mb] = (kThree && row < N) ? alpha_in[soff + row] : 0.f;
  }
  // With DSPLIT = 2 the grid's second dimension picks which half of the head
  // dims this workgroup accumulates and writes; both halves form the full
  // score tiles (and the row scalars, written by half 0 only).
  static_assert(G::kNB % DSPLIT == 0, "head-dim split");
  constexpr int kNBh = G::kNB / DSPLIT;
  const int nb0 = DSPLIT == 1 ? 0 : (int)blockIdx.y * kNBh;
  const bool write_scalars = DSPLIT == 1 || blockIdx.y == 0;
  constexpr int kNR = (kForm == kSixAcc) ? kNBh : 1;  // R accumulator only in the six-accumulator form
  floatx4 aDO[kNBh][MR], aOM[kNBh][MR], aB[kNBh][MR], aR[kNR][MR];
#pragma unroll
  for (int nb = 0; nb < kNBh; ++nb)
#pragma unroll
    for (int mb = 0; mb < MR; ++mb) aDO[nb][mb] = aOM[nb][mb] = aB[nb][mb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int nb = 0; nb < kNR; ++nb)
#pragma unroll
    for (int mb = 0; mb < MR; ++mb) aR[nb][mb] = floatx4{0.f, 0.f, 0.f, 0.f};
  float alpha[MR], e0[MR];
#pragma unroll
  for (int mb = 0; mb < MR; ++mb) alpha[mb] = e0[mb] = 0.f;
  const float c = scale * kLog2e;

  // transposed score tiles [s][t] = streamed . stationary, and the B-operand
  // fragments the accumulate step consumes
  floatx4 s[2][MR], dp[2][MR], f[2][MR], cc[2][MR];
  typename E::TFrag fP[MR], fPF[MR], fPPt[MR], fPdd[MR], fPdp[MR];

  auto score = [&](const T FB_LDS* Ks) {
    const T FB_LDS* Vs = Ks + G::kTileElems;
    const T FB_LDS* UKs = Vs + G::kTileElems;
    const T FB_LDS* UVs = UKs + G::kTileElems;
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int mb = 0; mb < MR; ++mb) {
        s[sb][mb] = f[sb][mb] = cc[sb][mb] = floatx4{0.f, 0.f, 0.f, 0.f};
        dp[sb][mb] = floatx4{-drow[mb], -drow[mb], -drow[mb], -drow[mb]};  // the dP tile starts at -D
      }
    // one score step: the five contractions of chunk kk of sub-block sb
    auto step = [&](int sb, int kk, const u32x4 (&a)[4]) {
#pragma unroll
      for (int mb = 0; mb < MR; ++mb) {
        s[sb][mb] = E::mma_chunk(a[0], qf[mb][kk], s[sb][mb]);        // S^T = K Q^T
        dp[sb][mb] = E::mma_chunk(a[1], dof[mb][kk], dp[sb][mb]);     // (dP - D)^T = V dO^T - D
        f[sb][mb] = E::mma_chunk(a[0], uqf[mb][kk], f[sb][mb]);       // (U_Q K^T)^T
        f[sb][mb] = E::mma_chunk(a[2], qf[mb][kk], f[sb][mb]);        // + (Q U_K^T)^T
        cc[sb][mb] = E::mma_chunk(a[3], dof[mb][kk], cc[sb][mb]);     // C^T = U_V dO^T
      }
    };
    auto read = [&](int sb, int kk, u32x4 (&a)[4]) {
      const int off = G::chunk_off(16 * sb + j, 4 * kk + g);
      a[0] = *(const u32x4 FB_LDS*)(Ks + off);
      a[1] = *(const u32x4 FB_LDS*)(Vs + off);
      a[2] = *(const u32x4 FB_LDS*)(UKs + off);
      a[3] = *(const u32x4 FB_LDS*)(UVs + off);
    };
    if constexpr (kPF >= 2) {
      // operands of step st + 1 are read before the MFMAs of step st
      constexpr int kSteps = 2 * G::kChunks;
      u32x4 nx[4];
      read(0, 0, nx);
#pragma unroll
      for (int st = 0; st < kSteps; ++st) {
        const u32x4 a[4] = {nx[0], nx[1], nx[2], nx[3]};
        if (st + 1 < kSteps) read((st + 1) / G::kChunks, (st + 1) % G::kChunks, nx);
        step(st / G::kChunks, st % G::kChunks, a);
      }
    } else {
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int kk = 0; kk < G::kChunks; ++kk) {
          u32x4 a[4];
          read(sb, kk, a);
          step(sb, kk, a);
        }
    }
  };
  // s holds exponents s*tau*log2e - L*log2e (masked entries -inf)
  auto elementwise = [&]() {
#pragma unroll
    for (int mb = 0; mb < MR; ++mb) {
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = fast_exp2(s[sb][mb][r]);
          const float fv = f[sb][mb][r] * scale;
          const float dd = dp[sb][mb][r];                         // dP - D
          const int i = 4 * sb + r;
          if constexpr (kThree) {
            // Pt with alpha known; fPF carries P h (h = F - alpha) here
            const float pt = __builtin_fmaf(-arow[mb], dd + drow[mb], __builtin_fmaf(fv, dd, cc[sb][mb][r]));
            const float ppt = p * pt;
            e0[mb] += ppt;
            fPF[mb].set(i, p * (fv - arow[mb]));
            fPPt[mb].set(i, ppt);
          } else {
            const float pt0 = __builtin_fmaf(fv, dd, cc[sb][mb][r]);
            const float pf = p * fv;
            const float ppt = p * pt0;
            alpha[mb] += pf;
            e0[mb] += ppt;
            fPF[mb].set(i, pf);
            fPPt[mb].set(i, ppt);
          }
          fP[mb].set(i, p);
          fPdd[mb].set(i, p * dd);
          if constexpr (kForm == kSixAcc) fPdp[mb].set(i, p * (dd + drow[mb]));
        }
    }
  };
  // accumulate: Acc^T[dim][t] += X^T[dim][s] T^T[s][t]
  // With kPF the step's transposed operand fragments are read one 16-dim
  // block ahead of the MFMAs that use them (block 0 before the elementwise
  // step), so the LDS latency of each block's reads overlaps the previous
  // block's MFMAs; it costs 16 registers (4 fragments).
  using AF = typename E::AFrag;
  auto load_frags = [&](const T FB_LDS* Ks, int nb, AF (&f)[4]) {
#pragma unroll
    for (int t = 0; t < 4; ++t) f[t] = G::load_afrag(Ks + t * G::kTileElems, 16 * (nb0 + nb));
  };
  auto accumulate = [&](const T FB_LDS* Ks, AF (&cur)[4]) {
#pragma unroll
    for (int nb = 0; nb < kNBh; ++nb) {
      AF ak, av, auk, auv;
      if constexpr (kPF) {
        ak = cur[0];
        av = cur[1];
        auk = cur[2];
        auv = cur[3];
        if (nb + 1 < kNBh) load_frags(Ks, nb + 1, cur);
      } else {
        ak = G::load_afrag(Ks, 16 * (nb0 + nb));
        av = G::load_afrag(Ks + G::kTileElems, 16 * (nb0 + nb));
        auk = G::load_afrag(Ks + 2 * G::kTileElems, 16 * (nb0 + nb));
        auv = G::load_afrag(Ks + 3 * G::kTileElems, 16 * (nb0 + nb));
      }
#pragma unroll
      for (int mb = 0; mb < MR; ++mb) {
        aB[nb][mb] = E::mma_acc(ak, fP[mb], aB[nb][mb]);
        if constexpr (kForm == kSixAcc) aR[nb][mb] = E::mma_acc(ak, fPdp[mb], aR[nb][mb]);
        aOM[nb][mb] = E::mma_acc(ak, fPPt[mb], aOM[nb][mb]);
        aOM[nb][mb] = E::mma_acc(auk, fPdd[mb], aOM[nb][mb]);
        aDO[nb][mb] = E::mma_acc(auv, fP[mb], aDO[nb][mb]);
        aDO[nb][mb] = E::mma_acc(av, fPF[mb], aDO[nb][mb]);
      }
    }
  };

  const T* const src[4] = {K + kvoff, V + kvoff, UK + kvoff, UV + kvoff};
  const int nT = (N + kBS - 1) / kBS;
  const int it_end = causal ? min(nT, (min(rb * BR + BR, N) - 1) / kBS + 1) : nT;
  const TileCopy<T, D, NW, 4> copy(wave_id());
  stream_loop<NSTAGE, tile_loads<T, D, NW, 4>()>(
      0, it_end,
      [&](int it, int st) { copy.issue(src, (T FB_LDS*)lds[st], it * kBS, N); },
      [&](int it, int st) {
        const int s0 = it * kBS;
        const int mode = tile_mode_rowmajor(s0, row0, row0 + 16 * MR - 1, N, causal != 0);
        if (mode == 0) return;
        const T FB_LDS* Ks = (const T FB_LDS*)lds[st];
        // bf16 d = 128: LLVM's exp-interleave scheduling strategy for the tile
        // (Pass 1 1.1-1.5% faster; slower at d = 64)
        if constexpr (std::is_same_v<T, bf16> && D == 128) __builtin_amdgcn_iglp_opt(3);
        score(Ks);
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int mb = 0; mb < MR; ++mb)
#pragma unroll
            for (int r = 0; r < 4; ++r) s[sb][mb][r] = __builtin_fmaf(s[sb][mb][r], c, -lb[mb]);
        AF f0[4];
        if constexpr (kPF) load_frags(Ks, 0, f0);
        if (mode == 2) mask_tile<true>(s, s0, row0 + j, N, causal != 0);
        elementwise();
        accumulate(Ks, f0);
      });

  // epilogue (eq. 8; for kAlphaGiven the delayed E correction alone)
#pragma unroll
  for (int mb = 0; mb < MR; ++mb) {
    const int row = row0 + 16 * mb + j;
    if constexpr (kThree) {
      const float ee = group_sum(e0[mb]);
      if (row < N) {
        if (g == 0 && write_scalars) E_out[soff + row] = ee;
#pragma unroll
        for (int nb = 0; nb < kNBh; ++nb) {
          const int64_t off = hoff + (int64_t)row * D + 16 * (nb0 + nb) + 4 * g;
          E::store4(dOt + off, aDO[nb][mb]);
          E::store4(Qt + off, scale * (aOM[nb][mb] - ee * aB[nb][mb]));
        }
      }
      continue;
    }
    const float al = group_sum(alpha[mb]);
    const float e0s = group_sum(e0[mb]);
    const float ee = e0s - al * drow[mb];
    if (row < N) {
      if (g == 0 && write_scalars) {
        alpha_out[soff + row] = al;
        E_out[soff + row] = ee;
      }
#pragma unroll
      for (int nb = 0; nb < kNBh; ++nb) {
        const int64_t off = hoff + (int64_t)row * D + 16 * (nb0 + nb) + 4 * g;
        const floatx4 o = E::load4(O + off);
        E::store4(dOt + off, aDO[nb][mb] - al * o);
        if (kDQ) {
          const floatx4 dq = E::load4(dQ + off);
          E::store4(Qt + off, scale * (aOM[nb][mb] - e0s * aB[nb][mb]) - al * dq);
        } else {
          E::store4(Qt + off, scale * (aOM[nb][mb] - al * aR[(kForm == kSixAcc) ? nb : 0][mb] - ee * aB[nb][mb]));
        }
      }
    }
  }
}

// ===========================================================================
// First sweep of the three-pass control schedule (App. "Three-pass versus
// two-pass", the sweep that the affine fusion of Prop. 3.1 removes): row-major,
// alpha_i = sum_j P_ij F_ij only.  Stationary: Q, U_Q rows.  Streamed: K, U_K
// tiles.  Per tile: S^T = K Q^T, F^T = tau (K U_Q^T + U_K Q^T) and the row
// sum of P F; no accumulate contractions.  Writes alpha once.
// ===========================================================================
template <typename T, int D, int MR, int NW, int OCC, int NSTAGE>
__global__ __launch_bounds__(NW * 64, OCC) void bob3_alpha_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ UQ,
    const T* __restrict__ UK, const float* __restrict__ L, float* __restrict__ alpha_out, int N, int nRB,
    int total, float scale, int causal, int grp) {
  using E = Elt<T>;
  using G = Geo<T, D>;
  constexpr int BR = 16 * MR * NW;
  __shared__ __attribute__((aligned(16))) T lds[NSTAGE][2 * G::kTileElems];

  int bh, rb;
  map_block(nRB, total, bh, rb, causal != 0);
  const int64_t hoff = (int64_t)bh * N * D;
  const int64_t soff = (int64_t)bh * N;
  const int64_t kvoff = (int64_t)(bh / grp) * N * D;  // key/value head of this query head
  const int l = lane_id(), g = l >> 4, j = l & 15;
  (void)l;
  const int row0 = rb * BR + wave_id() * 16 * MR;

  u32x4 qf[MR][G::kChunks], uqf[MR][G::kChunks];
  float lb[MR], alpha[MR];
#pragma unroll
  for (int mb = 0; mb < MR; ++mb) {
    const int row = row0 + 16 * mb + j;
    load_stationary<T, D>(qf[mb], Q + hoff, row, N);
    load_stationary<T, D>(uqf[mb], UQ + hoff, row, N);
    lb[mb] = row < N ? L[soff + row] * kLog2e : 0.f;
    alpha[mb] = 0.f;
  }
  const float c = scale * kLog2e;
  floatx4 s[2][MR], f[2][MR];

  const T* const src[2] = {K + kvoff, UK + kvoff};
  const int nT = (N + kBS - 1) / kBS;
  const int it_end = causal ? min(nT, (min(rb * BR + BR, N) - 1) / kBS + 1) : nT;
  const TileCopy<T, D, NW, 2> copy(wave_id());
  stream_loop<NSTAGE, tile_loads<T, D, NW, 2>()>(
      0, it_end,
      [&](int it, int st) { copy.issue(src, (T FB_LDS*)lds[st], it * kBS, N); },
      [&](int it, int st) {
        const int s0 = it * kBS;
        const int mode = tile_mode_rowmajor(s0, row0, row0 + 16 * MR - 1, N, causal != 0);
        if (mode == 0) return;
        const T FB_LDS* Ks = (const T FB_LDS*)lds[st];
        const T FB_LDS* UKs = Ks + G::kTileElems;
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int mb = 0; mb < MR; ++mb) s[sb][mb] = f[sb][mb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int kk = 0; kk < G::kChunks; ++kk) {
            const int off = G::chunk_off(16 * sb + j, 4 * kk + g);
            const u32x4 ak = *(const u32x4 FB_LDS*)(Ks + off);
            const u32x4 auk = *(const u32x4 FB_LDS*)(UKs + off);
#pragma unroll
            for (int mb = 0; mb < MR; ++mb) {
              s[sb][mb] = E::mma_chunk(ak, qf[mb][kk], s[sb][mb]);      // S^T = K Q^T
              f[sb][mb] = E::mma_chunk(ak, uqf[mb][kk], f[sb][mb]);     // (U_Q K^T)^T
              f[sb][mb] = E::mma_chunk(auk, qf[mb][kk], f[sb][mb]);     // + (Q U_K^T)^T
            }
          }
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int mb = 0; mb < MR; ++mb)
#pragma unroll
            for (int r = 0; r < 4; ++r) s[sb][mb][r] = __builtin_fmaf(s[sb][mb][r], c, -lb[mb]);
        if (mode == 2) mask_tile<true>(s, s0, row0 + j, N, causal != 0);
#pragma unroll
        for (int mb = 0; mb < MR; ++mb)
#pragma unroll
          for (int sb = 0; sb < 2; ++sb)
#pragma unroll
            for (int r = 0; r < 4; ++r) alpha[mb] = __builtin_fmaf(fast_exp2(s[sb][mb][r]), f[sb][mb][r], alpha[mb]);
      });
#pragma unroll
  for (int mb = 0; mb < MR; ++mb) {
    const int row = row0 + 16 * mb + j;
    const float al = group_sum(alpha[mb]) * scale;
    if (row < N && g == 0) alpha_out[soff + row] = al;
  }
}

// ===========================================================================
// BoB Pass 2 (column-major; Alg. 1/2 Pass 2).  Stationary: K, V, U_K, U_V
// rows.  Streamed: Q, U_Q, dO tiles with L, D, alpha, E.  Per tile:
//   h = F - alpha, dS = P (dP - D), Pt = C + F (dP - D) - alpha dP,
//   St = P (Pt - E);  Vt += (P h)^T dO,  Kt += tau (St^T Q + dS^T U_Q).
// Writes Kt, Vt once; no atomics.  Wave sets (KS) as in the column side of
// the first backward.  With kParts each column block is split over nparts
// workgroups, which store fp32 partial sums of Kt / tau and Vt / tau to
// parts_out ([nparts][2][B*Hkv][N][d]; bob_column_parts_reduce_kernel adds
// them); the grid then holds total * nparts jobs (map_column_job).
// ===========================================================================
template <typename T, int D, int MC, int NW, int OCC, int NSTAGE, bool kGQA, int KS, bool kPF,
          bool kParts = false, bool kFlush = false>
__global__ __launch_bounds__(KS * NW * 64, OCC) void bob_pass2_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    const T* __restrict__ dO, const T* __restrict__ UQ, const T* __restrict__ UK,
    const T* __restrict__ UV, const float* __restrict__ L, const float* __restrict__ Dv,
    const float* __restrict__ alpha_in, const float* __restrict__ E_in,
    T* __restrict__ Kt, T* __restrict__ Vt, int N, int nRB, int total, float scale, int causal, int grp,
    float* __restrict__ parts_out = nullptr, int nparts = 1, int flush_tiles = 0) {
  static_assert(KS == 1 || KS == 2, "wave sets");
  using E = Elt<T>;
  using G = Geo<T, D>;
  constexpr int BC = 16 * MC * NW;
  // The tile ring, and the raw L, D, alpha, E of NSTAGE tiles with two slots
  // of transformed ones, in one LDS variable: with separate __shared__
  // arrays this compiler made the first read of the current ring stage wait
  // (s_waitcnt vmcnt(0)) for the asynchronous copy of the next tile, issued
  // just before into the other stage, which exposed that copy's latency on
  // every tile; with one variable the reads run on and the copy overlaps the
  // score phase (Pass 2 4% faster at d = 128).
  struct Smem2 {
    T lds[KS][NSTAGE][3 * G::kTileElems];
    float rawsc[KS][NSTAGE][4 * kBS];
    float tsc[KS][2][4 * kBS];
  };
  __shared__ __attribute__((aligned(16))) Smem2 sm;
  auto& lds = sm.lds;
  auto& rawsc = sm.rawsc;
  auto& tsc = sm.tsc;

  int bh, rb, part = 0;
  if constexpr (kParts)
    map_column_job(nRB, total, nparts, bh, rb, part);
  else
    map_block(nRB, total, bh, rb);
  const int64_t hoff = (int64_t)bh * N * D;
  const int l = lane_id(), g = l >> 4, j = l & 15;
  const int ks = KS == 1 ? 0 : wave_id() / NW;       // wave set
  const int wl = KS == 1 ? wave_id() : wave_id() % NW;  // wave within its set
  const int col0 = rb * BC + wl * 16 * MC;

  u32x4 kf[MC][G::kChunks], vf[MC][G::kChunks], ukf[MC][G::kChunks], uvf[MC][G::kChunks];
#pragma unroll
  for (int mc = 0; mc < MC; ++mc) {
    const int col = col0 + 16 * mc + j;
    load_stationary<T, D>(kf[mc], K + hoff, col, N);
    load_stationary<T, D>(vf[mc], V + hoff, col, N);
    load_stationary<T, D>(ukf[mc], UK + hoff, col, N);
    load_stationary<T, D>(uvf[mc], UV + hoff, col, N);
  }
  floatx4 aK[G::kNB][MC], aV[G::kNB][MC];
#pragma unroll
  for (int nb = 0; nb < G::kNB; ++nb)
#pragma unroll
    for (int mc = 0; mc < MC; ++mc) aK[nb][mc] = aV[nb][mc] = floatx4{0.f, 0.f, 0.f, 0.f};
  SectionSums<kFlush, G::kNB, MC> sect;
  sect.init();
  const float c = scale * kLog2e;
  floatx4 s[2][MC], dp[2][MC], f[2][MC], cc[2][MC];
  typename E::TFrag fPh[MC], fSt[MC], fdS[MC];

  // Transformed row scalars (tsc, per streamed row): T0 = -L log2e, T1 = -D,
  // T2 = -alpha / tau, T3 = -(alpha D + E).  The score MFMAs start from
  // T1, T2, T3, so they produce dd = dP - D, u = F / tau - alpha / tau and
  // C - (alpha D + E) directly, and with h = tau u and
  // Pt - E = tau u dd + C - (alpha D + E):
  //   P h = tau (p u),  St = p (tau u dd + cc),  dS = p dd.
  // The tau of P h is applied to Vt once, at the end.
  // s holds exponents s*tau*log2e - L*log2e (masked entries -inf).
  auto elementwise = [&]() {
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) {
          const float p = fast_exp2(s[sb][mc][r]);
          const float u = f[sb][mc][r];
          const float dd = dp[sb][mc][r];
          const int i = 4 * sb + r;
          fPh[mc].set(i, p * u);
          fSt[mc].set(i, p * __builtin_fmaf(scale, u * dd, cc[sb][mc][r]));
          fdS[mc].set(i, p * dd);
        }
      }
    }
  };

  const int nT = (N + kBS - 1) / kBS;
  const int it_begin = causal ? (rb * BC) / kBS : 0;
  const float inv_scale = 1.0f / scale;
  const int nTh = nT - it_begin;
  const StreamSplit<kGQA, KS, kParts> sp{it_begin, nTh, kGQA ? grp * nTh : nTh, ks, bh, grp, part, nparts};
  const TileCopy<T, D, NW, 3> copy(wl);
  stream_loop_rs<NSTAGE, tile_loads<T, D, NW, 3>(), 2>(
      sp.begin(), sp.end(nT), __builtin_amdgcn_readfirstlane(wl) == 0,
      [&](int it, int rs) {
        const int64_t qs = (int64_t)sp.qhead(it) * N;
        float FB_LDS* dst = (float FB_LDS*)rawsc[ks][rs];
        issue_scalar_pair(dst, L + qs, Dv + qs, sp.tile(it) * kBS, N);
        issue_scalar_pair(dst + 2 * kBS, alpha_in + qs, E_in + qs, sp.tile(it) * kBS, N);
      },
      [&](int it, int st) {
        const int64_t qo = (int64_t)sp.qhead(it) * N * D;
        const T* const src[3] = {Q + qo, UQ + qo, dO + qo};
        copy.issue(src, (T FB_LDS*)lds[ks][st], sp.tile(it) * kBS, N);
      },
      [&](int it, int rs, int ts) {
        (void)it;
        if (l < kBS) {
          const float FB_LDS* raw = (const float FB_LDS*)rawsc[ks][rs];
          float FB_LDS* t = (float FB_LDS*)tsc[ks][ts];
          const float Lr = raw[l], Dr = raw[kBS + l], ar = raw[2 * kBS + l], Er = raw[3 * kBS + l];
          t[l] = -Lr * kLog2e;
          t[kBS + l] = -Dr;
          t[2 * kBS + l] = -ar * inv_scale;
          t[3 * kBS + l] = -__builtin_fmaf(ar, Dr, Er);
        }
      },
      [&](int it, int st, int ts, auto&& prep_next) {
        const int s0 = sp.tile(it) * kBS;
        const int mode = sp.live(it) ? tile_mode_colmajor(s0, col0, col0 + 16 * MC - 1, N, causal != 0) : 0;
        if (mode == 0) {
          prep_next();
          return;
        }
        const T FB_LDS* Qs = (const T FB_LDS*)lds[ks][st];
        const T FB_LDS* UQs = Qs + G::kTileElems;
        const T FB_LDS* dOs = UQs + G::kTileElems;
        const float FB_LDS* Ts = (const float FB_LDS*)tsc[ks][ts];
        // score tiles [s = query][t = key], started from the row terms
#pragma unroll
        for (int sb = 0; sb < 2; ++sb) {
          const floatx4 t1 = *(const floatx4 FB_LDS*)(Ts + kBS + 16 * sb + 4 * g);
          const floatx4 t2 = *(const floatx4 FB_LDS*)(Ts + 2 * kBS + 16 * sb + 4 * g);
          const floatx4 t3 = *(const floatx4 FB_LDS*)(Ts + 3 * kBS + 16 * sb + 4 * g);
#pragma unroll
          for (int mc = 0; mc < MC; ++mc) {
            s[sb][mc] = floatx4{0.f, 0.f, 0.f, 0.f};
            dp[sb][mc] = t1;
            f[sb][mc] = t2;
            cc[sb][mc] = t3;
          }
        }
        // one score step: the five contractions of chunk kk of sub-block sb
        auto score_step = [&](int sb, int kk, u32x4 aq, u32x4 auq, u32x4 ado) {
#pragma unroll
          for (int mc = 0; mc < MC; ++mc) {
            s[sb][mc] = E::mma_chunk(aq, kf[mc][kk], s[sb][mc]);        // S = Q K^T
            dp[sb][mc] = E::mma_chunk(ado, vf[mc][kk], dp[sb][mc]);     // dP - D
            f[sb][mc] = E::mma_chunk(auq, kf[mc][kk], f[sb][mc]);       // (U_Q K^T
            f[sb][mc] = E::mma_chunk(aq, ukf[mc][kk], f[sb][mc]);       //  + Q U_K^T) - alpha / tau
            cc[sb][mc] = E::mma_chunk(ado, uvf[mc][kk], cc[sb][mc]);    // C - (alpha D + E)
          }
        };
        auto read_step = [&](int sb, int kk, u32x4 (&o)[3]) {
          const int off = G::chunk_off(16 * sb + j, 4 * kk + g);
          o[0] = *(const u32x4 FB_LDS*)(Qs + off);
          o[1] = *(const u32x4 FB_LDS*)(UQs + off);
          o[2] = *(const u32x4 FB_LDS*)(dOs + off);
        };
        // score MFMAs at raised wave priority, as in the first backward
        __builtin_amdgcn_s_setprio(1);
        if constexpr (kPF) {
          // operands of step st + 1 are read before the MFMAs of step st
          constexpr int kSteps = 2 * G::kChunks;
          u32x4 nx[3];
          read_step(0, 0, nx);
#pragma unroll
          for (int st = 0; st < kSteps; ++st) {
            const u32x4 aq = nx[0], auq = nx[1], ado = nx[2];
            if (st + 1 < kSteps) read_step((st + 1) / G::kChunks, (st + 1) % G::kChunks, nx);
            score_step(st / G::kChunks, st % G::kChunks, aq, auq, ado);
          }
        } else {
#pragma unroll
          for (int sb = 0; sb < 2; ++sb)
#pragma unroll
            for (int kk = 0; kk < G::kChunks; ++kk) {
              u32x4 a[3];
              read_step(sb, kk, a);
              score_step(sb, kk, a[0], a[1], a[2]);
            }
        }
        __builtin_amdgcn_s_setprio(0);
        prep_next();
#pragma unroll
        for (int sb = 0; sb < 2; ++sb) {
          const floatx4 t0 = *(const floatx4 FB_LDS*)(Ts + 16 * sb + 4 * g);
#pragma unroll
          for (int mc = 0; mc < MC; ++mc)
#pragma unroll
            for (int r = 0; r < 4; ++r) s[sb][mc][r] = __builtin_fmaf(s[sb][mc][r], c, t0[r]);
        }
        // with kPF the accumulate operands are read one 16-dim block ahead
        // of their MFMAs, as in Pass 1
        typename E::AFrag cur[3];
        if constexpr (kPF) {
#pragma unroll
          for (int t = 0; t < 3; ++t) cur[t] = G::load_afrag(Qs + t * G::kTileElems, 0);
        }
        if (mode == 2) mask_tile<false>(s, s0, col0 + j, N, causal != 0);
        elementwise();
#pragma unroll
        for (int nb = 0; nb < G::kNB; ++nb) {
          typename E::AFrag aq, auq, ado;
          if constexpr (kPF) {
            aq = cur[0];
            auq = cur[1];
            ado = cur[2];
            if (nb + 1 < G::kNB) {
#pragma unroll
              for (int t = 0; t < 3; ++t) cur[t] = G::load_afrag(Qs + t * G::kTileElems, 16 * (nb + 1));
            }
          } else {
            aq = G::load_afrag(Qs, 16 * nb);
            auq = G::load_afrag(UQs, 16 * nb);
            ado = G::load_afrag(dOs, 16 * nb);
          }
#pragma unroll
          for (int mc = 0; mc < MC; ++mc) {
            aV[nb][mc] = E::mma_acc(ado, fPh[mc], aV[nb][mc]);
            aK[nb][mc] = E::mma_acc(aq, fSt[mc], aK[nb][mc]);
            aK[nb][mc] = E::mma_acc(auq, fdS[mc], aK[nb][mc]);
          }
        }
        sect.step(aK, aV, flush_tiles);
      });
  sect.finish(aK, aV);
  if constexpr (KS == 2) {
    static_assert(sizeof(lds) >= (size_t)NW * G::kNB * MC * 1024, "set merge buffer");
    merge_wave_sets(aK, aV, ks, wl, (floatx4 FB_LDS*)&lds[0][0][0]);
    if (ks != 0) return;
  }
  if constexpr (kParts) {
    store_column_part<D>(parts_out, (int64_t)(total / nRB) * N * D, part, hoff, col0, N, aK, aV);
    return;
  }
#pragma unroll
  for (int mc = 0; mc < MC; ++mc) {
    const int col = col0 + 16 * mc + j;
    if (col < N) {
#pragma unroll
      for (int nb = 0; nb < G::kNB; ++nb) {
        const int64_t off = hoff + (int64_t)col * D + 16 * nb + 4 * g;
        E::store4(Kt + off, aK[nb][mc] * scale);
        E::store4(Vt + off, aV[nb][mc] * scale);
      }
    }
  }
}

// ===========================================================================
// BoB Pass 2 (as bob_pass2_kernel) in wave pairs, for head dims whose
// stationary rows and key-side sums do not fit one wave at two waves per
// SIMD (bf16 d = 256: K, V, U_K, U_V fragments and the Kt, Vt sums of 16
// key rows take 256 registers).  The two waves of a pair own the same 16
// key rows and split the head dims: half h holds dims [h D/2, (h+1) D/2) of
// the stationary rows and accumulates those dims of Kt and Vt.  Per streamed
// tile each wave forms partial score tiles over its dims (the row terms
// enter through half 0's start values only), hands its partial sums of
// sub-block 1 - h to the partner through LDS and adds the partner's partial
// sums of sub-block h, so that it holds the full score tiles of one 16-row
// sub-block.  It does the elementwise step there, hands its half of the
// bf16 accumulate fragments to the partner, and both accumulate their dims
// over all 32 streamed rows.  The two hand-overs add two workgroup-wide
// barriers per tile; every wave runs them on every tile, whatever its tile
// mode.  Waves p and p + NP form pair p; the workgroup owns 16 NP key rows.
// ===========================================================================
template <typename T, int D, int NP, bool kGQA>
__global__ __launch_bounds__(2 * NP * 64, 2) void bob_pass2_pair_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    const T* __restrict__ dO, const T* __restrict__ UQ, const T* __restrict__ UK,
    const T* __restrict__ UV, const float* __restrict__ L, const float* __restrict__ Dv,
    const float* __restrict__ alpha_in, const float* __restrict__ E_in,
    T* __restrict__ Kt, T* __restrict__ Vt, int N, int nRB, int total, float scale, int causal, int grp) {
  static_assert(sizeof(T) == 2, "bf16 only");
  using E = Elt<T>;
  using G = Geo<T, D>;
  constexpr int NW = 2 * NP;
  constexpr int BC = 16 * NP;
  constexpr int kHC = G::kChunks / 2;   // score steps (32-dim chunks) per half
  constexpr int kHB = G::kNB / 2;       // 16-dim output blocks per half
  struct SmemPair {
    T lds[2][3 * G::kTileElems];
    float rawsc[2][4 * kBS];
    float tsc[2][4 * kBS];
    floatx4 xs[NW][4][64];   // partial score tiles handed to the partner
    u32x2 xf[NW][3][64];     // half accumulate fragments handed to the partner
  };
  __shared__ __attribute__((aligned(16))) SmemPair sm;

  int bh, rb;
  map_block(nRB, total, bh, rb);
  const int64_t hoff = (int64_t)bh * N * D;
  const int l = lane_id(), g = l >> 4, j = l & 15;
  const int w = wave_id();
  const int pr = w % NP;
  const int col0 = rb * BC + 16 * pr;
  const int col = col0 + j;
  const float c = scale * kLog2e;
  const float inv_scale = 1.0f / scale;
  const int nT = (N + kBS - 1) / kBS;
  const int it_begin = causal ? (rb * BC) / kBS : 0;
  const int nTh = nT - it_begin;
  const StreamSplit<kGQA, 1> sp{it_begin, nTh, kGQA ? grp * nTh : nTh, 0, bh, grp};
  const TileCopy<T, D, NW, 3> copy(w);

  // The half is a compile-time constant inside run(), so every chunk, block
  // and fragment-slot index below is static; the branch is wave-uniform.
  auto run = [&](auto H) {
    constexpr int h = decltype(H)::value;
    const int partner = pr + NP * (1 - h);

    // this half's chunks of the stationary rows: chunk c = kHC h + kk
    u32x4 kf[kHC], vf[kHC], ukf[kHC], uvf[kHC];
#pragma unroll
    for (int kk = 0; kk < kHC; ++kk) {
      const int64_t off = hoff + (int64_t)col * D + (kHC * h + kk) * E::kKC + g * (E::kKC / 4);
      const bool in = col < N;
      kf[kk] = in ? *(const u32x4*)(K + off) : u32x4{0u, 0u, 0u, 0u};
      vf[kk] = in ? *(const u32x4*)(V + off) : u32x4{0u, 0u, 0u, 0u};
      ukf[kk] = in ? *(const u32x4*)(UK + off) : u32x4{0u, 0u, 0u, 0u};
      uvf[kk] = in ? *(const u32x4*)(UV + off) : u32x4{0u, 0u, 0u, 0u};
    }
    floatx4 aK[kHB], aV[kHB];
#pragma unroll
    for (int nb = 0; nb < kHB; ++nb) aK[nb] = aV[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
    stream_loop_rs<2, tile_loads<T, D, NW, 3>(), 2>(
        sp.begin(), sp.end(nT), __builtin_amdgcn_readfirstlane(w) == 0,
        [&](int it, int rs) {
          const int64_t qs = (int64_t)sp.qhead(it) * N;
          float FB_LDS* dst = (float FB_LDS*)sm.rawsc[rs];
          issue_scalar_pair(dst, L + qs, Dv + qs, sp.tile(it) * kBS, N);
          issue_scalar_pair(dst + 2 * kBS, alpha_in + qs, E_in + qs, sp.tile(it) * kBS, N);
        },
        [&](int it, int st) {
          const int64_t qo = (int64_t)sp.qhead(it) * N * D;
          const T* const src[3] = {Q + qo, UQ + qo, dO + qo};
          copy.issue(src, (T FB_LDS*)sm.lds[st], sp.tile(it) * kBS, N);
        },
        [&](int it, int rs, int ts) {
          (void)it;
          if (l < kBS) {
            const float FB_LDS* raw = (const float FB_LDS*)sm.rawsc[rs];
            float FB_LDS* t = (float FB_LDS*)sm.tsc[ts];
            const float Lr = raw[l], Dr = raw[kBS + l], ar = raw[2 * kBS + l], Er = raw[3 * kBS + l];
            t[l] = -Lr * kLog2e;
            t[kBS + l] = -Dr;
            t[2 * kBS + l] = -ar * inv_scale;
            t[3 * kBS + l] = -__builtin_fmaf(ar, Dr, Er);
          }
        },
        [&](int it, int st, int ts, auto&& prep_next) {
          const int s0 = sp.tile(it) * kBS;
          const int mode = tile_mode_colmajor(s0, col0, col0 + 15, N, causal != 0);
          const T FB_LDS* Qs = (const T FB_LDS*)sm.lds[st];
          const T FB_LDS* UQs = Qs + G::kTileElems;
          const T FB_LDS* dOs = UQs + G::kTileElems;
          const float FB_LDS* Ts = (const float FB_LDS*)sm.tsc[ts];
          // partial score tiles [s = query][t = key] over this half's dims;
          // half 0 starts from the row terms (as bob_pass2_kernel), half 1 from 0
          floatx4 s[2], dp[2], f[2], cc[2];
          if (mode != 0) {
            // score MFMAs at raised wave priority, as in bob_pass2_kernel
            __builtin_amdgcn_s_setprio(1);
#pragma unroll
            for (int sb = 0; sb < 2; ++sb) {
              s[sb] = floatx4{0.f, 0.f, 0.f, 0.f};
              if constexpr (h == 0) {
                dp[sb] = *(const floatx4 FB_LDS*)(Ts + kBS + 16 * sb + 4 * g);
                f[sb] = *(const floatx4 FB_LDS*)(Ts + 2 * kBS + 16 * sb + 4 * g);
                cc[sb] = *(const floatx4 FB_LDS*)(Ts + 3 * kBS + 16 * sb + 4 * g);
              } else {
                dp[sb] = f[sb] = cc[sb] = floatx4{0.f, 0.f, 0.f, 0.f};
              }
            }
#pragma unroll
            for (int sb = 0; sb < 2; ++sb)
#pragma unroll
              for (int kk = 0; kk < kHC; ++kk) {
                const int off = G::chunk_off(16 * sb + j, 4 * (kHC * h + kk) + g);
                const u32x4 aq = *(const u32x4 FB_LDS*)(Qs + off);
                const u32x4 auq = *(const u32x4 FB_LDS*)(UQs + off);
                const u32x4 ado = *(const u32x4 FB_LDS*)(dOs + off);
                s[sb] = E::mma_chunk(aq, kf[kk], s[sb]);        // S = Q K^T
                dp[sb] = E::mma_chunk(ado, vf[kk], dp[sb]);     // dP - D
                f[sb] = E::mma_chunk(auq, kf[kk], f[sb]);       // (U_Q K^T
                f[sb] = E::mma_chunk(aq, ukf[kk], f[sb]);       //  + Q U_K^T) - alpha / tau
                cc[sb] = E::mma_chunk(ado, uvf[kk], cc[sb]);    // C - (alpha D + E)
              }
            __builtin_amdgcn_s_setprio(0);
          }
          prep_next();
          // hand-over 1: the partner finishes sub-block 1 - h
          if (mode != 0) {
            floatx4 FB_LDS* out = (floatx4 FB_LDS*)&sm.xs[w][0][l];
            constexpr int ob = 1 - h;
            out[0] = s[ob];
            out[64] = dp[ob];
            out[128] = f[ob];
            out[192] = cc[ob];
          }
          __syncthreads();
          typename E::TFrag fPh, fSt, fdS;
          if (mode != 0) {
            const floatx4 FB_LDS* in = (const floatx4 FB_LDS*)&sm.xs[partner][0][l];
            floatx4 ts_ = s[h] + in[0], tdp = dp[h] + in[64], tf = f[h] + in[128], tcc = cc[h] + in[192];
            const floatx4 t0 = *(const floatx4 FB_LDS*)(Ts + 16 * h + 4 * g);
#pragma unroll
            for (int r = 0; r < 4; ++r) ts_[r] = __builtin_fmaf(ts_[r], c, t0[r]);
            if (mode == 2) {
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const int sr = s0 + 16 * h + 4 * g + r;
                const bool ok = sr < N && (causal == 0 || sr >= col);
                ts_[r] = ok ? ts_[r] : -INFINITY;
              }
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float pv = fast_exp2(ts_[r]);
              const float u = tf[r];
              const float dd = tdp[r];
              const int i = 4 * h + r;
              fPh.set(i, pv * u);
              fSt.set(i, pv * __builtin_fmaf(scale, u * dd, tcc[r]));
              fdS.set(i, pv * dd);
            }
            // hand-over 2: this half's slots of the three fragments
            u32x2 FB_LDS* outf = (u32x2 FB_LDS*)&sm.xf[w][0][l];
            const u32x4 a = __builtin_bit_cast(u32x4, fPh.v), b = __builtin_bit_cast(u32x4, fSt.v),
                        d = __builtin_bit_cast(u32x4, fdS.v);
            outf[0] = u32x2{a[2 * h], a[2 * h + 1]};
            outf[64] = u32x2{b[2 * h], b[2 * h + 1]};
            outf[128] = u32x2{d[2 * h], d[2 * h + 1]};
          }
          __syncthreads();
          if (mode != 0) {
            const u32x2 FB_LDS* inf = (const u32x2 FB_LDS*)&sm.xf[partner][0][l];
            constexpr int o = 2 * (1 - h);
            auto fill = [&](typename E::TFrag& fr, u32x2 x) {
              u32x4 v = __builtin_bit_cast(u32x4, fr.v);
              v[o] = x[0];
              v[o + 1] = x[1];
              fr.v = __builtin_bit_cast(bf16x8, v);
            };
            fill(fPh, inf[0]);
            fill(fSt, inf[64]);
            fill(fdS, inf[128]);
#pragma unroll
            for (int nb = 0; nb < kHB; ++nb) {
              const int dim0 = 16 * (kHB * h + nb);
              const typename E::AFrag aq = G::load_afrag(Qs, dim0);
              const typename E::AFrag auq = G::load_afrag(UQs, dim0);
              const typename E::AFrag ado = G::load_afrag(dOs, dim0);
              aV[nb] = E::mma_acc(ado, fPh, aV[nb]);
              aK[nb] = E::mma_acc(aq, fSt, aK[nb]);
              aK[nb] = E::mma_acc(auq, fdS, aK[nb]);
            }
          }
        });
    if (col < N) {
#pragma unroll
      for (int nb = 0; nb < kHB; ++nb) {
        const int64_t off = hoff + (int64_t)col * D + 16 * (kHB * h + nb) + 4 * g;
        E::store4(Kt + off, aK[nb] * scale);
        E::store4(Vt + off, aV[nb] * scale);
      }
    }
  };
  if (__builtin_amdgcn_readfirstlane(w) < NP)
    run(std::integral_constant<int, 0>{});
  else
    run(std::integral_constant<int, 1>{});
}

// Sum of the nparts fp32 partial planes of a split column kernel (plane
// elements each, laid out [nparts][2][plane]), in part order, times scale_k
// (first plane of each part, into Kt) or scale_v (second, into Vt), rounded
// to the output type.  Pass 2 stores Kt / tau and Vt / tau (both scales
// tau); the first backward stores dK / tau and dV (scales tau and 1).
// plane is a multiple of 4.
template <typename T>
__global__ __launch_bounds__(256) void bob_column_parts_reduce_kernel(const float* __restrict__ parts, int nparts,
                                                                      int64_t plane, float scale_k, float scale_v,
                                                                      T* __restrict__ Kt, T* __restrict__ Vt) {
  using E = Elt<T>;
  const int64_t n4 = plane / 4;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < 2 * n4; i += (int64_t)gridDim.x * blockDim.x) {
    const int t = i < n4 ? 0 : 1;
    const int64_t off = 4 * (i - t * n4);
    floatx4 acc = *(const floatx4*)(parts + t * plane + off);
    for (int q = 1; q < nparts; ++q) acc += *(const floatx4*)(parts + (2 * (int64_t)q + t) * plane + off);
    E::store4((t == 0 ? Kt : Vt) + off, acc * (t == 0 ? scale_k : scale_v));
  }
}

}  // namespace fb
