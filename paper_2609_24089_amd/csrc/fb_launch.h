// Host side of libflashbob.so shared by its translation units: launch shapes,
// problem validation and the per-(dtype, head dim) launchers.  flashbob.hip
// holds the C ABI; fb_passes_d128.hip holds the bf16 d = 128 instances of the
// two BoB pass launchers, which are built with a different instruction
// scheduler (see that file), and every other unit refers to them through the
// extern template declarations at the end.
#pragma once
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <initializer_list>

#include "../../include/flashbob.h"
#include "fb_kernels.h"

namespace fb {

// Launch shapes per (element type, head dim) and kernel: MR = 16-row MFMA
// blocks per wave, NW = waves per workgroup (a workgroup owns 16*MR*NW
// stationary rows), OCC = waves per SIMD the register budget is held to, ST =
// LDS pipeline stages (tiles in flight + 1), DS = workgroups that share one
// row block, each accumulating 1/DS of the head dims (Pass 1 only), PF = 1 to
// read the accumulate operands one block ahead (Pass 1 and Pass 2; Pass 2
// then also reads its score operands one step ahead), 2 to also read Pass 1's
// score operands one step ahead.  KL = 1 keeps the first backward column
// kernel's stationary K rows in LDS instead of registers.
// kColsF and kP2F are the shapes of the column kernels' two-level
// (sectioned) accumulation for long streams (SectionSums), which holds a
// second set of key-side sums; mr = 0 where that form is not built.  kP2W
// is Pass 2 in wide workgroups (more waves sharing one copy of each streamed
// tile, one workgroup per CU), run on grids that fill the device without
// wave sets, parts or sections; mr = 0 where it is not built.  kP2P is Pass
// 2 in wave pairs that split the head dims (bob_pass2_pair_kernel, nw waves
// = nw / 2 pairs of 16 key rows), for head dims whose one-wave form holds
// one wave per SIMD; run where kP2W would be, dense or causal.
struct Shape {
  int mr, nw, occ, st, ds = 1, pf = 0, kl = 0;
};
constexpr Shape kNoForm{0, 1, 1, 2};
template <typename T, int D> struct Cfg;
template <> struct Cfg<bf16, 32> {
  static constexpr Shape kFwd{2, 4, 2, 2}, kRows{2, 4, 2, 2}, kCols{2, 4, 2, 2};
  static constexpr Shape kP1{1, 4, 3, 2}, kP1Six{2, 4, 2, 2}, kP2{2, 2, 2, 2};
  static constexpr Shape kAlpha{2, 4, 2, 2};
  static constexpr Shape kColsF{2, 4, 2, 2}, kP2F{2, 2, 2, 2}, kP2W = kNoForm, kP2P = kNoForm;
};
template <> struct Cfg<bf16, 64> {
  static constexpr Shape kFwd{2, 4, 2, 2}, kRows{2, 4, 2, 2}, kCols{2, 4, 2, 2, 1, 0, 1};
  static constexpr Shape kP1{1, 4, 2, 2}, kP1Six{1, 4, 2, 2}, kP2{2, 4, 2, 2};
  static constexpr Shape kAlpha{2, 4, 2, 2};
  static constexpr Shape kColsF{1, 4, 2, 2}, kP2F{1, 4, 3, 2}, kP2W = kNoForm, kP2P = kNoForm;
};
template <> struct Cfg<bf16, 128> {
  static constexpr Shape kFwd{2, 4, 2, 2}, kRows{2, 4, 2, 2}, kCols{2, 4, 2, 2, 1, 0, 1};
  static constexpr Shape kP1{1, 8, 2, 2, 1, 1}, kP1Six{1, 4, 1, 2}, kP2{1, 4, 2, 2, 1, 1};
  static constexpr Shape kAlpha{2, 4, 2, 2};
  static constexpr Shape kColsF{1, 4, 2, 2}, kP2F{1, 4, 1, 2, 1, 1}, kP2W{1, 8, 2, 2, 1, 1}, kP2P = kNoForm;
};
template <> struct Cfg<bf16, 256> {
  static constexpr Shape kFwd{1, 4, 2, 2}, kRows{1, 4, 2, 2}, kCols{1, 8, 2, 2, 1, 0, 1};
  static constexpr Shape kP1{1, 4, 1, 2}, kP1Six{1, 4, 1, 2, 2}, kP2{1, 4, 1, 2};
  static constexpr Shape kAlpha{1, 4, 2, 2};
  static constexpr Shape kColsF = kNoForm, kP2F = kNoForm, kP2W = kNoForm, kP2P{1, 8, 2, 2};
};
template <> struct Cfg<float, 32> {
  static constexpr Shape kFwd{1, 4, 1, 2}, kRows{1, 4, 1, 2}, kCols{1, 4, 1, 2};
  static constexpr Shape kP1{1, 4, 1, 2}, kP1Six{1, 4, 1, 2}, kP2{1, 4, 2, 2};
  static constexpr Shape kAlpha{1, 4, 1, 2};
  static constexpr Shape kColsF = kNoForm, kP2F = kNoForm, kP2W = kNoForm, kP2P = kNoForm;
};
template <> struct Cfg<float, 64> {
  static constexpr Shape kFwd{1, 4, 1, 2}, kRows{1, 4, 1, 2}, kCols{1, 4, 1, 2};
  static constexpr Shape kP1{1, 4, 1, 2}, kP1Six{1, 4, 1, 2}, kP2{1, 4, 2, 2};
  static constexpr Shape kAlpha{1, 4, 1, 2};
  static constexpr Shape kColsF = kNoForm, kP2F = kNoForm, kP2W = kNoForm, kP2P = kNoForm;
};
template <> struct Cfg<float, 128> {
  static constexpr Shape kFwd{1, 4, 1, 2}, kRows{1, 4, 1, 2}, kCols{1, 4, 1, 2};
  static constexpr Shape kP1{1, 4, 1, 2}, kP1Six{1, 4, 1, 2}, kP2{1, 4, 1, 2};
  static constexpr Shape kAlpha{1, 4, 1, 2};
  static constexpr Shape kColsF = kNoForm, kP2F = kNoForm, kP2W = kNoForm, kP2P = kNoForm;
};

constexpr int64_t kMaxN = int64_t(1) << 30;

inline bool aligned16(const void* p) { return p != nullptr && (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// H query heads per batch entry; Hkv key/value heads (H for multi-head
// attention, a divisor of H for grouped-query attention).
struct Problem {
  int32_t dtype;
  int64_t B, H, N, d;
  float scale;
  int32_t causal;
  int64_t Hkv;
};
inline int group(const Problem& p) { return (int)(p.H / p.Hkv); }

// (dtype, head dim) pairs built into the library: bf16 d = 32, 64, 128, 256;
// fp32 d = 32, 64, 128 (fp32 d = 256 would need twice the registers of bf16).
inline bool supported(int32_t dtype, int64_t d) {
  if (dtype == BOB_BF16) return d == 32 || d == 64 || d == 128 || d == 256;
  if (dtype == BOB_F32) return d == 32 || d == 64 || d == 128;
  return false;
}

// Returns BOB_OK to proceed, or an error; sets *empty for B*H*N == 0.
inline int32_t check_problem(const Problem& p, bool* empty) {
  *empty = false;
  if (p.dtype != BOB_F32 && p.dtype != BOB_BF16) return BOB_EINVAL;
  if (p.B < 0 || p.H < 0 || p.N < 0 || p.d < 1) return BOB_EINVAL;
  if (!std::isfinite(p.scale)) return BOB_EINVAL;
  if (p.causal != 0 && p.causal != 1) return BOB_EINVAL;
  if (p.Hkv < 0 || (p.H > 0 && (p.Hkv < 1 || p.H % p.Hkv != 0))) return BOB_EINVAL;
  if (!supported(p.dtype, p.d)) return BOB_EUNSUPPORTED;
  if (p.B == 0 || p.H == 0 || p.N == 0) {
    *empty = true;
    return BOB_OK;
  }
  if (p.N > kMaxN) return BOB_EINVAL;
  // 32-bit grid and loop counts: heads x row blocks (the smallest block is 64
  // rows) sizes the grid, and a column kernel streams up to H/Hkv heads of
  // ceil(N/32) tiles in one loop, so heads x 32-row tiles must fit an int
  const int64_t heads = p.B * p.H;
  if (p.B > INT32_MAX || p.H > INT32_MAX || heads > INT32_MAX) return BOB_EINVAL;
  if (heads * ((p.N + 31) / 32) > INT32_MAX) return BOB_EINVAL;
  return BOB_OK;
}

inline int32_t check_ptrs(std::initializer_list<const void*> ptrs) {
  for (const void* q : ptrs)
    if (!aligned16(q)) return BOB_EINVAL;
  return BOB_OK;
}

inline int32_t finish_launch() { return hipGetLastError() == hipSuccess ? BOB_OK : BOB_ELAUNCH; }

struct Grid {
  int nRB, total;
};
// Row kernels run over the query heads, column kernels over the key/value heads.
inline Grid grid_for(const Problem& p, int rows_per_block, bool kv_heads = false) {
  Grid g;
  g.nRB = (int)((p.N + rows_per_block - 1) / rows_per_block);
  g.total = (int)(p.B * (kv_heads ? p.Hkv : p.H) * g.nRB);
  return g;
}

// ---------------------------------------------------------------------------
// Column kernels (the first backward's dK, dV and Pass 2's Kt, Vt): how one
// problem's column blocks are laid out over workgroups.
//  * parts: workgroups per column block (kParts forms; 1 = unsplit).  Split,
//    each part stores fp32 partial sums to a caller's workspace and
//    bob_column_parts_reduce_kernel adds them.
//  * sets: wave sets per workgroup (KS = 2 fills a CU with one workgroup when
//    the grid has no more workgroups than the device has CUs; shapes held to
//    two waves per SIMD whose two LDS rings fit 160 KB and hold the merge
//    buffer).
//  * flush_tiles: streamed tiles per MFMA accumulation section (SectionSums;
//    0 = one chain over the whole stream), with the kColsF / kP2F shape.
// The caller's requests (bob_column_opts; 0 = automatic) are resolved here,
// deterministically from the problem and the device's CU count, so the
// workspace query and the call that uses the workspace agree.
// ---------------------------------------------------------------------------
constexpr int kMaxParts = 8;
// Automatic sections: a stream longer than kLongChain tiles per accumulator
// chain is cut into sections of kSectionTiles.  Measured on the zero column
// sums (B1 H1 d64 bf16): at chains of 16384 tiles the residual stays at the
// bf16 rounding floor (about 3e-3), at 32768 it is 8.8e-3 and at 65536
// 2.9e-2; in sections of 1024 it stays at the floor up to N = 2^22.
constexpr int64_t kLongChain = 16384;
constexpr int kSectionTiles = 1024;

struct ColumnOpts {
  int parts = 0, wave_sets = 0, flush_tiles = 0;
};
struct ColumnPlan {
  Grid g{0, 0};
  int parts = 1, sets = 1, flush_tiles = 0;
  bool wide = false;   // Pass 2 in the kP2W shape
  bool pairs = false;  // Pass 2 in wave pairs (kP2P)
};

// Compute units of the current device (0 if it cannot be read).
int device_cus();

// Automatic (requested = 0) or forced part count for a column grid of
// `workgroups` with `iters` streamed iterations per block.
int resolve_parts(int requested, int workgroups, bool causal, bool pass2, int64_t iters);

// Automatic (requested = 0: two sets when the grid has no more workgroups
// than the device has CUs) or forced (1, 2) wave sets.
inline bool resolve_two_sets(int requested, int workgroups) {
  if (requested == 1) return false;
  if (requested == 2) return true;
  return workgroups <= device_cus();
}

template <typename T, int D, int MC, int NW, int OCC, int NSTAGE, int NTENS, int NSCAL, bool KL = false>
constexpr bool two_sets_fit() {
  constexpr size_t ring = (size_t)NSTAGE * NTENS * Geo<T, D>::kTileElems * sizeof(T);
  constexpr size_t scal = (size_t)(NSTAGE + 2) * NSCAL * kBS * sizeof(float);
  constexpr size_t kst = KL ? (size_t)NW * Geo<T, D>::kTileElems * sizeof(T) : 0;  // shared by both sets
  return OCC == 2 && NW <= 4 && 2 * (ring + scal) + kst <= 160 * 1024 &&
         2 * ring >= (size_t)NW * Geo<T, D>::kNB * MC * 1024;
}

// Streamed iterations of one column block: its group's query heads times
// 32-row query tiles (the first block under the causal mask streams them all).
inline int64_t column_iters(const Problem& p) { return (int64_t)group(p) * ((p.N + 31) / 32); }

// fp32 workspace of a split column kernel: parts x {Kt, Vt} (or {dK, dV})
// x B*Hkv*N*d.
inline int64_t column_workspace_bytes(const Problem& p, int parts) {
  return parts > 1 ? (int64_t)parts * 2 * p.B * p.Hkv * p.N * p.d * (int64_t)sizeof(float) : 0;
}

template <typename T, int D, bool kPass2, bool kF>
struct ColumnShape {
  static constexpr Shape kS =
      kPass2 ? (kF ? Cfg<T, D>::kP2F : Cfg<T, D>::kP2) : (kF ? Cfg<T, D>::kColsF : Cfg<T, D>::kCols);
  static constexpr bool kTwoFit =
      kS.mr > 0 && two_sets_fit<T, D, kS.mr, kS.nw, kS.occ, kS.st, kPass2 ? 3 : 2, kPass2 ? 4 : 2, kS.kl != 0>();
};

// Plan of a validated, non-empty, supported problem.  BOB_EINVAL for a
// request out of range, BOB_EUNSUPPORTED for sections requested where the
// sectioned form is not built.
template <typename T, int D, bool kPass2>
int32_t plan_columns(const Problem& p, const ColumnOpts& o, ColumnPlan* out) {
  if (o.parts < 0 || o.parts > kMaxParts || o.wave_sets < 0 || o.wave_sets > 2 || o.flush_tiles < -1)
    return BOB_EINVAL;
  using S0 = ColumnShape<T, D, kPass2, false>;
  using SF = ColumnShape<T, D, kPass2, true>;
  auto fill = [&](const Shape& s, bool two_fit) {
    ColumnPlan c;
    c.g = grid_for(p, 16 * s.mr * s.nw, true);
    c.parts = resolve_parts(o.parts, c.g.total, p.causal != 0, kPass2, column_iters(p));
    if ((int64_t)c.g.total * c.parts > INT32_MAX) c.parts = 1;
    c.sets = (c.parts == 1 && two_fit && resolve_two_sets(o.wave_sets, c.g.total)) ? 2 : 1;
    return c;
  };
  ColumnPlan c = fill(S0::kS, S0::kTwoFit);
  int ft = o.flush_tiles;
  if (ft == 0) {
    const int64_t per = (int64_t)c.parts * c.sets;
    const int64_t chain = (column_iters(p) + per - 1) / per;
    ft = (SF::kS.mr > 0 && chain > kLongChain) ? kSectionTiles : -1;
  }
  if (ft > 0) {
    if (SF::kS.mr == 0) return BOB_EUNSUPPORTED;
    c = fill(SF::kS, SF::kTwoFit);
    c.flush_tiles = ft;
  }
  // Wide Pass 2 workgroups on dense grids that fill every CU with them
  // (under the causal mask the larger blocks balance worse), when the wave
  // sets are automatic: 3-4% faster at N = 16384, d = 128 with 16 and with 4
  // key/value heads, outputs bit for bit those of the narrow form (each wave
  // does the same arithmetic), which a forced wave_sets = 1 still runs.
  if constexpr (kPass2 && Cfg<T, D>::kP2W.mr > 0) {
    constexpr Shape w = Cfg<T, D>::kP2W;
    const int cus = device_cus();
    if (o.wave_sets == 0 && !p.causal && c.parts == 1 && c.sets == 1 && c.flush_tiles <= 0 && cus > 0) {
      const Grid gw = grid_for(p, 16 * w.mr * w.nw, true);
      if (gw.total >= cus) {
        c.g = gw;
        c.wide = true;
      }
    }
  }
  // Wave pairs where the one-wave Pass 2 holds one wave per SIMD, on the
  // same unsplit, single-set, one-section layouts (the pairs' column blocks
  // have the one-wave form's 16 key rows per pair).
  if constexpr (kPass2 && Cfg<T, D>::kP2P.mr > 0) {
    constexpr Shape q = Cfg<T, D>::kP2P;
    if (o.wave_sets == 0 && c.parts == 1 && c.sets == 1 && c.flush_tiles <= 0) {
      c.g = grid_for(p, 16 * (q.nw / 2), true);
      c.pairs = true;
    }
  }
  *out = c;
  return BOB_OK;
}

template <typename T, int D>
int32_t launch_fwd(const Problem& p, const void* Q, const void* K, const void* V, void* O, float* L,
                   hipStream_t s) {
  constexpr Shape c = Cfg<T, D>::kFwd;
  const Grid g = grid_for(p, 16 * c.mr * c.nw);
  (void)hipGetLastError();
  hipLaunchKernelGGL((attn_fwd_kernel<T, D, c.mr, c.nw, c.occ, c.st>), dim3(g.total), dim3(64 * c.nw), 0, s,
                     (const T*)Q, (const T*)K, (const T*)V, (T*)O, L, (int)p.N, g.nRB, g.total, p.scale, p.causal, group(p));
  return finish_launch();
}

template <typename T, int D, bool kF>
int32_t launch_bwd_cols(const Problem& p, const void* Q, const void* K, const void* V, const void* dO,
                        const float* L, const float* Dv, void* dK, void* dV, hipStream_t s, const ColumnPlan& cp,
                        float* parts_ws) {
  constexpr Shape cc = ColumnShape<T, D, false, kF>::kS;
  if constexpr (cc.mr == 0) {
    return BOB_EUNSUPPORTED;
  } else {
    const Grid& gc = cp.g;
    (void)hipGetLastError();
    if (cp.parts > 1) {
      // each column block split over cp.parts workgroups, then one reduction
      hipLaunchKernelGGL((attn_bwd_cols_kernel<T, D, cc.mr, cc.nw, cc.occ, cc.st, true, 1, true, kF, cc.kl != 0>),
                         dim3(gc.total * cp.parts), dim3(64 * cc.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V,
                         (const T*)dO, L, Dv, (T*)dK, (T*)dV, (int)p.N, gc.nRB, gc.total, p.scale, p.causal,
                         group(p), parts_ws, cp.parts, cp.flush_tiles);
      const int64_t plane = p.B * p.Hkv * p.N * p.d;
      const int blocks = (int)std::min<int64_t>((plane / 2 + 255) / 256, 4096);
      hipLaunchKernelGGL((bob_column_parts_reduce_kernel<T>), dim3(blocks), dim3(256), 0, s, (const float*)parts_ws,
                         cp.parts, plane, p.scale, 1.0f, (T*)dK, (T*)dV);
      return finish_launch();
    }
    auto cols = [&](auto gqa, auto ks) {
      hipLaunchKernelGGL((attn_bwd_cols_kernel<T, D, cc.mr, cc.nw, cc.occ, cc.st, decltype(gqa)::value,
                                               decltype(ks)::value, false, kF, cc.kl != 0>),
                         dim3(gc.total), dim3(64 * cc.nw * decltype(ks)::value), 0, s, (const T*)Q, (const T*)K,
                         (const T*)V, (const T*)dO, L, Dv, (T*)dK, (T*)dV, (int)p.N, gc.nRB, gc.total, p.scale,
                         p.causal, group(p), (float*)nullptr, 1, cp.flush_tiles);
    };
    const bool gqa = group(p) != 1;
    if constexpr (ColumnShape<T, D, false, kF>::kTwoFit) {
      if (cp.sets == 2) {
        gqa ? cols(std::true_type{}, std::integral_constant<int, 2>{})
            : cols(std::false_type{}, std::integral_constant<int, 2>{});
        return finish_launch();
      }
    }
    gqa ? cols(std::true_type{}, std::integral_constant<int, 1>{})
        : cols(std::false_type{}, std::integral_constant<int, 1>{});
    return finish_launch();
  }
}

// The first backward: the row kernel (dQ, D), then the column kernel (dK, dV)
// laid out by `cp` (plan_columns<T, D, false>); parts_ws is the caller's
// workspace when cp.parts > 1.
template <typename T, int D>
int32_t launch_bwd(const Problem& p, const void* Q, const void* K, const void* V, const void* O,
                   const void* dO, const float* L, void* dQ, void* dK, void* dV, float* Dv,
                   hipStream_t s, const ColumnPlan& cp, float* parts_ws) {
  constexpr Shape cr = Cfg<T, D>::kRows;
  const Grid gr = grid_for(p, 16 * cr.mr * cr.nw);
  (void)hipGetLastError();
  hipLaunchKernelGGL((attn_bwd_rows_kernel<T, D, cr.mr, cr.nw, cr.occ, cr.st>), dim3(gr.total), dim3(64 * cr.nw), 0, s,
                     (const T*)Q, (const T*)K, (const T*)V, (const T*)O, (const T*)dO, L, (T*)dQ, Dv,
                     (int)p.N, gr.nRB, gr.total, p.scale, p.causal, group(p));
  int32_t rc = finish_launch();
  if (rc != BOB_OK) return rc;
  if (cp.flush_tiles > 0)
    return launch_bwd_cols<T, D, true>(p, Q, K, V, dO, L, Dv, dK, dV, s, cp, parts_ws);
  return launch_bwd_cols<T, D, false>(p, Q, K, V, dO, L, Dv, dK, dV, s, cp, parts_ws);
}


template <typename T, int D>
int32_t launch_pass1(const Problem& p, const void* Q, const void* K, const void* V, const void* O,
                     const void* dO, const void* UQ, const void* UK, const void* UV, const float* L,
                     const float* Dv, const void* dQ, void* Qt, void* dOt, float* alpha, float* E,
                     hipStream_t s) {
  (void)hipGetLastError();
  if (dQ != nullptr) {
    constexpr Shape c = Cfg<T, D>::kP1;
    const Grid g = grid_for(p, 16 * c.mr * c.nw);
    hipLaunchKernelGGL((bob_pass1_kernel<T, D, c.mr, c.nw, c.occ, c.st, kWithDQ, c.ds, c.pf>), dim3(g.total, c.ds),
                       dim3(64 * c.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V, (const T*)O,
                       (const T*)dO, (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, (const T*)dQ,
                       (const float*)nullptr, (T*)Qt, (T*)dOt, alpha, E, (int)p.N, g.nRB, g.total, p.scale,
                       p.causal, group(p));
  } else {
    constexpr Shape c = Cfg<T, D>::kP1Six;
    const Grid g = grid_for(p, 16 * c.mr * c.nw);
    hipLaunchKernelGGL((bob_pass1_kernel<T, D, c.mr, c.nw, c.occ, c.st, kSixAcc, c.ds, c.pf>), dim3(g.total, c.ds),
                       dim3(64 * c.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V, (const T*)O,
                       (const T*)dO, (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, (const T*)nullptr,
                       (const float*)nullptr, (T*)Qt, (T*)dOt, alpha, E, (int)p.N, g.nRB, g.total, p.scale,
                       p.causal, group(p));
  }
  return finish_launch();
}

// Three-pass control schedule: the alpha-only sweep and the second row sweep.
template <typename T, int D>
int32_t launch_alpha3(const Problem& p, const void* Q, const void* K, const void* UQ, const void* UK,
                      const float* L, float* alpha, hipStream_t s) {
  constexpr Shape c = Cfg<T, D>::kAlpha;
  const Grid g = grid_for(p, 16 * c.mr * c.nw);
  (void)hipGetLastError();
  hipLaunchKernelGGL((bob3_alpha_kernel<T, D, c.mr, c.nw, c.occ, c.st>), dim3(g.total), dim3(64 * c.nw), 0, s,
                     (const T*)Q, (const T*)K, (const T*)UQ, (const T*)UK, L, alpha, (int)p.N, g.nRB, g.total,
                     p.scale, p.causal, group(p));
  return finish_launch();
}

template <typename T, int D>
int32_t launch_rows3(const Problem& p, const void* Q, const void* K, const void* V, const void* dO,
                     const void* UQ, const void* UK, const void* UV, const float* L, const float* Dv,
                     const float* alpha, void* Qt, void* dOt, float* E, hipStream_t s) {
  constexpr Shape c = Cfg<T, D>::kP1;
  const Grid g = grid_for(p, 16 * c.mr * c.nw);
  (void)hipGetLastError();
  hipLaunchKernelGGL((bob_pass1_kernel<T, D, c.mr, c.nw, c.occ, c.st, kAlphaGiven, c.ds, c.pf>), dim3(g.total, c.ds),
                     dim3(64 * c.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V, (const T*)nullptr,
                     (const T*)dO, (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, (const T*)nullptr, alpha,
                     (T*)Qt, (T*)dOt, (float*)nullptr, E, (int)p.N, g.nRB, g.total, p.scale, p.causal, group(p));
  return finish_launch();
}

template <typename T, int D, bool kF>
int32_t launch_pass2_form(const Problem& p, const void* Q, const void* K, const void* V, const void* dO,
                          const void* UQ, const void* UK, const void* UV, const float* L, const float* Dv,
                          const float* alpha, const float* E, void* Kt, void* Vt, hipStream_t s,
                          const ColumnPlan& cp, float* parts_ws) {
  constexpr Shape c = ColumnShape<T, D, true, kF>::kS;
  if constexpr (c.mr == 0) {
    return BOB_EUNSUPPORTED;
  } else {
    const Grid& g = cp.g;
    (void)hipGetLastError();
    if (cp.parts > 1) {
      // each column block split over cp.parts workgroups, then one reduction
      hipLaunchKernelGGL((bob_pass2_kernel<T, D, c.mr, c.nw, c.occ, c.st, true, 1, c.pf != 0, true, kF>),
                         dim3(g.total * cp.parts), dim3(64 * c.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V,
                         (const T*)dO, (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, alpha, E, (T*)Kt, (T*)Vt,
                         (int)p.N, g.nRB, g.total, p.scale, p.causal, group(p), parts_ws, cp.parts,
                         cp.flush_tiles);
      const int64_t plane = p.B * p.Hkv * p.N * p.d;
      const int blocks = (int)std::min<int64_t>((plane / 2 + 255) / 256, 4096);
      hipLaunchKernelGGL((bob_column_parts_reduce_kernel<T>), dim3(blocks), dim3(256), 0, s, (const float*)parts_ws,
                         cp.parts, plane, p.scale, p.scale, (T*)Kt, (T*)Vt);
      return finish_launch();
    }
    const bool gqa = group(p) != 1;
    if constexpr (!kF && Cfg<T, D>::kP2W.mr > 0) {
      constexpr Shape w = Cfg<T, D>::kP2W;
      auto wide = [&](auto kv) {
        hipLaunchKernelGGL((bob_pass2_kernel<T, D, w.mr, w.nw, w.occ, w.st, decltype(kv)::value, 1, w.pf != 0>),
                           dim3(g.total), dim3(64 * w.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V, (const T*)dO,
                           (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, alpha, E, (T*)Kt, (T*)Vt, (int)p.N,
                           g.nRB, g.total, p.scale, p.causal, group(p), (float*)nullptr, 1, 0);
      };
      if (cp.wide) {
        gqa ? wide(std::true_type{}) : wide(std::false_type{});
        return finish_launch();
      }
    }
    if constexpr (!kF && Cfg<T, D>::kP2P.mr > 0) {
      constexpr Shape q = Cfg<T, D>::kP2P;
      auto pairs = [&](auto kv) {
        hipLaunchKernelGGL((bob_pass2_pair_kernel<T, D, q.nw / 2, decltype(kv)::value>), dim3(g.total),
                           dim3(64 * q.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V, (const T*)dO,
                           (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, alpha, E, (T*)Kt, (T*)Vt, (int)p.N,
                           g.nRB, g.total, p.scale, p.causal, group(p));
      };
      if (cp.pairs) {
        gqa ? pairs(std::true_type{}) : pairs(std::false_type{});
        return finish_launch();
      }
    }
    auto pass2 = [&](auto gqa, auto ks) {
      hipLaunchKernelGGL((bob_pass2_kernel<T, D, c.mr, c.nw, c.occ, c.st, decltype(gqa)::value, decltype(ks)::value,
                                           c.pf != 0, false, kF>),
                         dim3(g.total), dim3(64 * c.nw * decltype(ks)::value), 0, s, (const T*)Q, (const T*)K,
                         (const T*)V, (const T*)dO, (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, alpha, E,
                         (T*)Kt, (T*)Vt, (int)p.N, g.nRB, g.total, p.scale, p.causal, group(p), (float*)nullptr, 1,
                         cp.flush_tiles);
    };
    if constexpr (ColumnShape<T, D, true, kF>::kTwoFit) {
      if (cp.sets == 2) {
        gqa ? pass2(std::true_type{}, std::integral_constant<int, 2>{})
            : pass2(std::false_type{}, std::integral_constant<int, 2>{});
        return finish_launch();
      }
    }
    gqa ? pass2(std::true_type{}, std::integral_constant<int, 1>{})
        : pass2(std::false_type{}, std::integral_constant<int, 1>{});
    return finish_launch();
  }
}

// Pass 2 laid out by `cp` (plan_columns<T, D, true>); parts_ws is the
// caller's workspace when cp.parts > 1.
template <typename T, int D>
int32_t launch_pass2(const Problem& p, const void* Q, const void* K, const void* V, const void* dO,
                     const void* UQ, const void* UK, const void* UV, const float* L, const float* Dv,
                     const float* alpha, const float* E, void* Kt, void* Vt, hipStream_t s, const ColumnPlan& cp,
                     float* parts_ws) {
  if (cp.flush_tiles > 0)
    return launch_pass2_form<T, D, true>(p, Q, K, V, dO, UQ, UK, UV, L, Dv, alpha, E, Kt, Vt, s, cp, parts_ws);
  return launch_pass2_form<T, D, false>(p, Q, K, V, dO, UQ, UK, UV, L, Dv, alpha, E, Kt, Vt, s, cp, parts_ws);
}

// Built in fb_passes_d128.hip.
extern template int32_t launch_pass1<bf16, 128>(const Problem&, const void*, const void*, const void*, const void*,
                                                const void*, const void*, const void*, const void*, const float*,
                                                const float*, const void*, void*, void*, float*, float*, hipStream_t);
extern template int32_t launch_pass2<bf16, 128>(const Problem&, const void*, const void*, const void*, const void*,
                                                const void*, const void*, const void*, const float*, const float*,
                                                const float*, const float*, void*, void*, hipStream_t,
                                                const ColumnPlan&, float*);

}  // namespace fb
