// Host side of libflashbob.so shared by its translation units: launch shapes,
// problem validation and the per-(dtype, head dim) launchers.  flashbob.hip
// holds the C ABI; fb_passes_d128.hip holds the bf16 d = 128 instances of the
// two BoB pass launchers, which are built with a different instruction
// scheduler (see that file), and every other unit refers to them through the
// extern template declarations at the end.
#pragma once
#include <algorithm>
#include <atomic>
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
// read the accumulate operands one block ahead (Pass 1 and Pass 2).
struct Shape {
  int mr, nw, occ, st, ds = 1, pf = 0;
};
template <typename T, int D> struct Cfg;
template <> struct Cfg<bf16, 32> {
  static constexpr Shape kFwd{2, 4, 2, 2}, kRows{2, 4, 2, 2}, kCols{2, 4, 2, 2};
  static constexpr Shape kP1{2, 4, 2, 2}, kP1Six{2, 4, 2, 2}, kP2{2, 2, 2, 2};
  static constexpr Shape kAlpha{2, 4, 2, 2};
};
template <> struct Cfg<bf16, 64> {
  static constexpr Shape kFwd{2, 8, 2, 2}, kRows{2, 4, 2, 2}, kCols{2, 4, 2, 2};
  static constexpr Shape kP1{1, 4, 2, 2}, kP1Six{1, 4, 2, 2}, kP2{2, 4, 2, 2};
  static constexpr Shape kAlpha{2, 4, 2, 2};
};
template <> struct Cfg<bf16, 128> {
  static constexpr Shape kFwd{1, 8, 2, 2}, kRows{2, 4, 2, 2}, kCols{1, 4, 2, 2};
  static constexpr Shape kP1{1, 8, 2, 2, 1, 1}, kP1Six{1, 8, 2, 3, 2}, kP2{1, 4, 2, 2, 1, 1};
  static constexpr Shape kAlpha{2, 4, 2, 2};
};
template <> struct Cfg<bf16, 256> {
  static constexpr Shape kFwd{1, 4, 2, 2}, kRows{1, 4, 2, 2}, kCols{1, 4, 1, 2};
  static constexpr Shape kP1{1, 4, 1, 2, 2}, kP1Six{1, 4, 1, 2, 2}, kP2{1, 4, 1, 2};
  static constexpr Shape kAlpha{1, 4, 2, 2};
};
template <> struct Cfg<float, 32> {
  static constexpr Shape kFwd{1, 4, 1, 2}, kRows{1, 4, 1, 2}, kCols{1, 4, 1, 2};
  static constexpr Shape kP1{1, 4, 1, 2}, kP1Six{1, 4, 1, 2}, kP2{1, 4, 2, 2};
  static constexpr Shape kAlpha{1, 4, 1, 2};
};
template <> struct Cfg<float, 64> {
  static constexpr Shape kFwd{1, 4, 1, 2}, kRows{1, 4, 1, 2}, kCols{1, 4, 1, 2};
  static constexpr Shape kP1{1, 4, 1, 2}, kP1Six{1, 4, 1, 2}, kP2{1, 4, 2, 2};
  static constexpr Shape kAlpha{1, 4, 1, 2};
};
template <> struct Cfg<float, 128> {
  static constexpr Shape kFwd{1, 4, 1, 2}, kRows{1, 4, 1, 2}, kCols{1, 4, 1, 2};
  static constexpr Shape kP1{1, 4, 1, 2}, kP1Six{1, 4, 1, 2}, kP2{1, 4, 1, 2};
  static constexpr Shape kAlpha{1, 4, 1, 2};
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

// Compute units of the current device (0 if it cannot be read), read once per
// device.
int device_cus();

// Column kernels (bwd cols, Pass 2) run two wave sets per workgroup when the
// grid has no more workgroups than the device has CUs (few key/value heads
// times few column blocks, e.g. multi-query attention): one 4-wave workgroup
// per CU leaves half of its wave slots empty, and the two sets split the
// streamed tiles instead.  That applies to shapes held to two waves per SIMD
// (a one-wave shape already fills a CU with one workgroup), and needs the two
// LDS rings (NTENS tiles and NSCAL row scalars per stage each) to fit a
// workgroup's 160 KB and the sets' merge buffer to fit in the rings.
// Whether a column kernel with this many workgroups runs two wave sets, from
// the mode set by bob_set_column_wave_sets (default: automatic).
bool use_two_sets(int workgroups);

template <typename T, int D, int MC, int NW, int OCC, int NSTAGE, int NTENS, int NSCAL>
constexpr bool two_sets_fit() {
  constexpr size_t ring = (size_t)NSTAGE * NTENS * Geo<T, D>::kTileElems * sizeof(T);
  constexpr size_t scal = (size_t)(NSTAGE + 2) * NSCAL * kBS * sizeof(float);
  return OCC == 2 && 2 * (ring + scal) <= 160 * 1024 &&
         2 * ring >= (size_t)NW * Geo<T, D>::kNB * MC * 1024;
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

template <typename T, int D>
int32_t launch_bwd(const Problem& p, const void* Q, const void* K, const void* V, const void* O,
                   const void* dO, const float* L, void* dQ, void* dK, void* dV, float* Dv,
                   hipStream_t s, float* parts_ws = nullptr, int parts = 1) {
  constexpr Shape cr = Cfg<T, D>::kRows, cc = Cfg<T, D>::kCols;
  const Grid gr = grid_for(p, 16 * cr.mr * cr.nw);
  (void)hipGetLastError();
  hipLaunchKernelGGL((attn_bwd_rows_kernel<T, D, cr.mr, cr.nw, cr.occ, cr.st>), dim3(gr.total), dim3(64 * cr.nw), 0, s,
                     (const T*)Q, (const T*)K, (const T*)V, (const T*)O, (const T*)dO, L, (T*)dQ, Dv,
                     (int)p.N, gr.nRB, gr.total, p.scale, p.causal, group(p));
  int32_t rc = finish_launch();
  if (rc != BOB_OK) return rc;
  const Grid gc = grid_for(p, 16 * cc.mr * cc.nw, true);
  const bool two = use_two_sets(gc.total);
  (void)hipGetLastError();
  if (parts > 1) {
    // each column block split over `parts` workgroups, then one reduction
    hipLaunchKernelGGL((attn_bwd_cols_kernel<T, D, cc.mr, cc.nw, cc.occ, cc.st, true, 1, true>),
                       dim3(gc.total * parts), dim3(64 * cc.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V,
                       (const T*)dO, L, (const float*)Dv, (T*)dK, (T*)dV, (int)p.N, gc.nRB, gc.total, p.scale,
                       p.causal, group(p), parts_ws, parts);
    const int64_t plane = p.B * p.Hkv * p.N * p.d;
    const int blocks = (int)std::min<int64_t>((plane / 2 + 255) / 256, 4096);
    hipLaunchKernelGGL((bob_column_parts_reduce_kernel<T>), dim3(blocks), dim3(256), 0, s, (const float*)parts_ws,
                       parts, plane, p.scale, 1.0f, (T*)dK, (T*)dV);
    return finish_launch();
  }
  auto cols = [&](auto gqa, auto ks) {
    hipLaunchKernelGGL((attn_bwd_cols_kernel<T, D, cc.mr, cc.nw, cc.occ, cc.st, decltype(gqa)::value, decltype(ks)::value>),
                       dim3(gc.total), dim3(64 * cc.nw * decltype(ks)::value), 0, s, (const T*)Q, (const T*)K, (const T*)V,
                       (const T*)dO, L, (const float*)Dv, (T*)dK, (T*)dV, (int)p.N, gc.nRB, gc.total, p.scale,
                       p.causal, group(p));
  };
  const bool gqa = group(p) != 1;
  if constexpr (two_sets_fit<T, D, cc.mr, cc.nw, cc.occ, cc.st, 2, 2>()) {
    if (two) {
      gqa ? cols(std::true_type{}, std::integral_constant<int, 2>{}) : cols(std::false_type{}, std::integral_constant<int, 2>{});
      return finish_launch();
    }
  }
  gqa ? cols(std::true_type{}, std::integral_constant<int, 1>{}) : cols(std::false_type{}, std::integral_constant<int, 1>{});
  return finish_launch();
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
    hipLaunchKernelGGL((bob_pass1_kernel<T, D, c.mr, c.nw, c.occ, c.st, kWithDQ, c.ds, c.pf != 0>), dim3(g.total, c.ds),
                       dim3(64 * c.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V, (const T*)O,
                       (const T*)dO, (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, (const T*)dQ,
                       (const float*)nullptr, (T*)Qt, (T*)dOt, alpha, E, (int)p.N, g.nRB, g.total, p.scale,
                       p.causal, group(p));
  } else {
    constexpr Shape c = Cfg<T, D>::kP1Six;
    const Grid g = grid_for(p, 16 * c.mr * c.nw);
    hipLaunchKernelGGL((bob_pass1_kernel<T, D, c.mr, c.nw, c.occ, c.st, kSixAcc, c.ds, c.pf != 0>), dim3(g.total, c.ds),
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
  hipLaunchKernelGGL((bob_pass1_kernel<T, D, c.mr, c.nw, c.occ, c.st, kAlphaGiven, c.ds, c.pf != 0>), dim3(g.total, c.ds),
                     dim3(64 * c.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V, (const T*)nullptr,
                     (const T*)dO, (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, (const T*)nullptr, alpha,
                     (T*)Qt, (T*)dOt, (float*)nullptr, E, (int)p.N, g.nRB, g.total, p.scale, p.causal, group(p));
  return finish_launch();
}

template <typename T, int D>
int32_t launch_pass2(const Problem& p, const void* Q, const void* K, const void* V, const void* dO,
                     const void* UQ, const void* UK, const void* UV, const float* L, const float* Dv,
                     const float* alpha, const float* E, void* Kt, void* Vt, hipStream_t s,
                     float* parts_ws = nullptr, int parts = 1) {
  constexpr Shape c = Cfg<T, D>::kP2;
  const Grid g = grid_for(p, 16 * c.mr * c.nw, true);
  (void)hipGetLastError();
  if (parts > 1) {
    // each column block split over `parts` workgroups, then one reduction
    hipLaunchKernelGGL((bob_pass2_kernel<T, D, c.mr, c.nw, c.occ, c.st, true, 1, c.pf != 0, true>),
                       dim3(g.total * parts), dim3(64 * c.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V,
                       (const T*)dO, (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, alpha, E, (T*)Kt, (T*)Vt,
                       (int)p.N, g.nRB, g.total, p.scale, p.causal, group(p), parts_ws, parts);
    const int64_t plane = p.B * p.Hkv * p.N * p.d;
    const int blocks = (int)std::min<int64_t>((plane / 2 + 255) / 256, 4096);
    hipLaunchKernelGGL((bob_column_parts_reduce_kernel<T>), dim3(blocks), dim3(256), 0, s, (const float*)parts_ws,
                       parts, plane, p.scale, p.scale, (T*)Kt, (T*)Vt);
    return finish_launch();
  }
  const bool two = use_two_sets(g.total);
  auto pass2 = [&](auto gqa, auto ks) {
    hipLaunchKernelGGL((bob_pass2_kernel<T, D, c.mr, c.nw, c.occ, c.st, decltype(gqa)::value, decltype(ks)::value, c.pf != 0>), dim3(g.total),
                       dim3(64 * c.nw * decltype(ks)::value), 0, s, (const T*)Q, (const T*)K, (const T*)V, (const T*)dO,
                       (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, alpha, E, (T*)Kt, (T*)Vt, (int)p.N,
                       g.nRB, g.total, p.scale, p.causal, group(p));
  };
  const bool gqa = group(p) != 1;
  if constexpr (two_sets_fit<T, D, c.mr, c.nw, c.occ, c.st, 3, 4>()) {
    if (two) {
      gqa ? pass2(std::true_type{}, std::integral_constant<int, 2>{}) : pass2(std::false_type{}, std::integral_constant<int, 2>{});
      return finish_launch();
    }
  }
  gqa ? pass2(std::true_type{}, std::integral_constant<int, 1>{}) : pass2(std::false_type{}, std::integral_constant<int, 1>{});
  return finish_launch();
}

// How many workgroups share a column block of the first backward's or Pass
// 2's column kernel (1: no split), from the mode set by
// bob_set_column_split, the kernel's column grid and the mask.
int column_parts(int workgroups, bool causal, bool pass2, int64_t iters_per_block);

// Streamed iterations of one column block: its group's query heads times
// 32-row query tiles (fewer under the causal mask).
inline int64_t column_iters(const Problem& p) { return (int64_t)group(p) * ((p.N + 31) / 32); }

template <typename T, int D>
int bwd_parts(const Problem& p) {
  constexpr Shape c = Cfg<T, D>::kCols;
  const Grid g = grid_for(p, 16 * c.mr * c.nw, true);
  const int parts = column_parts(g.total, p.causal != 0, false, column_iters(p));
  return (int64_t)g.total * parts > INT32_MAX ? 1 : parts;
}

template <typename T, int D>
int pass2_parts(const Problem& p) {
  constexpr Shape c = Cfg<T, D>::kP2;
  const Grid g = grid_for(p, 16 * c.mr * c.nw, true);
  const int parts = column_parts(g.total, p.causal != 0, true, column_iters(p));
  return (int64_t)g.total * parts > INT32_MAX ? 1 : parts;
}

// fp32 workspace of a split column kernel: parts x {Kt, Vt} (or {dK, dV})
// x B*Hkv*N*d.
inline int64_t column_workspace_bytes(const Problem& p, int parts) {
  return parts > 1 ? (int64_t)parts * 2 * p.B * p.Hkv * p.N * p.d * (int64_t)sizeof(float) : 0;
}

// Built in fb_passes_d128.hip.
extern template int32_t launch_pass1<bf16, 128>(const Problem&, const void*, const void*, const void*, const void*,
                                                const void*, const void*, const void*, const void*, const float*,
                                                const float*, const void*, void*, void*, float*, float*, hipStream_t);
extern template int32_t launch_pass2<bf16, 128>(const Problem&, const void*, const void*, const void*, const void*,
                                                const void*, const void*, const void*, const float*, const float*,
                                                const float*, const float*, void*, void*, hipStream_t, float*,
                                                int);

}  // namespace fb
