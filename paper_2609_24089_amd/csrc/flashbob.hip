// C ABI of libflashbob.so: argument validation and kernel dispatch.
// The entry points are declared (and documented) in include/flashbob.h.
#include <atomic>
#include <cmath>
#include <cstdint>

#include "../../include/flashbob.h"
#include "fb_kernels.h"

namespace fb {
namespace {

// Launch shapes per (element type, head dim) and kernel: MR = 16-row MFMA
// blocks per wave, NW = waves per workgroup (a workgroup owns 16*MR*NW
// stationary rows), OCC = waves per SIMD the register budget is held to, ST =
// LDS pipeline stages (tiles in flight + 1), DS = workgroups that share one
// row block, each accumulating 1/DS of the head dims (Pass 1 only).
struct Shape {
  int mr, nw, occ, st, ds = 1;
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
  static constexpr Shape kP1{1, 8, 2, 2}, kP1Six{1, 8, 2, 3, 2}, kP2{1, 4, 2, 2};
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

bool aligned16(const void* p) { return p != nullptr && (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// H query heads per batch entry; Hkv key/value heads (H for multi-head
// attention, a divisor of H for grouped-query attention).
struct Problem {
  int32_t dtype;
  int64_t B, H, N, d;
  float scale;
  int32_t causal;
  int64_t Hkv;
};
int group(const Problem& p) { return (int)(p.H / p.Hkv); }

// (dtype, head dim) pairs built into the library: bf16 d = 32, 64, 128, 256;
// fp32 d = 32, 64, 128 (fp32 d = 256 would need twice the registers of bf16).
bool supported(int32_t dtype, int64_t d) {
  if (dtype == BOB_BF16) return d == 32 || d == 64 || d == 128 || d == 256;
  if (dtype == BOB_F32) return d == 32 || d == 64 || d == 128;
  return false;
}

// Returns BOB_OK to proceed, or an error; sets *empty for B*H*N == 0.
int32_t check_problem(const Problem& p, bool* empty) {
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
  // grid size: heads x row blocks must fit a 32-bit grid (smallest block is 64 rows)
  const int64_t heads = p.B * p.H;
  if (p.B > INT32_MAX || p.H > INT32_MAX || heads > INT32_MAX) return BOB_EINVAL;
  if (heads * ((p.N + 63) / 64) > INT32_MAX) return BOB_EINVAL;
  return BOB_OK;
}

int32_t check_ptrs(std::initializer_list<const void*> ptrs) {
  for (const void* q : ptrs)
    if (!aligned16(q)) return BOB_EINVAL;
  return BOB_OK;
}

int32_t finish_launch() { return hipGetLastError() == hipSuccess ? BOB_OK : BOB_ELAUNCH; }

struct Grid {
  int nRB, total;
};
// Row kernels run over the query heads, column kernels over the key/value heads.
Grid grid_for(const Problem& p, int rows_per_block, bool kv_heads = false) {
  Grid g;
  g.nRB = (int)((p.N + rows_per_block - 1) / rows_per_block);
  g.total = (int)(p.B * (kv_heads ? p.Hkv : p.H) * g.nRB);
  return g;
}

// Compute units of the current device (0 if it cannot be read), read once per
// device.
int device_cus() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 0;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Column kernels (bwd cols, Pass 2) run two wave sets per workgroup when the
// grid has no more workgroups than the device has CUs (few key/value heads
// times few column blocks, e.g. multi-query attention): one 4-wave workgroup
// per CU leaves half of its wave slots empty, and the two sets split the
// streamed tiles instead.  That applies to shapes held to two waves per SIMD
// (a one-wave shape already fills a CU with one workgroup), and needs the two
// LDS rings (NTENS tiles and NSCAL row scalars per stage each) to fit a
// workgroup's 160 KB and the sets' merge buffer to fit in the rings.
// 0: two sets whenever the grid has no more workgroups than the device has
// CUs; 1: never; 2: wherever the shape allows (bob_set_column_wave_sets).
std::atomic<int> g_wave_sets{0};
bool use_two_sets(int workgroups) {
  const int mode = g_wave_sets.load(std::memory_order_relaxed);
  if (mode == 1) return false;
  if (mode == 2) return true;
  return workgroups <= device_cus();
}

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
                   hipStream_t s) {
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
    hipLaunchKernelGGL((bob_pass1_kernel<T, D, c.mr, c.nw, c.occ, c.st, kWithDQ, c.ds>), dim3(g.total, c.ds),
                       dim3(64 * c.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V, (const T*)O,
                       (const T*)dO, (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, (const T*)dQ,
                       (const float*)nullptr, (T*)Qt, (T*)dOt, alpha, E, (int)p.N, g.nRB, g.total, p.scale,
                       p.causal, group(p));
  } else {
    constexpr Shape c = Cfg<T, D>::kP1Six;
    const Grid g = grid_for(p, 16 * c.mr * c.nw);
    hipLaunchKernelGGL((bob_pass1_kernel<T, D, c.mr, c.nw, c.occ, c.st, kSixAcc, c.ds>), dim3(g.total, c.ds),
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
  hipLaunchKernelGGL((bob_pass1_kernel<T, D, c.mr, c.nw, c.occ, c.st, kAlphaGiven, c.ds>), dim3(g.total, c.ds),
                     dim3(64 * c.nw), 0, s, (const T*)Q, (const T*)K, (const T*)V, (const T*)nullptr,
                     (const T*)dO, (const T*)UQ, (const T*)UK, (const T*)UV, L, Dv, (const T*)nullptr, alpha,
                     (T*)Qt, (T*)dOt, (float*)nullptr, E, (int)p.N, g.nRB, g.total, p.scale, p.causal, group(p));
  return finish_launch();
}

template <typename T, int D>
int32_t launch_pass2(const Problem& p, const void* Q, const void* K, const void* V, const void* dO,
                     const void* UQ, const void* UK, const void* UV, const float* L, const float* Dv,
                     const float* alpha, const float* E, void* Kt, void* Vt, hipStream_t s) {
  constexpr Shape c = Cfg<T, D>::kP2;
  const Grid g = grid_for(p, 16 * c.mr * c.nw, true);
  const bool two = use_two_sets(g.total);
  (void)hipGetLastError();
  auto pass2 = [&](auto gqa, auto ks) {
    hipLaunchKernelGGL((bob_pass2_kernel<T, D, c.mr, c.nw, c.occ, c.st, decltype(gqa)::value, decltype(ks)::value>), dim3(g.total),
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

// Dispatch on (dtype, d) to a templated launcher.
#define FB_DISPATCH(p, FN, ...)                                                  \
  do {                                                                           \
    if ((p).dtype == BOB_BF16 && (p).d == 32) return FN<fb::bf16, 32>(__VA_ARGS__);  \
    if ((p).dtype == BOB_BF16 && (p).d == 64) return FN<fb::bf16, 64>(__VA_ARGS__);  \
    if ((p).dtype == BOB_BF16 && (p).d == 128) return FN<fb::bf16, 128>(__VA_ARGS__); \
    if ((p).dtype == BOB_BF16 && (p).d == 256) return FN<fb::bf16, 256>(__VA_ARGS__); \
    if ((p).dtype == BOB_F32 && (p).d == 32) return FN<float, 32>(__VA_ARGS__);  \
    if ((p).dtype == BOB_F32 && (p).d == 64) return FN<float, 64>(__VA_ARGS__);  \
    if ((p).dtype == BOB_F32 && (p).d == 128) return FN<float, 128>(__VA_ARGS__); \
    return BOB_EUNSUPPORTED;                                                     \
  } while (0)

}  // namespace
}  // namespace fb

using fb::Problem;

extern "C" {

int32_t attn_fwd_lse(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale, int32_t causal,
                     const void* Q, const void* K, const void* V, void* O, float* L, void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, H};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, V, O, L});
  if (rc != BOB_OK) return rc;
  FB_DISPATCH(p, fb::launch_fwd, p, Q, K, V, O, L, (hipStream_t)stream);
}

int32_t attn_bwd(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale, int32_t causal,
                 const void* Q, const void* K, const void* V, const void* O, const void* dO,
                 const float* L, void* dQ, void* dK, void* dV, float* D, void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, H};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, V, O, dO, L, dQ, dK, dV, D});
  if (rc != BOB_OK) return rc;
  FB_DISPATCH(p, fb::launch_bwd, p, Q, K, V, O, dO, L, dQ, dK, dV, D, (hipStream_t)stream);
}

int32_t attn_bob_pass1_rows(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale, int32_t causal,
                            const void* Q, const void* K, const void* V, const void* O,
                            const void* dO, const void* gdQ, const void* gdK, const void* gdV,
                            const float* L, const float* D, const void* dQ, void* Qt, void* dOt,
                            float* alpha, float* E, void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, H};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, V, O, dO, gdQ, gdK, gdV, L, D, Qt, dOt, alpha, E});
  if (rc != BOB_OK) return rc;
  if (dQ != nullptr && !fb::aligned16(dQ)) return BOB_EINVAL;
  FB_DISPATCH(p, fb::launch_pass1, p, Q, K, V, O, dO, gdQ, gdK, gdV, L, D, dQ, Qt, dOt, alpha, E,
              (hipStream_t)stream);
}

int32_t attn_bob_pass2_cols(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale, int32_t causal,
                            const void* Q, const void* K, const void* V, const void* dO,
                            const void* gdQ, const void* gdK, const void* gdV, const float* L,
                            const float* D, const float* alpha, const float* E, void* Kt, void* Vt,
                            void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, H};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, Kt, Vt});
  if (rc != BOB_OK) return rc;
  FB_DISPATCH(p, fb::launch_pass2, p, Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, Kt, Vt,
              (hipStream_t)stream);
}

// Grouped key/value heads: as above with Hkv key/value heads shared by the H
// query heads (H a multiple of Hkv).
int32_t attn_fwd_lse_gqa(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d, float scale,
                         int32_t causal, const void* Q, const void* K, const void* V, void* O, float* L,
                         void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, Hkv};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, V, O, L});
  if (rc != BOB_OK) return rc;
  FB_DISPATCH(p, fb::launch_fwd, p, Q, K, V, O, L, (hipStream_t)stream);
}

int32_t attn_bwd_gqa(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d, float scale,
                     int32_t causal, const void* Q, const void* K, const void* V, const void* O, const void* dO,
                     const float* L, void* dQ, void* dK, void* dV, float* D, void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, Hkv};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, V, O, dO, L, dQ, dK, dV, D});
  if (rc != BOB_OK) return rc;
  FB_DISPATCH(p, fb::launch_bwd, p, Q, K, V, O, dO, L, dQ, dK, dV, D, (hipStream_t)stream);
}

int32_t attn_bob_pass1_rows_gqa(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                float scale, int32_t causal, const void* Q, const void* K, const void* V,
                                const void* O, const void* dO, const void* gdQ, const void* gdK,
                                const void* gdV, const float* L, const float* D, const void* dQ, void* Qt,
                                void* dOt, float* alpha, float* E, void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, Hkv};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, V, O, dO, gdQ, gdK, gdV, L, D, Qt, dOt, alpha, E});
  if (rc != BOB_OK) return rc;
  if (dQ != nullptr && !fb::aligned16(dQ)) return BOB_EINVAL;
  FB_DISPATCH(p, fb::launch_pass1, p, Q, K, V, O, dO, gdQ, gdK, gdV, L, D, dQ, Qt, dOt, alpha, E,
              (hipStream_t)stream);
}

int32_t attn_bob_pass2_cols_gqa(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                float scale, int32_t causal, const void* Q, const void* K, const void* V,
                                const void* dO, const void* gdQ, const void* gdK, const void* gdV,
                                const float* L, const float* D, const float* alpha, const float* E, void* Kt,
                                void* Vt, void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, Hkv};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, Kt, Vt});
  if (rc != BOB_OK) return rc;
  FB_DISPATCH(p, fb::launch_pass2, p, Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, Kt, Vt,
              (hipStream_t)stream);
}

int32_t attn_bob3_alpha_rows(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale,
                             int32_t causal, const void* Q, const void* K, const void* gdQ, const void* gdK,
                             const float* L, float* alpha, void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, H};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, gdQ, gdK, L, alpha});
  if (rc != BOB_OK) return rc;
  FB_DISPATCH(p, fb::launch_alpha3, p, Q, K, gdQ, gdK, L, alpha, (hipStream_t)stream);
}

int32_t attn_bob3_rows(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale, int32_t causal,
                       const void* Q, const void* K, const void* V, const void* dO, const void* gdQ,
                       const void* gdK, const void* gdV, const float* L, const float* D, const float* alpha,
                       void* Qt, void* dOt, float* E, void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, H};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, Qt, dOt, E});
  if (rc != BOB_OK) return rc;
  FB_DISPATCH(p, fb::launch_rows3, p, Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, Qt, dOt, E,
              (hipStream_t)stream);
}

int32_t bob_supported(int32_t dtype, int64_t d) {
  return fb::supported(dtype, d) ? 1 : 0;
}

const char* bob_status_string(int32_t status) {
  switch (status) {
    case BOB_OK: return "BOB_OK: success";
    case BOB_EINVAL: return "BOB_EINVAL: invalid argument (size, scale, dtype, or NULL/misaligned pointer)";
    case BOB_EUNSUPPORTED:
      return "BOB_EUNSUPPORTED: (dtype, head dim) not built; bf16 d = 32, 64, 128, 256; fp32 d = 32, 64, 128";
    case BOB_ELAUNCH: return "BOB_ELAUNCH: HIP kernel launch failed";
    default: return "unknown bob_status";
  }
}

const char* bob_version(void) { return "flashbob-gfx950 0.1"; }

int32_t bob_set_column_wave_sets(int32_t mode) {
  if (mode < 0 || mode > 2) return BOB_EINVAL;
  fb::g_wave_sets.store(mode, std::memory_order_relaxed);
  return BOB_OK;
}

}  // extern "C"
