// C ABI of libflashbob.so: argument validation and kernel dispatch.
// The entry points are declared (and documented) in include/flashbob.h.
#include "fb_launch.h"

namespace fb {

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

// The mode of bob_set_column_wave_sets (0 automatic, 1 one set, 2 two sets).
static std::atomic<int> g_wave_sets{0};

bool use_two_sets(int workgroups) {
  const int mode = g_wave_sets.load(std::memory_order_relaxed);
  if (mode == 1) return false;
  if (mode == 2) return true;
  return workgroups <= device_cus();
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
