// C ABI of libflashbob.so: argument validation and kernel dispatch.
// The entry points are declared (and documented) in include/flashbob.h.
#include <type_traits>

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

// The mode of bob_set_column_split (0 automatic, 1 never, 2..8 that many
// parts wherever the kernels run).
static std::atomic<int> g_split{0};
constexpr int kMaxParts = 8;

// Automatic choice, from interleaved timing at B1 H16 N16384 d128 bf16 with
// 1, 2, 4 and 16 key/value heads.  Causal: a column block's work grows with
// the query tiles at or below its diagonal, and splitting until there are
// about 8 jobs per CU made the heaviest block's share short enough to
// balance (Pass 2 and the first backward 1.3-2x faster with 1-4 key/value
// heads; no gain with 16).  Dense Pass 2: blocks are equal, and the only gain
// was filling both workgroup slots of each CU on a grid smaller than the CU
// count (6% with one key/value head, against two wave sets in one
// workgroup).  The dense first backward gained from the same 8 jobs per CU
// as the causal one (9-18% with 1 and 4 key/value heads).  Either kernel
// only splits blocks of at least 1024 streamed iterations (query heads per
// group x 32-row query tiles): on the causal B4 H12 problems at N = 2048 and
// 4096 (64 and 128 iterations), the parts' fp32 round trip through HBM cost
// more than the balance gained (up to 14% slower), while every gain above
// came from blocks of 2048 iterations or more.
int column_parts(int workgroups, bool causal, bool pass2, int64_t iters_per_block) {
  const int mode = g_split.load(std::memory_order_relaxed);
  if (mode >= 2) return mode;
  if (mode == 1 || workgroups <= 0 || iters_per_block < 1024) return 1;
  const int cus = device_cus();
  const bool fill_only = pass2 && !causal;
  if (cus <= 0 || (fill_only && workgroups > cus)) return 1;
  const int64_t target = (int64_t)(fill_only ? 2 : 8) * cus;
  const int64_t parts = (target + workgroups - 1) / workgroups;
  return parts < 2 ? 1 : (int)std::min<int64_t>(parts, kMaxParts);
}

// Parts of a validated, supported problem's column kernel: Pass 2's
// (pass2 = true) or the first backward's.
static int column_parts_of(const Problem& p, bool pass2) {
#define FB_PARTS(TT, DD) \
  if (p.dtype == (std::is_same<TT, float>::value ? BOB_F32 : BOB_BF16) && p.d == DD) \
    return pass2 ? pass2_parts<TT, DD>(p) : bwd_parts<TT, DD>(p);
  FB_PARTS(bf16, 32)
  FB_PARTS(bf16, 64)
  FB_PARTS(bf16, 128)
  FB_PARTS(bf16, 256)
  FB_PARTS(float, 32)
  FB_PARTS(float, 64)
  FB_PARTS(float, 128)
#undef FB_PARTS
  return 1;
}

// Workspace of a column kernel's split for the *_ws entry points (0 when
// it would not split, or for an empty or invalid problem).
static int64_t column_ws_bytes(const Problem& p, bool pass2) {
  bool empty;
  if (check_problem(p, &empty) != BOB_OK || empty) return 0;
  return column_workspace_bytes(p, column_parts_of(p, pass2));
}

// The workspace checks of a *_ws entry point for a valid, non-empty problem
// that splits into `parts` (> 1).
static int32_t check_workspace(const Problem& p, int parts, const void* ws, int64_t bytes) {
  if (ws == nullptr || bytes < column_workspace_bytes(p, parts) || check_ptrs({ws}) != BOB_OK) return BOB_EINVAL;
  return BOB_OK;
}

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

int64_t bob_pass2_workspace_bytes(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                  int32_t causal) {
  return fb::column_ws_bytes(Problem{dtype, B, H, N, d, 1.0f, causal, Hkv}, true);
}

int64_t bob_bwd_workspace_bytes(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                int32_t causal) {
  return fb::column_ws_bytes(Problem{dtype, B, H, N, d, 1.0f, causal, Hkv}, false);
}

int32_t attn_bwd_gqa_ws(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d, float scale,
                        int32_t causal, const void* Q, const void* K, const void* V, const void* O, const void* dO,
                        const float* L, void* dQ, void* dK, void* dV, float* D, void* workspace,
                        int64_t workspace_bytes, void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, Hkv};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, V, O, dO, L, dQ, dK, dV, D});
  if (rc != BOB_OK) return rc;
  const int parts = fb::column_parts_of(p, false);
  if (parts > 1 && (rc = fb::check_workspace(p, parts, workspace, workspace_bytes)) != BOB_OK) return rc;
  FB_DISPATCH(p, fb::launch_bwd, p, Q, K, V, O, dO, L, dQ, dK, dV, D, (hipStream_t)stream, (float*)workspace,
              parts);
}

int32_t attn_bob_pass2_cols_gqa_ws(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                   float scale, int32_t causal, const void* Q, const void* K, const void* V,
                                   const void* dO, const void* gdQ, const void* gdK, const void* gdV,
                                   const float* L, const float* D, const float* alpha, const float* E, void* Kt,
                                   void* Vt, void* workspace, int64_t workspace_bytes, void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, Hkv};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK || empty) return rc;
  rc = fb::check_ptrs({Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, Kt, Vt});
  if (rc != BOB_OK) return rc;
  const int parts = fb::column_parts_of(p, true);
  if (parts > 1 && (rc = fb::check_workspace(p, parts, workspace, workspace_bytes)) != BOB_OK) return rc;
  FB_DISPATCH(p, fb::launch_pass2, p, Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, Kt, Vt,
              (hipStream_t)stream, (float*)workspace, parts);
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

int32_t bob_set_column_split(int32_t parts) {
  if (parts < 0 || parts > fb::kMaxParts) return BOB_EINVAL;
  fb::g_split.store(parts, std::memory_order_relaxed);
  return BOB_OK;
}

}  // extern "C"
