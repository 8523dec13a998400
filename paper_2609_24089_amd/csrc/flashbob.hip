// C ABI of libflashbob.so: argument validation and kernel dispatch.
// The entry points are declared (and documented) in include/flashbob.h.
#include <atomic>
#include <type_traits>

#include "fb_launch.h"

namespace fb {

// Compute units of the current device, read from the runtime on every call
// (the library keeps no state of its own).
int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 0;
  return n;
}

// Dispatch on (dtype, d) to a templated function.
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

// Automatic choice (requested = 0), from interleaved timing at B1 H16 N16384
// d128 bf16 with 1, 2, 4 and 16 key/value heads.  Causal: a column block's
// work grows with the query tiles at or below its diagonal, and splitting
// until there are about 8 jobs per CU made the heaviest block's share short
// enough to balance (Pass 2 and the first backward 1.3-2x faster with 1-4
// key/value heads; no gain with 16).  Dense Pass 2: blocks are equal, and the
// only gain was filling both workgroup slots of each CU on a grid smaller
// than the CU count (6% with one key/value head, against two wave sets in
// one workgroup).  The dense first backward gained from the same 8 jobs per
// CU as the causal one (9-18% with 1 and 4 key/value heads).  Either kernel
// only splits blocks of at least 1024 streamed iterations (query heads per
// group x 32-row query tiles): on the causal B4 H12 problems at N = 2048 and
// 4096 (64 and 128 iterations), the parts' fp32 round trip through HBM cost
// more than the balance gained (up to 14% slower), while every gain above
// came from blocks of 2048 iterations or more.  Requested 1..8: that many.
int resolve_parts(int requested, int workgroups, bool causal, bool pass2, int64_t iters) {
  if (requested >= 1) return requested;
  if (workgroups <= 0 || iters < 1024) return 1;
  const int cus = device_cus();
  const bool fill_only = pass2 && !causal;
  if (cus <= 0 || (fill_only && workgroups > cus)) return 1;
  const int64_t target = (int64_t)(fill_only ? 2 : 8) * cus;
  const int64_t parts = (target + workgroups - 1) / workgroups;
  return parts < 2 ? 1 : (int)std::min<int64_t>(parts, kMaxParts);
}

static ColumnOpts opts_of(const bob_column_opts* o) {
  ColumnOpts c;
  if (o != nullptr) {
    c.parts = o->parts;
    c.wave_sets = o->wave_sets;
    c.flush_tiles = o->flush_tiles;
  }
  return c;
}

// The plain (non-_ws) entry points never split a column block: they have no
// workspace.  Wave sets and sections are automatic.
constexpr ColumnOpts kUnsplit{1, 0, 0};

template <typename T, int D>
int32_t plan_bwd(const Problem& p, const ColumnOpts& o, ColumnPlan* c) {
  return plan_columns<T, D, false>(p, o, c);
}
template <typename T, int D>
int32_t plan_pass2(const Problem& p, const ColumnOpts& o, ColumnPlan* c) {
  return plan_columns<T, D, true>(p, o, c);
}

// Plan of a column kernel (pass2: Pass 2, else the first backward's) for a
// valid problem; an empty problem gets the trivial plan.
static int32_t column_plan(const Problem& p, bool pass2, const ColumnOpts& o, ColumnPlan* c) {
  bool empty;
  int32_t rc = check_problem(p, &empty);
  if (rc != BOB_OK) return rc;
  if (empty) {
    if (o.parts < 0 || o.parts > kMaxParts || o.wave_sets < 0 || o.wave_sets > 2 || o.flush_tiles < -1)
      return BOB_EINVAL;
    *c = ColumnPlan{};
    return BOB_OK;
  }
  if (pass2) FB_DISPATCH(p, plan_pass2, p, o, c);
  FB_DISPATCH(p, plan_bwd, p, o, c);
}

// The workspace checks of a *_ws entry point for a plan that splits.
static int32_t check_workspace(const Problem& p, const ColumnPlan& c, const void* ws, int64_t bytes) {
  if (c.parts <= 1) return BOB_OK;
  if (ws == nullptr || bytes < column_workspace_bytes(p, c.parts) || check_ptrs({ws}) != BOB_OK) return BOB_EINVAL;
  return BOB_OK;
}

static int32_t run_bwd(const Problem& p, const ColumnOpts& o, const void* Q, const void* K, const void* V,
                       const void* O, const void* dO, const float* L, void* dQ, void* dK, void* dV, float* D,
                       void* ws, int64_t ws_bytes, void* stream) {
  bool empty;
  int32_t rc = check_problem(p, &empty);
  if (rc != BOB_OK) return rc;
  ColumnPlan c;
  if ((rc = column_plan(p, false, o, &c)) != BOB_OK || empty) return rc;
  if ((rc = check_ptrs({Q, K, V, O, dO, L, dQ, dK, dV, D})) != BOB_OK) return rc;
  if ((rc = check_workspace(p, c, ws, ws_bytes)) != BOB_OK) return rc;
  FB_DISPATCH(p, launch_bwd, p, Q, K, V, O, dO, L, dQ, dK, dV, D, (hipStream_t)stream, c, (float*)ws);
}

static int32_t run_pass2(const Problem& p, const ColumnOpts& o, const void* Q, const void* K, const void* V,
                         const void* dO, const void* gdQ, const void* gdK, const void* gdV, const float* L,
                         const float* D, const float* alpha, const float* E, void* Kt, void* Vt, void* ws,
                         int64_t ws_bytes, void* stream) {
  bool empty;
  int32_t rc = check_problem(p, &empty);
  if (rc != BOB_OK) return rc;
  ColumnPlan c;
  if ((rc = column_plan(p, true, o, &c)) != BOB_OK || empty) return rc;
  if ((rc = check_ptrs({Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, Kt, Vt})) != BOB_OK) return rc;
  if ((rc = check_workspace(p, c, ws, ws_bytes)) != BOB_OK) return rc;
  FB_DISPATCH(p, launch_pass2, p, Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, Kt, Vt, (hipStream_t)stream, c,
              (float*)ws);
}

// Scratch of attn_bob_pass2_cols_gqa_noalloc, for callers that cannot
// allocate: the fp32 partial sums of a split Pass 2 (the *_ws workspace).
// Each device the library runs on holds its own copy until the process
// ends.  In host code `scratch` names a host-side stand-in, not device
// memory: kernels get the address hipGetSymbolAddress returns for the
// current device, read once per device and kept in scratch_dev.
constexpr int64_t kScratchBytes = int64_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
static std::atomic<void*> scratch_dev[kMaxDevices];

// Device address of `scratch` on the current device, or nullptr if it
// cannot be read.
static void* scratch_ptr() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void* ptr = scratch_dev[dev].load(std::memory_order_acquire);
  if (ptr == nullptr) {
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return nullptr;
    scratch_dev[dev].store(ptr, std::memory_order_release);   // the same address on every call
  }
  return ptr;
}

// The layout of Pass 2 with its workspace in `scratch`: as requested; when
// the part count is automatic and its workspace would not fit, the largest
// part count that fits (or none).  A forced part count that does not fit
// gives BOB_ESCRATCH.
static int32_t noalloc_plan(const Problem& p, const ColumnOpts& o, ColumnPlan* c) {
  int32_t rc = column_plan(p, true, o, c);
  if (rc != BOB_OK || column_workspace_bytes(p, c->parts) <= kScratchBytes) return rc;
  if (o.parts != 0) return BOB_ESCRATCH;
  const int64_t per_part = column_workspace_bytes(p, 2) / 2;
  const int fit = (int)std::min<int64_t>(kScratchBytes / per_part, kMaxParts);
  ColumnOpts capped = o;
  capped.parts = fit >= 2 ? std::min(fit, c->parts) : 1;
  return column_plan(p, true, capped, c);
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
  return fb::run_bwd(Problem{dtype, B, H, N, d, scale, causal, H}, fb::kUnsplit, Q, K, V, O, dO, L, dQ, dK, dV, D,
                     nullptr, 0, stream);
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
  return fb::run_pass2(Problem{dtype, B, H, N, d, scale, causal, H}, fb::kUnsplit, Q, K, V, dO, gdQ, gdK, gdV, L,
                       D, alpha, E, Kt, Vt, nullptr, 0, stream);
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
  return fb::run_bwd(Problem{dtype, B, H, N, d, scale, causal, Hkv}, fb::kUnsplit, Q, K, V, O, dO, L, dQ, dK, dV,
                     D, nullptr, 0, stream);
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
  return fb::run_pass2(Problem{dtype, B, H, N, d, scale, causal, Hkv}, fb::kUnsplit, Q, K, V, dO, gdQ, gdK, gdV,
                       L, D, alpha, E, Kt, Vt, nullptr, 0, stream);
}

int64_t bob_pass2_workspace_bytes(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                  int32_t causal, const bob_column_opts* opts) {
  const Problem p{dtype, B, H, N, d, 1.0f, causal, Hkv};
  fb::ColumnPlan c;
  return fb::column_plan(p, true, fb::opts_of(opts), &c) == BOB_OK ? fb::column_workspace_bytes(p, c.parts) : 0;
}

int64_t bob_bwd_workspace_bytes(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                int32_t causal, const bob_column_opts* opts) {
  const Problem p{dtype, B, H, N, d, 1.0f, causal, Hkv};
  fb::ColumnPlan c;
  return fb::column_plan(p, false, fb::opts_of(opts), &c) == BOB_OK ? fb::column_workspace_bytes(p, c.parts) : 0;
}

int32_t bob_column_layout(int32_t kernel, int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                          int32_t causal, const bob_column_opts* opts, bob_column_opts* resolved,
                          int64_t* workspace_bytes) {
  if (kernel != BOB_COLUMNS_BWD && kernel != BOB_COLUMNS_PASS2) return BOB_EINVAL;
  const Problem p{dtype, B, H, N, d, 1.0f, causal, Hkv};
  fb::ColumnPlan c;
  const int32_t rc = fb::column_plan(p, kernel == BOB_COLUMNS_PASS2, fb::opts_of(opts), &c);
  if (rc != BOB_OK) return rc;
  if (resolved != nullptr) {
    resolved->parts = c.parts;
    resolved->wave_sets = c.sets;
    resolved->flush_tiles = c.flush_tiles > 0 ? c.flush_tiles : -1;
  }
  if (workspace_bytes != nullptr) *workspace_bytes = fb::column_workspace_bytes(p, c.parts);
  return BOB_OK;
}

int32_t attn_bwd_gqa_ws(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d, float scale,
                        int32_t causal, const void* Q, const void* K, const void* V, const void* O, const void* dO,
                        const float* L, void* dQ, void* dK, void* dV, float* D, const bob_column_opts* opts,
                        void* workspace, int64_t workspace_bytes, void* stream) {
  return fb::run_bwd(Problem{dtype, B, H, N, d, scale, causal, Hkv}, fb::opts_of(opts), Q, K, V, O, dO, L, dQ, dK,
                     dV, D, workspace, workspace_bytes, stream);
}

int32_t attn_bob_pass2_cols_gqa_ws(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                   float scale, int32_t causal, const void* Q, const void* K, const void* V,
                                   const void* dO, const void* gdQ, const void* gdK, const void* gdV,
                                   const float* L, const float* D, const float* alpha, const float* E, void* Kt,
                                   void* Vt, const bob_column_opts* opts, void* workspace, int64_t workspace_bytes,
                                   void* stream) {
  return fb::run_pass2(Problem{dtype, B, H, N, d, scale, causal, Hkv}, fb::opts_of(opts), Q, K, V, dO, gdQ, gdK,
                       gdV, L, D, alpha, E, Kt, Vt, workspace, workspace_bytes, stream);
}

int32_t attn_bob_pass2_cols_gqa_noalloc(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                        float scale, int32_t causal, const void* Q, const void* K, const void* V,
                                        const void* dO, const void* gdQ, const void* gdK, const void* gdV,
                                        const float* L, const float* D, const float* alpha, const float* E,
                                        void* Kt, void* Vt, const bob_column_opts* opts, void* stream) {
  const Problem p{dtype, B, H, N, d, scale, causal, Hkv};
  bool empty;
  int32_t rc = fb::check_problem(p, &empty);
  if (rc != BOB_OK) return rc;
  fb::ColumnPlan c;
  if ((rc = fb::noalloc_plan(p, fb::opts_of(opts), &c)) != BOB_OK || empty) return rc;
  if ((rc = fb::check_ptrs({Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, Kt, Vt})) != BOB_OK) return rc;
  float* ws = nullptr;
  if (c.parts > 1 && (ws = (float*)fb::scratch_ptr()) == nullptr) return BOB_ELAUNCH;
  FB_DISPATCH(p, fb::launch_pass2, p, Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, Kt, Vt, (hipStream_t)stream, c,
              ws);
}

int64_t bob_scratch_bytes(void) { return fb::kScratchBytes; }

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
    case BOB_ESCRATCH:
      return "BOB_ESCRATCH: the requested layout needs more scratch than the library's static buffer "
             "(bob_scratch_bytes())";
    default: return "unknown bob_status";
  }
}

const char* bob_version(void) { return "flashbob-gfx950 0.2"; }


}  // extern "C"
