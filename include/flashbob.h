/*
 * flashbob.h -- C ABI of libflashbob.so: exact backward-over-backward (BoB)
 * for softmax attention on AMD Instinct MI355X (gfx950).
 *
 * The method is FlashBoB (arXiv 2609.24089).  Given Q, K, V, dO and
 * cotangents U_Q, U_K, U_V on the first-backward outputs (dQ, dK, dV), BoB
 * returns the gradients of Phi = <dQ,U_Q> + <dK,U_K> + <dV,U_V> with respect
 * to Q, K, V and dO (Sec. 3.1, eqs. 4-5).  The library computes them with
 * the two-pass schedule of Alg. 1: Pass 1 holds a block of query rows and
 * streams key blocks, finishing alpha, E, Qt and dOt through the affine
 * fusion of Prop. 3.1 (eq. 8); Pass 2 holds a block of key rows and streams
 * query blocks, finishing Kt and Vt.  The forward (eq. 1) and first backward
 * (eqs. 2-3) that produce the row state (O, L, D) are provided as well.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  dtype   BOB_F32 (fp32 tensors, fp32 arithmetic throughout) or BOB_BF16
 *          (bf16 tensors; bf16 MFMA operands with fp32 accumulation; fp32
 *          row scalars and elementwise math; outputs rounded to nearest even).
 *  B, H, N, d  batch, heads, sequence length and head dimension.  Matrices
 *          are contiguous row-major [B, H, N, d] in the tensor dtype; row
 *          vectors (L, D, alpha, E) are contiguous fp32 [B, H, N].
 *          Supported head dimensions: d = 32, 64, 128, 256 for bf16 and
 *          d = 32, 64, 128 for fp32 (bob_supported() reports the set).
 *  scale   the softmax scale tau of eq. 1 (the paper uses 1/sqrt(d)); any
 *          finite value is accepted.  L is the natural-log normalizer
 *          L_i = log sum_{j valid} exp(S_ij) with S = tau Q K^T.
 *  causal  0: no mask, every key is visible to every query (dense
 *          attention).  1: the causal mask of eq. 1 (M_ij = -inf for j > i),
 *          so every row sum runs over keys j <= i; the kernels skip tiles
 *          above the diagonal.  All four calls of one problem must use the
 *          same value.
 *  pointers  device pointers owned by the caller, 16-byte aligned, on the
 *          current HIP device (the kernels run there).  The library
 *          allocates no memory (the *_ws calls take their workspace from
 *          the caller); its only state is the modes set by
 *          bob_set_column_wave_sets and bob_set_column_split and a
 *          per-device count of compute units.
 *          Outputs must not alias inputs.
 *  stream  a hipStream_t of the current device passed as void* (NULL = the
 *          default stream).  Work
 *          is enqueued asynchronously; the call returns before it finishes.
 *          Calls that consume another call's outputs (attn_bwd after
 *          attn_fwd_lse, pass 2 after pass 1) must be ordered on one stream
 *          or with events by the caller.
 *
 * Errors: every argument check happens before any HIP call, so a rejected
 * call has no effect.  BOB_EINVAL: negative B/H/N, non-finite scale, causal
 * not 0/1, a NULL
 * or misaligned pointer for a non-empty problem, or a problem too large for
 * the launch grid.  BOB_EUNSUPPORTED: a (dtype, d) pair that is not built.
 * BOB_ELAUNCH: the HIP launch itself reported an error.  B*H*N == 0 is a
 * valid empty problem and returns BOB_OK without touching memory.  No
 * exception crosses the ABI and the library never aborts.
 */
#ifndef FLASHBOB_H
#define FLASHBOB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { BOB_F32 = 0, BOB_BF16 = 1 } bob_dtype;

typedef enum {
  BOB_OK = 0,
  BOB_EINVAL = 1,
  BOB_EUNSUPPORTED = 2,
  BOB_ELAUNCH = 3
} bob_status;

/* Forward attention (eq. 1) with its log-normalizer (Sec. 2).
 * In:  Q, K, V  [B,H,N,d].
 * Out: O = softmax(scale Q K^T) V  [B,H,N,d];  L (fp32 [B,H,N]). */
int32_t attn_fwd_lse(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale, int32_t causal,
                     const void* Q, const void* K, const void* V,
                     void* O, float* L, void* stream);

/* First backward (eqs. 2-3) from the saved forward state.
 * In:  Q, K, V, O, dO [B,H,N,d];  L fp32 [B,H,N] from attn_fwd_lse.
 * Out: dQ, dK, dV [B,H,N,d];  D fp32 [B,H,N], D_i = do_i . o_i.
 * D is written by the row kernel before the column kernel reads it (both
 * are enqueued on `stream` by this call). */
int32_t attn_bwd(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale, int32_t causal,
                 const void* Q, const void* K, const void* V, const void* O, const void* dO,
                 const float* L, void* dQ, void* dK, void* dV, float* D, void* stream);

/* BoB Pass 1, row-major (Alg. 1 Pass 1; Prop. 3.1 and eq. 8).
 * In:  Q, K, V, O, dO, gdQ (= U_Q), gdK (= U_K), gdV (= U_V) [B,H,N,d];
 *      L, D fp32 [B,H,N] from attn_fwd_lse / attn_bwd;
 *      dQ [B,H,N,d] from attn_bwd, OPTIONAL (may be NULL).
 * Out: Qt, dOt [B,H,N,d];  alpha, E fp32 [B,H,N] -- the two row scalars
 *      alpha_i = sum_j P_ij F_ij and E_i = sum_j P_ij Pt_ij that Pass 2 reads.
 * With dQ == NULL the kernel keeps the six row accumulators of Prop. 3.1.
 * With dQ given it drops R = sum_j P_ij dP_ij k_j, using R = dQ/scale + D B
 * (so Qt = scale (Omega - E0 B) - alpha dQ, E0 = E + alpha D); the result is
 * the same up to rounding and the d = 128 kernel fits two waves per SIMD. */
int32_t attn_bob_pass1_rows(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale, int32_t causal,
                            const void* Q, const void* K, const void* V, const void* O,
                            const void* dO, const void* gdQ, const void* gdK, const void* gdV,
                            const float* L, const float* D, const void* dQ,
                            void* Qt, void* dOt, float* alpha, float* E, void* stream);

/* BoB Pass 2, column-major (Alg. 1 Pass 2).
 * In:  Q, K, V, dO, gdQ, gdK, gdV [B,H,N,d];  L, D, alpha, E fp32 [B,H,N].
 * Out: Kt, Vt [B,H,N,d].  Must run after Pass 1 has written alpha and E. */
int32_t attn_bob_pass2_cols(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale, int32_t causal,
                            const void* Q, const void* K, const void* V, const void* dO,
                            const void* gdQ, const void* gdK, const void* gdV,
                            const float* L, const float* D, const float* alpha, const float* E,
                            void* Kt, void* Vt, void* stream);

/* Grouped key/value heads (GQA; MQA when Hkv = 1), the extension the
 * paper's limitations paragraph names and says the affine-fusion structure
 * does not obstruct.  Hkv key/value heads are shared by the H query heads,
 * H a multiple of Hkv: query head h of a batch entry uses key/value head
 * h / (H / Hkv).  Query-side tensors (Q, dO, gdQ, O, dQ, Qt, dOt; L, D,
 * alpha, E) are [B,H,N,d] or [B,H,N]; key-side tensors (K, V, gdK, gdV, dK,
 * dV, Kt, Vt) are [B,Hkv,N,d].  The first-backward dK, dV of a key/value
 * head sum its H / Hkv query heads' contributions, so Phi is the multi-head
 * Phi with K, V, gdK, gdV repeated per query head: Qt, dOt, alpha, E are
 * per query head and Kt, Vt sum over each group (written once, no atomics).
 * Arguments and errors are those of the calls above, plus BOB_EINVAL when
 * Hkv < 1 or H is not a multiple of Hkv for a non-empty problem.  With
 * Hkv = H each call equals its multi-head counterpart. */
int32_t attn_fwd_lse_gqa(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d, float scale,
                         int32_t causal, const void* Q, const void* K, const void* V, void* O, float* L,
                         void* stream);
int32_t attn_bwd_gqa(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d, float scale,
                     int32_t causal, const void* Q, const void* K, const void* V, const void* O, const void* dO,
                     const float* L, void* dQ, void* dK, void* dV, float* D, void* stream);
int32_t attn_bob_pass1_rows_gqa(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                float scale, int32_t causal, const void* Q, const void* K, const void* V,
                                const void* O, const void* dO, const void* gdQ, const void* gdK,
                                const void* gdV, const float* L, const float* D, const void* dQ, void* Qt,
                                void* dOt, float* alpha, float* E, void* stream);
int32_t attn_bob_pass2_cols_gqa(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                float scale, int32_t causal, const void* Q, const void* K, const void* V,
                                const void* dO, const void* gdQ, const void* gdK, const void* gdV,
                                const float* L, const float* D, const float* alpha, const float* E, void* Kt,
                                void* Vt, void* stream);

/* Pass 2 with each key/value column block split over several workgroups,
 * for grids too small to fill the device.  Under the causal mask a column
 * block's work is proportional to the query tiles at or below its diagonal,
 * so with few key/value heads (e.g. multi-query attention) the first blocks
 * would set the time; split, every part takes an equal share of its block's
 * (query head, query tile) iterations and stores fp32 partial Kt and Vt to
 * `workspace`, and a second kernel on the same stream adds the parts in
 * part order and writes Kt, Vt.
 * Arguments as attn_bob_pass2_cols_gqa, plus:
 *  workspace, workspace_bytes  device memory owned by the caller, 16-byte
 *          aligned, of at least bob_pass2_workspace_bytes() bytes for this
 *          problem; it needs no initial contents and holds nothing useful
 *          afterwards.  It must not be reused before the call's kernels have
 *          finished on `stream`.
 * When bob_pass2_workspace_bytes() is 0 the call runs the unsplit kernels
 * and ignores workspace (it may be NULL).  Otherwise a NULL, misaligned or
 * too small workspace gives BOB_EINVAL.  Split and unsplit results differ by
 * the order of the fp32 sums; each is deterministic. */
int32_t attn_bob_pass2_cols_gqa_ws(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                   float scale, int32_t causal, const void* Q, const void* K, const void* V,
                                   const void* dO, const void* gdQ, const void* gdK, const void* gdV,
                                   const float* L, const float* D, const float* alpha, const float* E, void* Kt,
                                   void* Vt, void* workspace, int64_t workspace_bytes, void* stream);

/* The first backward with its column kernel (dK, dV) split the same way:
 * arguments as attn_bwd_gqa plus workspace and workspace_bytes, with the
 * rules of attn_bob_pass2_cols_gqa_ws (its size from
 * bob_bwd_workspace_bytes).  dQ and D do not depend on the split. */
int32_t attn_bwd_gqa_ws(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d, float scale,
                        int32_t causal, const void* Q, const void* K, const void* V, const void* O, const void* dO,
                        const float* L, void* dQ, void* dK, void* dV, float* D, void* workspace,
                        int64_t workspace_bytes, void* stream);

/* Workspace bytes attn_bwd_gqa_ws needs, as bob_pass2_workspace_bytes (the
 * first backward's column workgroups own their own number of key rows, so
 * the part count can differ from Pass 2's). */
int64_t bob_bwd_workspace_bytes(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                int32_t causal);

/* Workspace bytes attn_bob_pass2_cols_gqa_ws needs for this problem on the
 * current device under the current bob_set_column_split mode: 0 when it
 * would not split (and for an empty or invalid problem, which that call
 * reports), else parts x 2 x B x Hkv x N x d x 4. */
int64_t bob_pass2_workspace_bytes(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                  int32_t causal);

/* Three-pass control schedule (App. "Three-pass versus two-pass" and the
 * three-pass overlay of App. "Dependency graphs"): the schedule that the
 * affine fusion of Prop. 3.1 improves on, kept for the 2- vs 3-pass ablation
 * (Table 7).  Sweep 1 is attn_bob3_alpha_rows, sweep 2 attn_bob3_rows, sweep 3
 * the shared column pass attn_bob_pass2_cols.  The results equal those of
 * attn_bob_pass1_rows up to rounding.
 *
 * Sweep 1, row-major: alpha_i = sum_j P_ij F_ij alone (F = scale (U_Q K^T +
 * Q U_K^T)), streaming only K and U_K.
 * In:  Q, K, gdQ (= U_Q), gdK (= U_K) [B,H,N,d];  L fp32 [B,H,N].
 * Out: alpha fp32 [B,H,N]. */
int32_t attn_bob3_alpha_rows(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale,
                             int32_t causal, const void* Q, const void* K, const void* gdQ, const void* gdK,
                             const float* L, float* alpha, void* stream);

/* Sweep 2, row-major, with alpha from sweep 1: forms Pt = C + F (dP - D) -
 * alpha dP and h = F - alpha directly and applies one delayed correction,
 * Qt = scale (sum_j P Pt k_j + dS U_K - E sum_j P k_j), dOt = P U_V + (P h) V.
 * In:  Q, K, V, dO, gdQ, gdK, gdV [B,H,N,d];  L, D, alpha fp32 [B,H,N].
 * Out: Qt, dOt [B,H,N,d];  E fp32 [B,H,N]. */
int32_t attn_bob3_rows(int32_t dtype, int64_t B, int64_t H, int64_t N, int64_t d, float scale, int32_t causal,
                       const void* Q, const void* K, const void* V, const void* dO, const void* gdQ,
                       const void* gdK, const void* gdV, const float* L, const float* D, const float* alpha,
                       void* Qt, void* dOt, float* E, void* stream);

/* 1 if (dtype, d) is built into this library, else 0. */
int32_t bob_supported(int32_t dtype, int64_t d);

/* Static, NUL-terminated description of a status code (never NULL). */
const char* bob_status_string(int32_t status);

/* Static version string of the library. */
const char* bob_version(void);

/* How the column-owned kernels (the dK, dV half of attn_bwd, and Pass 2)
 * spread a key/value column block over a CU.  By default (mode 0) a column
 * block whose grid has no more workgroups than the device has compute units
 * (few key/value heads and short sequences, e.g. multi-query attention) is
 * given two wave sets in one workgroup, which take alternate streamed tiles
 * and add their fp32 partial sums in a fixed order at the end; larger grids
 * use one set.  Mode 1 always uses one set, mode 2 uses two wherever the
 * launch shape has room (bf16 d <= 128, fp32 Pass 2 with d <= 64).  The two
 * forms sum in different orders, so their results differ by rounding; for a
 * given mode, device and problem the result is deterministic.  Process-wide
 * (all devices); not ordered against launches in flight.  Returns BOB_OK, or
 * BOB_EINVAL for a mode outside 0..2. */
int32_t bob_set_column_wave_sets(int32_t mode);

/* How many workgroups attn_bwd_gqa_ws and attn_bob_pass2_cols_gqa_ws give
 * each column block.  0 (default): automatic, from the column grid, the
 * device's compute units and the mask; 1: never split; 2..8: always that
 * many parts.  Process-wide (all devices); read by the *_workspace_bytes
 * queries and by the calls themselves, which must see the same mode.  Returns BOB_OK, or BOB_EINVAL for a value
 * outside 0..8. */
int32_t bob_set_column_split(int32_t parts);

#ifdef __cplusplus
}
#endif

#endif /* FLASHBOB_H */
