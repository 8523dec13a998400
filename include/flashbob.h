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
 *          the caller) and keeps no state apart from the device address of
 *          the static scratch buffer of attn_bob_pass2_cols_gqa_noalloc:
 *          every choice it makes depends only on the arguments and on the
 *          current device's compute-unit count, so the entry points are
 *          thread-safe (two _noalloc calls that overlap on one device race
 *          on its scratch, see there).
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
  BOB_ELAUNCH = 3,
  BOB_ESCRATCH = 4
} bob_status;

/* Layout of a column-owned kernel: the first backward's dK, dV kernel or
 * Pass 2's Kt, Vt kernel (bob_column_layout: BOB_COLUMNS_BWD,
 * BOB_COLUMNS_PASS2).  Each such kernel owns one block of key rows per
 * workgroup and streams every query tile of the block's query heads past it
 * (Alg. 1 Pass 2), so each output element is one long fp32 sum.  Requests
 * (0 = automatic in every field):
 *  parts        workgroups that share one column block, 1..8.  With more than
 *               one, each part sums an equal share of the block's streamed
 *               tiles and stores fp32 partial sums to the caller's workspace,
 *               and a second kernel adds them in part order (for grids too
 *               small, or too uneven under the causal mask, to fill the
 *               device).  Automatic: causal grids to about 8 workgroups per
 *               compute unit, dense Pass 2 grids smaller than the compute-unit
 *               count to 2 per unit, the dense first backward to 8 per unit;
 *               never for blocks of fewer than 1024 streamed tiles.
 *  wave_sets    1 or 2 wave sets per workgroup; two take alternate streamed
 *               tiles and add their fp32 sums through LDS at the end.
 *               Automatic: two when the grid has no more workgroups than the
 *               device has compute units (and the shape has room: bf16
 *               d <= 128, fp32 Pass 2 with d <= 64); a split block uses one.
 *               On a dense unsplit grid that fills the device, the
 *               automatic bf16 d = 128 Pass 2 runs one set in workgroups of
 *               twice the waves (one copy of each streamed tile serves
 *               more key rows), with results equal bit for bit to those of
 *               a forced wave_sets = 1.  The automatic bf16 d = 256 Pass 2
 *               on an unsplit block runs in wave pairs that split the head
 *               dims and exchange partial score tiles through LDS; its
 *               results differ from a forced wave_sets = 1 in the order of
 *               fp32 sums inside the score tiles.
 *  flush_tiles  streamed tiles per accumulation section, >= 1, or -1 for one
 *               section.  The MFMA's fp32 accumulation drops the low bits of
 *               small addends toward one side, so a chain of tens of
 *               thousands of tiles into one accumulator drifts (the zero
 *               column sums of Kt, Vt, dK grow with N); in sections, each
 *               chain restarts from zero and is added into fp32 sums with
 *               round-to-nearest adds.  Automatic: sections of 1024 tiles
 *               when a chain would exceed 16384 tiles (bf16 d <= 128; other
 *               (dtype, d) run one section, and asking for sections there
 *               gives BOB_EUNSUPPORTED).
 * Different layouts sum in different orders, so results differ in the last
 * bits; each layout is deterministic. */
typedef struct {
  int32_t parts;
  int32_t wave_sets;
  int32_t flush_tiles;
} bob_column_opts;

enum { BOB_COLUMNS_BWD = 0, BOB_COLUMNS_PASS2 = 1 };

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
 * are enqueued on `stream` by this call).  The column kernel runs unsplit
 * with automatic wave sets and sections (bob_column_opts {1, 0, 0}). */
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
 * Out: Kt, Vt [B,H,N,d].  Must run after Pass 1 has written alpha and E.
 * Runs unsplit with automatic wave sets and sections (bob_column_opts
 * {1, 0, 0}). */
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

/* Pass 2 and the first backward with their column kernels laid out by
 * `opts` (bob_column_opts; NULL = all automatic), which may split a column
 * block over workgroups and then needs a workspace.
 * Arguments as attn_bob_pass2_cols_gqa / attn_bwd_gqa, plus:
 *  opts    the caller's layout requests (read during the call only).
 *  workspace, workspace_bytes  device memory owned by the caller, 16-byte
 *          aligned, of at least bob_pass2_workspace_bytes() /
 *          bob_bwd_workspace_bytes() for the same problem and opts; it needs
 *          no initial contents and holds nothing useful afterwards.  It
 *          must not be reused before the call's kernels have finished on
 *          `stream`.  When that size is 0 (the layout does not split) the
 *          workspace is ignored and may be NULL; otherwise a NULL,
 *          misaligned or too small workspace gives BOB_EINVAL.
 * A request out of range (parts outside 0..8, wave_sets outside 0..2,
 * flush_tiles below -1) gives BOB_EINVAL.  dQ and D of the first backward do
 * not depend on the layout. */
int32_t attn_bob_pass2_cols_gqa_ws(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                   float scale, int32_t causal, const void* Q, const void* K, const void* V,
                                   const void* dO, const void* gdQ, const void* gdK, const void* gdV,
                                   const float* L, const float* D, const float* alpha, const float* E, void* Kt,
                                   void* Vt, const bob_column_opts* opts, void* workspace, int64_t workspace_bytes,
                                   void* stream);
int32_t attn_bwd_gqa_ws(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d, float scale,
                        int32_t causal, const void* Q, const void* K, const void* V, const void* O, const void* dO,
                        const float* L, void* dQ, void* dK, void* dV, float* D, const bob_column_opts* opts,
                        void* workspace, int64_t workspace_bytes, void* stream);

/* Workspace bytes attn_bob_pass2_cols_gqa_ws / attn_bwd_gqa_ws need for this
 * problem and opts on the current device: 0 when the layout does not split
 * (and for an empty or invalid problem or request, which the calls report),
 * else parts x 2 x B x Hkv x N x d x 4. */
int64_t bob_pass2_workspace_bytes(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                  int32_t causal, const bob_column_opts* opts);
int64_t bob_bwd_workspace_bytes(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                int32_t causal, const bob_column_opts* opts);

/* The layout a column kernel (kernel: BOB_COLUMNS_BWD or BOB_COLUMNS_PASS2)
 * would run for this problem and opts on the current device: `resolved`
 * (may be NULL) receives parts >= 1, wave_sets (1 or 2) and flush_tiles
 * (-1 for one section), `workspace_bytes` (may be NULL) the workspace the
 * *_ws call needs.  Returns BOB_OK, or the status the call would return
 * for the problem and opts (pointers aside). */
int32_t bob_column_layout(int32_t kernel, int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                          int32_t causal, const bob_column_opts* opts, bob_column_opts* resolved,
                          int64_t* workspace_bytes);

/* Pass 2 for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): as
 * attn_bob_pass2_cols_gqa_ws, but a split layout keeps its fp32 partial sums
 * in a scratch buffer the library holds in static device memory instead of
 * a caller's workspace.  The call itself allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); the caller passes inputs and
 * outputs as usual.
 *  scratch  bob_scratch_bytes() (64 MiB) per device, part of the library's
 *          code object, held by every device the library runs on until the
 *          process ends.  A split needs parts x 2 x B x Hkv x N x d x 4 bytes
 *          of it.  With parts automatic (opts NULL or opts->parts == 0) the
 *          call uses the largest automatic part count that fits, or runs
 *          unsplit; a forced opts->parts whose split does not fit gives
 *          BOB_ESCRATCH before any launch.
 *  races   every call on one device shares that device's scratch, which
 *          keeps the last call's contents (a split writes every element it
 *          later reads, so nothing needs clearing).  Two calls that overlap
 *          on one device (different streams, or different host threads)
 *          race on it and give wrong results: order them on one stream or
 *          with events.  Calls that do not split do not touch it.
 * Results equal those of attn_bob_pass2_cols_gqa_ws with the same resolved
 * layout (bob_column_layout with the same part count), bit for bit.
 * Errors as attn_bob_pass2_cols_gqa_ws, plus BOB_ESCRATCH, and BOB_ELAUNCH
 * if the scratch buffer's device address cannot be read. */
int32_t attn_bob_pass2_cols_gqa_noalloc(int32_t dtype, int64_t B, int64_t H, int64_t Hkv, int64_t N, int64_t d,
                                        float scale, int32_t causal, const void* Q, const void* K, const void* V,
                                        const void* dO, const void* gdQ, const void* gdK, const void* gdV,
                                        const float* L, const float* D, const float* alpha, const float* E,
                                        void* Kt, void* Vt, const bob_column_opts* opts, void* stream);

/* Bytes of the static scratch buffer attn_bob_pass2_cols_gqa_noalloc uses. */
int64_t bob_scratch_bytes(void);

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

#ifdef __cplusplus
}
#endif

#endif /* FLASHBOB_H */
