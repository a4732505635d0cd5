/*
 * ozaki2.h -- FP64 matrix multiply emulated on CDNA4 (gfx950) FP8 matrix
 * cores through the CRT-based Ozaki Scheme II.
 *
 * Method: Matsuoka, "FP8 is All You Need (Part 1)", arXiv 2606.06510,
 * Algorithm 1 (Ozaki II dense GEMM at phase level):
 *   Phase 1  power-of-two row/column scaling to integers, Eq. (scale), with the
 *            max-magnitude estimation pass (the "+1" of alpha = 3r+1);
 *   Phase 2  r modular GEMMs, Eq. (modgemm), each as three FP8 plane products
 *            (Eq. (sq-shortcut) for square moduli, Eq. (kar) for nonsquare
 *            ones) accumulated exactly in FP32, Eq. (accum-exact);
 *   Phase 3  CRT reconstruction of the exact integer, Eq. (garner) / (M-bound),
 *            one rounded conversion back to FP64, and the native-FP64
 *            fallback for rows the scaling cannot certify.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Layout: column-major (BLAS), no transposes: C (m x n) = A (m x k) * B (k x n).
 * A, B, C and the workspace are DEVICE pointers owned by the caller; the
 * library keeps no reference to them after a call returns, except that a plan
 * borrows A and B from ozaki2_deconstruct until its ozaki2_reconstruct (the
 * fallback recomputes flagged rows from them).
 * `stream` is a hipStream_t passed as void* (NULL = the default stream).  Work
 * is enqueued asynchronously; nothing synchronises except ozaki2_plan_query
 * and ozaki2_finalize.
 * Validation happens before any launch: on an error nothing is written.
 * Asynchronous device faults surface at the caller's next synchronisation.
 * num_moduli (r) must be in [8, 16]: the paper works with 8-12 moduli and up
 * to a conservative 15; with fewer the modulus product leaves too few bits for
 * anything near FP64 accuracy (r = 8 already stops near 1e-11 on the
 * lognormal workload), so r < 8 returns OZ2_E_INVALID.  The moduli are the paper's r = 12 set
 * (1089, 1024, 961, 841, 625, 529, 511, 509, 503, 499, 491, 487) extended by
 * the nonsquare 481, 479, 467, 463 and truncated to the r largest.
 * Limits: m, n, k >= 0 and m*k, k*n, m*n each below 2^40.
 * Accuracy contract: entries of rows/columns that are not flagged are the
 * IEEE round-to-nearest-even value of the exact rational D^-1 (A~ B~) E^-1,
 * where A~ = RN(D A), B~ = RN(B E) are the quantised integer matrices; an
 * exactly zero result is +0.0.  Flagged rows of A (columns of B) -- any
 * NaN/Inf (T1), or a nonzero entry that quantises to zero (T2) -- are
 * recomputed in native FP64 (products and sums in a fixed order; within the
 * FP64 dot-product error bound).
 */
#ifndef OZAKI2_H
#define OZAKI2_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
enum {
  OZ2_OK = 0,
  OZ2_E_INVALID = -1,      /* bad size, leading dimension, pointer, r or flags */
  OZ2_E_NOMEM = -2,        /* internal workspace allocation failed */
  OZ2_E_DEVICE = -3,       /* a HIP runtime call or a kernel launch failed */
  OZ2_E_UNSUPPORTED = -4,  /* not a gfx950 device */
  OZ2_E_WORKSPACE = -5     /* caller workspace NULL or smaller than required */
};

/* flags (bitwise or) */
enum {
  OZ2_ACCUMULATE = 1u,     /* C <- C + A*B: one extra IEEE RN addition per entry */
  OZ2_SCALE_FIXED = 2u,    /* no max-magnitude pass: mu = k max|A~| max|B~| (alpha = 3r) */
  OZ2_QUANT_TZ = 4u,       /* quantise by truncation toward zero instead of RN-even */
  OZ2_NO_FALLBACK = 8u,    /* never recompute flagged rows natively */
  OZ2_FORCE_FALLBACK = 16u,/* recompute every row natively (testing aid) */
  OZ2_KEEP_RESIDUES = 32u, /* materialise the r residues of every output in the workspace
                              (the staged route, which every call takes unless OZ2_FUSED is
                              given or ozaki2_dgemm_ex takes its tall-skinny route: the flag
                              forbids OZ2_FUSED alongside it and keeps that route off) */
  OZ2_TIME_STAGES = 64u,   /* plans only: record HIP events between the stages on the
                              stream of each call (OZ2_Q_STAGE_TIMES) */
  OZ2_FUSED = 128u         /* the residue GEMMs and the reconstruction as one kernel that
                              keeps every output's residues on chip (r <= 12 and k <= 32768;
                              OZ2_E_UNSUPPORTED otherwise): nothing of them is written to the
                              workspace, so ozaki2_workspace_bytes is smaller.  In a plan,
                              ozaki2_residue_gemm then only marks its stage and
                              ozaki2_reconstruct runs the fused kernel; OZ2_Q_RESIDUES and
                              OZ2_Q_INTEGERS are not available.  Results are those of the
                              staged route bit for bit; on MI355X it is the slower route (see
                              ozaki2_dgemm_ex), so it is taken only when asked for */,
  OZ2_REUSE_A_SCALES = 256u /* ozaki2_gemv_batched only: the workspace still holds A's row
                              scales, flags and fallback list from the previous call on it,
                              made with the same A (contents), lda, m, k, num_moduli and
                              other flags (the caller's promise: nothing checks it); the
                              scan of A is skipped, as an operand-stationary A in an
                              iterative method allows.  Results are those of a full call */
};

/* C = A*B with the default flags (accumulation: ozaki2_dgemm_ex).
 * Uses a library-internal, grow-only workspace per device (hipMalloc'd on
 * first use and when a call needs more; released by ozaki2_finalize).  Calls
 * on one device share it, so concurrent calls on different streams must use
 * ozaki2_dgemm_ex with workspaces of their own.
 * Returns OZ2_OK or an error code; on error nothing is enqueued. */
int ozaki2_dgemm(int m, int n, int k, const double* A, int lda, const double* B,
                 int ldb, double* C, int ldc, int num_moduli, void* stream);

/* C = A*B, or C = C + A*B with OZ2_ACCUMULATE, using the caller's workspace
 * (device memory of at least ozaki2_workspace_bytes(m, n, k, r, flags) bytes,
 * 256-byte aligned; contents on entry are ignored and on exit undefined).
 * With OZ2_SCALE_FIXED, n <= 16 and none of OZ2_ACCUMULATE, OZ2_FUSED,
 * OZ2_KEEP_RESIDUES, the product runs as the fused GEMV of ozaki2_gemv_batched
 * (A deconstructed on the fly, the fused mode for tall-skinny products of
 * Section "On-Chip Tile Fusion"): the same results as the staged path, bit for
 * bit, without A's digit planes. */
int ozaki2_dgemm_ex(int m, int n, int k, const double* A, int lda,
                    const double* B, int ldb, double* C, int ldc,
                    int num_moduli, unsigned flags, void* workspace,
                    size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): C = A*B as
 * ozaki2_dgemm, with the workspace taken from a device array of
 * OZ2_STATIC_SCRATCH_BYTES (64 MiB) that the library holds on every GPU it
 * runs on until the process ends.  No hipMalloc, hipFree or other allocating
 * call is made (the first call on a device looks the array's address up once).
 * Products whose workspace (ozaki2_workspace_bytes(m, n, k, r, 0)) exceeds
 * the array -- e.g. beyond about 768^3 at r = 12 or 704^3 at r = 16 -- return
 * OZ2_E_WORKSPACE before any launch.  Every call on a GPU uses that GPU's one
 * array: calls that overlap in time on one GPU (different streams or host
 * threads without ordering) race and give undefined results; calls ordered on
 * one stream are safe.  Same results as ozaki2_dgemm. */
#define OZ2_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
int ozaki2_dgemm_static(int m, int n, int k, const double* A, int lda, const double* B,
                        int ldb, double* C, int ldc, int num_moduli, void* stream);

/* batch independent products C_b = A_b * B_b, A_b = A + b*strideA (elements),
 * likewise B_b, C_b; each with the layout rules above.  Strides must keep the
 * output matrices disjoint. Internal workspace as for ozaki2_dgemm. */
int ozaki2_dgemm_strided_batched(int m, int n, int k, const double* A, int lda,
                                 long long strideA, const double* B, int ldb,
                                 long long strideB, double* C, int ldc,
                                 long long strideC, int batch, int num_moduli,
                                 void* stream);

/* Batched GEMV, the paper's fused Ozaki-II GEMV (Alg. 2, section "Strategy
 * 1: Batched GEMV"): Y = A X for A (m x k, lda), X (k x nrhs, ldx) with
 * 1 <= nrhs <= 16 right-hand sides, Y (m x nrhs, ldy), all column-major FP64
 * device memory.  A is read twice in FP64 -- once for its row exponents,
 * once by the fused kernel that quantises, reduces and splits it into E4M3
 * digit planes on the fly and multiplies them on FP8 MFMA against X's planes
 * with all r moduli's accumulators in registers -- and never written in any
 * other form.  The scaling is the fixed rule (Alg. 1's mu = k max|A~| max|X~|,
 * as OZ2_SCALE_FIXED): entries of unflagged rows and columns are the IEEE
 * RN-even value of D^-1 (A~ X~) E^-1 exactly as ozaki2_dgemm_ex with
 * OZ2_SCALE_FIXED computes it; flagged rows of A / columns of X (T1, T2) are
 * recomputed natively.  flags: OZ2_QUANT_TZ, OZ2_NO_FALLBACK,
 * OZ2_FORCE_FALLBACK, OZ2_REUSE_A_SCALES (others: OZ2_E_INVALID).  workspace: device memory of
 * ozaki2_gemv_workspace_bytes(m, k, nrhs, r) bytes, 256-byte aligned.  k = 0
 * gives Y = 0; m = 0 or nrhs = 0 is a no-op.  Validation as for
 * ozaki2_dgemm_ex (nrhs > 16: OZ2_E_INVALID). */
int ozaki2_gemv_batched(int m, int k, int nrhs, const double* A, int lda, const double* X,
                        int ldx, double* Y, int ldy, int num_moduli, unsigned flags,
                        void* workspace, size_t ws_bytes, void* stream);

/* Workspace bytes of ozaki2_gemv_batched (0 on invalid arguments). */
size_t ozaki2_gemv_workspace_bytes(int m, int k, int nrhs, int num_moduli);

/* Workspace bytes ozaki2_dgemm_ex / ozaki2_plan_create need (0 on invalid
 * arguments; for the tall-skinny fixed-scale route of ozaki2_dgemm_ex, enough
 * for both it and a plan). */
size_t ozaki2_workspace_bytes(int m, int n, int k, int num_moduli, unsigned flags);

/* The r moduli in ascending (reconstruction) order into host_out[0..r-1]. */
int ozaki2_moduli(int num_moduli, int* host_out);

/* ---------------------------------------------------------------- staged API
 * The three phases of Alg. 1 as separately callable stages over one plan.
 * A plan borrows a caller workspace (ozaki2_workspace_bytes) and is not
 * re-entrant; different plans may run on different streams. */
typedef struct ozaki2_plan_s* ozaki2_plan_t;

int ozaki2_plan_create(ozaki2_plan_t* out, int m, int n, int k, int num_moduli,
                       unsigned flags, void* workspace, size_t ws_bytes);
int ozaki2_plan_destroy(ozaki2_plan_t plan);

/* Phase 1: scan (exponents, T1 flags), max-magnitude pass (codes, the code
 * GEMM on FP8 MFMA, row/column maxima), scales, quantisation, centred
 * residues and their E4M3 digit planes (T2 flags).  Borrows A and B. */
int ozaki2_deconstruct(ozaki2_plan_t plan, const double* A, int lda,
                       const double* B, int ldb, void* stream);

/* Operand-stationary use (the paper's Mode P, deferred deconstruction of a
 * fixed operand, here for a dense one): re-run phase 1 for one operand only
 * and keep the other operand's planes, scales and flags from an earlier
 * ozaki2_deconstruct / ozaki2_deconstruct_a / ozaki2_deconstruct_b of this
 * plan.  Only for plans created with OZ2_SCALE_FIXED, where the scale of a row
 * of A depends on A alone and that of a column of B on B alone (no
 * max-magnitude pass); the results are then those of ozaki2_deconstruct on
 * the same pair.  Returns OZ2_E_INVALID for a plan without OZ2_SCALE_FIXED, a
 * null pointer or lda < max(1, m) / ldb < max(1, k).  ozaki2_residue_gemm
 * needs both operands deconstructed; the kept operand's device memory must
 * stay unchanged while the plan uses it (the native-FP64 fallback of
 * ozaki2_reconstruct reads it). */
int ozaki2_deconstruct_a(ozaki2_plan_t plan, const double* A, int lda, void* stream);
int ozaki2_deconstruct_b(ozaki2_plan_t plan, const double* B, int ldb, void* stream);

/* Phase 2: the 3r FP8 plane products and their exact modular accumulation;
 * writes, per modulus, a representative of every output's residue into the
 * workspace (OZ2_Q_RESIDUES). */
int ozaki2_residue_gemm(ozaki2_plan_t plan, void* stream);

/* Phase 3: CRT reconstruction, inverse scaling with one rounding, then the
 * native-FP64 fallback of flagged rows/columns (reads the A, B given to
 * ozaki2_deconstruct).  With OZ2_ACCUMULATE in the plan's flags, C += .. */
int ozaki2_reconstruct(ozaki2_plan_t plan, double* C, int ldc, void* stream);

/* Diagnostics for tests: synchronises the device, then copies a plan
 * quantity to host memory.  ozaki2_plan_query_bytes gives the size. */
enum {
  OZ2_Q_EXPONENTS = 1,     /* int32 E^A[m] then E^B[n]: frexp exponent of the row/col maximum
                              as the scale kernel computed it (0 for a zero or T1 row) */
  OZ2_Q_MAXIMA = 2,        /* uint64 R[m] then K[n] (code-product row/col maxima) */
  OZ2_Q_SCALES = 3,        /* int32 s[m] then t[n] (power-of-two scales) */
  OZ2_Q_FLAGS = 4,         /* uint32 flagsA[m] then flagsB[n]: bit0 T1, bit1 T2 */
  OZ2_Q_CODES = 5,         /* uint8 codes of A [m][k] then of B [n][k] (E4M3 bytes) */
  OZ2_Q_PLANES = 6,        /* uint8 planes of A [p_store][m][k] then of B [p_store][n][k] */
  OZ2_Q_RESIDUES = 7,      /* int16 [r][n][m]: per modulus the representative of C~ mod m_i the
                              residue GEMMs left for the reconstruction (any value congruent
                              to C~ with magnitude <= m_i/2 + 32; after residue_gemm) */
  OZ2_Q_INTEGERS = 8,      /* uint32 [n][m][5]: exact integer, two's complement, 160 bits LE,
                              formed from those residues by the reconstruction's own routine */
  OZ2_Q_FALLBACK_COUNT = 9,/* int32 [2]: rows of A, columns of B the reconstruction recomputes natively */
  OZ2_Q_STAGE_TIMES = 10   /* float [6], milliseconds, of the last deconstruct / residue_gemm /
                              reconstruct of an OZ2_TIME_STAGES plan: scan + codes (a1, a2),
                              max-magnitude GEMM (a3), scales + split (a4), residue GEMMs
                              (a5), reconstruction (a6), native fallback (a7); OZ2_E_INVALID
                              unless all three stages ran since the last deconstruct */
};
size_t ozaki2_plan_query_bytes(ozaki2_plan_t plan, int what);
int ozaki2_plan_query(ozaki2_plan_t plan, int what, void* host_out, size_t bytes);

const char* ozaki2_status_string(int status);

/* Releases the internal workspaces of ozaki2_dgemm (synchronises). */
void ozaki2_finalize(void);

#ifdef __cplusplus
}
#endif
#endif /* OZAKI2_H */
