/*
 * kronq.h -- C ABI of the KronQ per-layer quantisation path for AMD MI355X (gfx950).
 *
 * KronQ (arxiv 2607.07964) quantises one linear layer W [d_out x d_in] with a
 * Kronecker-factored Hessian H ~ H_X (x) H_G. The path is:
 *   1. covariances H_X = X^T X and H_G = G^T G over N calibration tokens   (Sec. 4.1, eq. kfac);
 *   2. traces and the sensitivity score s = tr(H_G) tr(H_X)                (Sec. 4.3, eq. sensitivity);
 *   3. bidirectional incoherence processing: rescaling and randomised
 *      Hadamard rotations on both sides                                   (Sec. 4.2, eqs. rescale, biip; Alg. 1);
 *   4. damping and the inverse-Cholesky factor of H_X                      (Alg. 2, first lines);
 *   5. the column-wise OBS sweep with group quantisation, in lazy blocks   (eq. obs_update, Prop. 1; Alg. 2).
 * With the drift correction of GPTAQ (the paper's default, KronQ+GPTAQ; eqs. gptaq_obj,
 * kronq_full, kronq_update) the path also accumulates D = dX^T X (dX = X~ - X, the input drift),
 * transforms it with H_X's input-side BiIP, forms P = alpha ((D U^T) . M_U) U and sweeps with
 * W_j P[j, :] added to every compensation.
 *
 * Conventions (all entry points):
 *   - Matrices are row-major with an explicit leading dimension (elements). Pointers marked
 *     "device" are device memory owned by the caller; the library never frees them.
 *   - Every call is ordered on `stream` (a hipStream_t; NULL = the default stream), returns
 *     after enqueueing, and keeps no state between calls apart from the optional profiler.
 *   - Scratch memory comes from the caller: `ws` (device, 256-byte aligned) of `ws_bytes`
 *     bytes, at least kronq_workspace_bytes() for that operation. ws may be NULL when that
 *     size is 0.
 *   - Scalar results (traces, loss, info) are written to device memory; synchronise the
 *     stream before reading them.
 *   - Return value: KRONQ_OK or a negative KRONQ_ERR_* code; kronq_last_error() then holds a
 *     message (thread-local). Nothing is enqueued when an argument check fails.
 *
 * Readings of the paper that fix the semantics (the paper is silent or garbled there):
 *   covariances are plain sums; the inverse-Cholesky factor is the upper U with
 *   inv(H~) = U^T U and the sweep uses its rows; the paper's lower L (inv(H~) = L L^T) of the
 *   drift correction is U^T and its mask M_U is strictly upper; the drift term uses each column
 *   as it stood when it was quantised; the quantiser is the asymmetric min-max grid per row and
 *   group of columns (128, or wider up to the whole row: the per-channel grid),
 *   with scale = float32((xmax - xmin) / (2^b - 1)), zero = rint(-xmin / scale),
 *   q = clamp(rint(w / scale) + zero, 0, 2^b - 1), divisions in IEEE float64, rint half to even.
 */
#ifndef KRONQ_H
#define KRONQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------------------------- */
#define KRONQ_OK 0
#define KRONQ_ERR_INVALID_ARG (-1) /* null pointer, non-positive size, bad leading dim, misalignment */
#define KRONQ_ERR_SHAPE (-2)       /* sizes inconsistent with each other (e.g. d_in % group) */
#define KRONQ_ERR_NOT_PD (-3)      /* reported by the host binding after reading *info */
#define KRONQ_ERR_HIP (-4)         /* a HIP launch or runtime call failed */
#define KRONQ_ERR_WORKSPACE (-5)   /* ws_bytes smaller than kronq_workspace_bytes() */
#define KRONQ_ERR_UNSUPPORTED (-6) /* valid but not implemented: group not a multiple of 128,
                                      block != 128, rotated dimension not 2^k or 28 * 2^k */

/* ---- element types --------------------------------------------------------------------- */
#define KRONQ_BF16 1
#define KRONQ_FP32 2

/* ---- kronq_rotate flags ------------------------------------------------------------------ */
#define KRONQ_RESCALE_IN 1   /* S_X = diag(H_X,jj / ||W_:,j||^2)^(1/4)        (eq. rescale) */
#define KRONQ_RESCALE_OUT 2  /* S_G = diag(H_G,ii / ||W_i,:||^2)^(1/4)        (eq. rescale) */
#define KRONQ_ROT_IN 4       /* V: W <- W V^T, H_X <- V H_X V^T              (eq. biip)    */
#define KRONQ_ROT_OUT 8      /* U: W <- U W, H_G <- U H_G U^T                 (eq. biip)    */
#define KRONQ_INVERSE 16     /* revert W only: W <- S_G^-1 U^T W V S_X^-1     (Alg. 2, last line) */
#define KRONQ_BIIP (KRONQ_RESCALE_IN | KRONQ_RESCALE_OUT | KRONQ_ROT_IN | KRONQ_ROT_OUT)
/* Split forms of the forward transform, so that the H_X side (which the factorisation needs)
 * can run as soon as H_X exists while H_G is still being accumulated:
 *   KRONQ_HX_ONLY:  compute sx (from W_in and diag H_X) and transform H_X only; W (may be NULL),
 *                   H_G and sg are not touched.
 *   KRONQ_SX_GIVEN: sx is an input (from a KRONQ_HX_ONLY call with the same W_in); compute sg and
 *                   transform W and H_G; H_X is not touched (may be NULL).
 * HX_ONLY followed by SX_GIVEN gives exactly the result of one call without either flag.
 * The H_G side splits the same way, so that W (which the sweep needs) does not wait for H_G:
 *   KRONQ_HG_DIAG:  HG points at diag(H_G) only, d_out contiguous floats (ldg ignored; from
 *                   kronq_cov_diag or any other source); sg comes from it, W (and H_X unless
 *                   KRONQ_SX_GIVEN) is transformed, H_G is not. Not with KRONQ_HX_ONLY,
 *                   KRONQ_SG_GIVEN or KRONQ_INVERSE.
 *   KRONQ_SG_GIVEN: with KRONQ_SX_GIVEN only: sg is an input (from a KRONQ_HG_DIAG call);
 *                   transform H_G only. W_in and W are not read (may be NULL; d_out and d_in
 *                   still size the workspace).
 * HX_ONLY, then SX_GIVEN | HG_DIAG with diag(H_G), then SX_GIVEN | SG_GIVEN gives exactly the
 * result of one call without flags. */
#define KRONQ_HX_ONLY 32
#define KRONQ_SX_GIVEN 64
#define KRONQ_HG_DIAG 128
#define KRONQ_SG_GIVEN 256

/* ---- workspace queries ------------------------------------------------------------------- */
#define KRONQ_OP_COV 1
#define KRONQ_OP_ROTATE 2
#define KRONQ_OP_CHOL 3
#define KRONQ_OP_OBS 4
#define KRONQ_OP_LOSS 5
#define KRONQ_OP_CROSS 6         /* kronq_accumulate_cross: d as d_in, tokens as n_rows */
#define KRONQ_OP_ROTATE_DRIFT 7  /* kronq_rotate_drift: d_in */
#define KRONQ_OP_GPTAQ 8         /* kronq_gptaq_correction: d as d_in */
#define KRONQ_OP_OBS_DRIFT 9     /* kronq_obs_quantize_layer_drift: d_out, d_in */
#define KRONQ_OP_ONLINE 10       /* kronq_online_matvec: d_out, d_in, batch as n_rows */
#define KRONQ_OP_STATS 11        /* kronq_matrix_stats: rows as d_out, cols as d_in */
#define KRONQ_OP_EIGH 12         /* kronq_eigh: d as d_in */
#define KRONQ_OP_PROXY 13        /* kronq_proxy_loss_factors: d_out, d_in */
#define KRONQ_OP_COV_DIAG 14     /* kronq_cov_diag: d as d_in, tokens as n_rows */

/* Bytes of scratch the operation needs for these sizes. For KRONQ_OP_COV pass the covariance
 * dimension d as d_in and the token count as n_rows (d_out ignored); for KRONQ_OP_CHOL pass
 * the matrix order as d_in. Returns 0 for invalid sizes. Host only, never fails. */
size_t kronq_workspace_bytes(int op, int64_t d_out, int64_t d_in, int64_t n_rows);

/* Message of the last failed call on this thread ("" if none). */
const char* kronq_last_error(void);

/* Library version (major * 10000 + minor * 100 + patch). */
int kronq_version(void);

/* ---- 1. covariances (Sec. 4.1 eq. kfac; Alg. 1 first line; reading: plain sums) ----------
 * H <- beta * H + alpha * A^T A, for token-major A [n_rows x d] (X with d = d_in, or G with
 * d = d_out). The full symmetric d x d matrix is written. Calls can be chained over token
 * chunks with beta = 1. beta = 0 never reads H (NaNs in it do not propagate).
 *   A     device, dtype KRONQ_BF16 (products exact in fp32, fp32 accumulation on MFMA) or
 *         KRONQ_FP32 (fp32 FMA); rows of lda elements; A and lda*elem_size 16-byte aligned.
 *   H     device fp32 [d x ldh], ldh >= d.
 *   n_rows may be 0 (then H <- beta * H). */
int kronq_accumulate_cov(const void* A, int dtype, int64_t n_rows, int64_t d, int64_t lda,
                         float* H, int64_t ldh, float alpha, float beta, void* ws,
                         size_t ws_bytes, void* stream);

/* As kronq_accumulate_cov, with the bf16 interior-tile kernel holding at most max_cus compute
 * units at once (persistent workgroups, one per CU, rounded down to a multiple of 8; 0: the
 * whole chip). For a caller that runs latency-bound work on another stream meanwhile (the
 * factorisation beside the H_G covariance): a covariance workgroup holds its CU for the whole
 * of its tile, so without a cap the other stream's kernels wait for CUs. The token slices
 * (split-K) are chosen to fill whole rounds of the capped workgroups, never more slices than
 * kronq_accumulate_cov takes (so the same workspace serves), so the result equals
 * kronq_accumulate_cov's up to the order of the fp32 sums, and bit for bit when both choose the
 * same slices. max_cus < 0: KRONQ_ERR_INVALID_ARG. */
int kronq_accumulate_cov_limited(const void* A, int dtype, int64_t n_rows, int64_t d,
                                 int64_t lda, float* H, int64_t ldh, float alpha, float beta,
                                 int max_cus, void* ws, size_t ws_bytes, void* stream);

/* ---- 1a. covariance diagonal (Sec. 4.1 eq. kfac; the h of eq. rescale) --------------------
 * hdiag[j] = sum_t A[t][j]^2 = (A^T A)_jj for token-major A [n_rows x d], without the
 * covariance: one read of A at HBM speed. Squares are summed in fp64 (exact products for bf16)
 * and rounded once to fp32; the summation order is fixed, so the result is reproducible bit
 * for bit. For a caller that needs a side's rescaling (KRONQ_HG_DIAG) before that side's
 * covariance exists.
 *   A      device, KRONQ_BF16 or KRONQ_FP32, rows of lda elements; A 16-byte aligned, lda
 *          divisible by 8 (bf16) or 4 (fp32).
 *   hdiag  device fp32 [d], written. n_rows = 0 writes zeros (A may then be NULL).
 *   max_cus  0: enough workgroups to fill the chip; > 0: at most max(max_cus, ceil(d / 512))
 *          workgroups, for a caller that runs latency-bound work beside it (the result is the
 *          same either way up to the order of the fp64 sums). < 0: KRONQ_ERR_INVALID_ARG.
 *   ws     kronq_workspace_bytes(KRONQ_OP_COV_DIAG, 0, d, n_rows) bytes. */
int kronq_cov_diag(const void* A, int dtype, int64_t n_rows, int64_t d, int64_t lda,
                   float* hdiag, int max_cus, void* ws, size_t ws_bytes, void* stream);

/* kronq_cov_diag without a workspace and without allocating, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc). Same arguments, kernels and result (bit for bit) as kronq_cov_diag. The chunk
 * partials live in a fixed device array of KRONQ_NOALLOC_SCRATCH_BYTES inside the library, one
 * copy per GPU, held until the process ends; its address on a device is taken once, on the
 * first call for that device (the stream's device; the current one for the NULL stream). The
 * call allocates nothing and calls no allocating routine. Every call on a GPU shares that
 * GPU's array: calls that overlap on one GPU (other streams, other threads) race and must be
 * ordered by the caller. Nothing in the array needs to start at zero: each call writes every
 * partial it reads. Sizes whose partials exceed the array (for any d <= 2^21 they fit: at
 * most 512 x 4096 partial sums) return KRONQ_ERR_WORKSPACE before anything is enqueued. */
#define KRONQ_NOALLOC_SCRATCH_BYTES (16u << 20)
int kronq_cov_diag_noalloc(const void* A, int dtype, int64_t n_rows, int64_t d, int64_t lda,
                           float* hdiag, int max_cus, void* stream);

/* ---- 1b. drift statistic (Alg. 1 first line; eq. gptaq_obj) ------------------------------
 * C <- beta * C + alpha * A^T B for token-major A, B [n_rows x d] with the same leading
 * dimension ld; every entry of the d x d matrix C is written (it is not symmetric). With
 * A = dX (the full-precision model's input minus the quantised model's, bf16) and B = X this
 * is the paper's dX X^T. Chainable over token chunks with beta = 1, like kronq_accumulate_cov.
 *   A, B  device, dtype KRONQ_BF16 (exact products, fp32 accumulation on MFMA) or KRONQ_FP32;
 *         16-byte aligned, ld * elem_size a multiple of 16 for bf16.
 *   C     device fp32 [d x ldc], ldc >= d. Workspace: KRONQ_OP_CROSS. */
int kronq_accumulate_cross(const void* A, const void* B, int dtype, int64_t n_rows, int64_t d,
                           int64_t ld, float* C, int64_t ldc, float alpha, float beta, void* ws,
                           size_t ws_bytes, void* stream);

/* As kronq_accumulate_cross, with the bf16 interior-tile kernel holding at most max_cus compute
 * units at once (as kronq_accumulate_cov_limited: persistent workgroups, a multiple of 8; 0: the
 * whole chip), for a caller that runs the factorisation on another stream meanwhile. Token
 * slices as kronq_accumulate_cov_limited chooses them, so the result equals
 * kronq_accumulate_cross's up to the order of the fp32 sums (bit for bit when both take the
 * same slices). max_cus < 0: KRONQ_ERR_INVALID_ARG. */
int kronq_accumulate_cross_limited(const void* A, const void* B, int dtype, int64_t n_rows,
                                   int64_t d, int64_t ld, float* C, int64_t ldc, float alpha,
                                   float beta, int max_cus, void* ws, size_t ws_bytes,
                                   void* stream);

/* ---- 2. traces and sensitivity (Sec. 4.3 eq. sensitivity) --------------------------------
 * out3[0] = tr H_X, out3[1] = tr H_G, out3[2] = tr H_X * tr H_G, accumulated in fp64.
 * Call before and/or after kronq_rotate (the score of the paper uses post-BiIP traces).
 *   HX device fp32 [d_in x ldx]; HG device fp32 [d_out x ldg]; out3 device double[3]. */
int kronq_traces(const float* HX, int64_t d_in, int64_t ldx, const float* HG, int64_t d_out,
                 int64_t ldg, double* out3, void* stream);
/* Either matrix may be NULL: its slot of out3 is then taken as already holding that trace
 * (written by an earlier call on the same out3, ordered before this one), and out3[2] is the
 * product of the two slots. This lets the two traces be taken on different streams. */

/* ---- 3. bidirectional incoherence processing (Sec. 4.2 eqs. rescale, biip; Alg. 1) -------
 * Forward (no KRONQ_INVERSE):
 *   a_j = ||W_in[:, j]||^2, b_i = ||W_in[i, :]||^2 (original W), sx_j = (H_X,jj / a_j)^(1/4),
 *   sg_i = (H_G,ii / b_i)^(1/4) (1 when a side is off or a norm/diagonal is 0);
 *   W  <- U diag(sg) W_in diag(sx) V^T                 (written to W, fp32)
 *   HX <- V diag(1/sx) HX diag(1/sx) V^T               (in place)
 *   HG <- U diag(1/sg) HG diag(1/sg) U^T               (in place, skipped if HG is NULL)
 * with V = H_{d_in} diag(sign_in) / sqrt(d_in) for d_in = 2^k, or
 * (Q28_in (x) H_{d_in/28} / sqrt(d_in/28)) diag(sign_in) for d_in = 28 * 2^k (28-point factor
 * on the slow index), and U likewise from sign_out / q28_out. H is the Sylvester Hadamard.
 * Inverse (KRONQ_INVERSE, W only, sx and sg are inputs):
 *   W <- diag(1/sg) U^T W_in V diag(1/sx).
 *   W_in   device, w_dtype KRONQ_BF16 or KRONQ_FP32, [d_out x ldw_in], 16-byte aligned rows
 *          (ldw_in divisible by 8 for bf16, by 4 for fp32); may alias W when fp32.
 *   W      device fp32 [d_out x ldw].
 *   HX     device fp32 [d_in x ldx] (forward; may be NULL for INVERSE).
 *   HG     device fp32 [d_out x ldg] or NULL; required by KRONQ_RESCALE_OUT (with
 *          KRONQ_HG_DIAG: fp32 [d_out], the diagonal only).
 *   sign_in/sign_out  device int8 (+1/-1) [d_in]/[d_out]; required when that side rotates.
 *   q28_in/q28_out    device fp32 [28 x 28] row-major; required iff that dimension is
 *                     28 * 2^k and rotates; ignored otherwise.
 *   sx/sg  device fp32 [d_in]/[d_out]: outputs (forward), inputs (inverse; sx with
 *          KRONQ_SX_GIVEN, sg with KRONQ_SG_GIVEN).
 * Rotated dimensions must be 2^k (k >= 1) or 28 * 2^k with 2^k <= 16384. */
int kronq_rotate(const void* W_in, int w_dtype, int64_t ldw_in, float* W, int64_t d_out,
                 int64_t d_in, int64_t ldw, float* HX, int64_t ldx, float* HG, int64_t ldg,
                 const int8_t* sign_in, const int8_t* sign_out, const float* q28_in,
                 const float* q28_out, float* sx, float* sg, int flags, void* ws,
                 size_t ws_bytes, void* stream);

/* ---- 3b. BiIP of the drift statistic (Alg. 1; Sec. 4.2) -------------------------------------
 * D <- V diag(1/sx) D diag(1/sx) V^T, the input-side transform that kronq_rotate applies to H_X,
 * for the drift statistic (the objective eq. kronq_full is then unchanged).
 *   D       device fp32 [d_in x ldd], in place (16-byte aligned, ldd % 4 == 0).
 *   sx      device fp32 [d_in] from the forward kronq_rotate; read with KRONQ_RESCALE_IN.
 *   sign_in, q28_in  the input-side rotation draw (as for kronq_rotate); read with KRONQ_ROT_IN.
 *   flags   a subset of KRONQ_RESCALE_IN | KRONQ_ROT_IN (the input-side flags of that call).
 * Workspace: KRONQ_OP_ROTATE_DRIFT. */
int kronq_rotate_drift(float* D, int64_t d_in, int64_t ldd, const float* sx,
                       const int8_t* sign_in, const float* q28_in, int flags, void* ws,
                       size_t ws_bytes, void* stream);

/* ---- 4. damping + inverse-Cholesky factor (Alg. 2 first two lines; Prop. 1) --------------
 * H <- H + damp_rel * mean(diag H) * I (in place), then Uout = upper-triangular U with
 * inv(H) = U^T U (zeros below the diagonal are written). U = R^-1 where H = R R^T, R upper
 * (a Cholesky factorisation in reversed index order followed by a triangular inverse, fp32).
 *   H    device fp32 [d x ldh], symmetric (both triangles read).
 *   Uout device fp32 [d x ldu]; must not alias H.
 *   info device int32: 0 on success, else the 1-based column of H (original order) whose
 *        pivot was not positive; Uout is then undefined. The host reads it after a sync. */
int kronq_cholesky_inv(float* H, int64_t d, int64_t ldh, float damp_rel, float* Uout,
                       int64_t ldu, int* info, void* ws, size_t ws_bytes, void* stream);

/* ---- 4b. drift correction (Prop. 1 eq. kronq_update; Alg. 2 third line) ------------------
 * P = alpha ((D U^T) . M_U) U with U from kronq_cholesky_inv (the paper's L is U^T) and M_U the
 * strictly upper mask; P is strictly upper triangular (zeros on and below the diagonal are
 * written). Row p of P is alpha D[p, p+1:] inv(H~[p+1:, p+1:]). fp32 products, 2 d^3 / 3 flops.
 *   D  device fp32 [d x ldd]: the transformed drift statistic (kronq_rotate_drift).
 *   U  device fp32 [d x ldu], upper.   P  device fp32 [d x ldp]; must not alias D or U.
 *   All 16-byte aligned with leading dimensions divisible by 4. Workspace: KRONQ_OP_GPTAQ. */
int kronq_gptaq_correction(const float* D, int64_t d, int64_t ldd, const float* U, int64_t ldu,
                           float alpha, float* P, int64_t ldp, void* ws, size_t ws_bytes,
                           void* stream);

/* ---- 5. lazy-block column-wise OBS with group quantisation (Alg. 2 with P = 0) -----------
 * For each block of `block` columns and each column p in it: group parameters per row are
 * taken from the current W when p is a group start; q = quant(W[:, p]);
 * e_p = (W[:, p] - w_hat_p) / U[p, p]; W[:, p:blk_end] -= e_p U[p, p:blk_end]; after the
 * block W[:, blk_end:] -= E_blk U[blk, blk_end:]. Column p is left holding w_hat_p.
 *   W      device fp32 [d_out x ldw], consumed (ends as the dequantised W_hat).
 *   U      device fp32 upper [d_in x ldu] from kronq_cholesky_inv.
 *   bits   2 to 8; block must be 128; group a multiple of 128 dividing d_in (group = d_in is
 *          the per-channel grid: one scale and zero per row, from the row before the sweep).
 *   codes  device uint8 [d_out x d_in] (ld = d_in), one code per byte.
 *   scales, zeros  device fp32 [d_out x d_in/group] (zeros are integer-valued).
 *   err    device fp32 [d_out x d_in] or NULL: the scaled errors e (ld = d_in).
 *   W_hat  device fp32 [d_out x d_in] or NULL: a copy of the dequantised values (ld = d_in). */
int kronq_obs_quantize_layer(float* W, int64_t d_out, int64_t d_in, int64_t ldw,
                             const float* U, int64_t ldu, int bits, int group, int block,
                             uint8_t* codes, float* scales, float* zeros, float* err,
                             float* W_hat, void* ws, size_t ws_bytes, void* stream);

/* ---- 5b. the sweep with the drift correction (Alg. 2; Prop. 1 eq. kronq_update) ------------
 * As kronq_obs_quantize_layer, with every compensation of the sweep and of the trailing updates
 * also adding w_p P[p, cols] (w_p: column p as it stood when it was quantised):
 * W[:, p:blk_end] += w_p P[p, p:blk_end]; after the block W[:, blk_end:] += W_blk P[blk, blk_end:].
 *   P  device fp32 [d_in x ldp] from kronq_gptaq_correction (strictly upper), not NULL.
 * Workspace: KRONQ_OP_OBS_DRIFT. */
int kronq_obs_quantize_layer_drift(float* W, int64_t d_out, int64_t d_in, int64_t ldw,
                                   const float* U, int64_t ldu, const float* P, int64_t ldp,
                                   int bits, int group, int block, uint8_t* codes, float* scales,
                                   float* zeros, float* err, float* W_hat, void* ws,
                                   size_t ws_bytes, void* stream);

/* ---- 7. inference with the quantised layer (Sec. 3.2, 4.2; Limitations; Alg. 2 last line) ----
 * The rotations are applied online around a matvec on the packed codes:
 *   y = S_G^-1 U^T W_hat' V S_X^-1 x,   W_hat' = scale * (code - zero) per row and group,
 * i.e. the original-space dequantised layer, without forming it.
 *
 * kronq_pack_codes: codes uint8 [d_out x ldq] (from the sweep) -> packed uint32 [d_out x ldp]:
 * each run of 32 consecutive codes of a row becomes one 32 * bits-bit little-endian string
 * (code j at bits [j * bits, (j + 1) * bits)) in `bits` words; ldp >= d_in * bits / 32.
 * bits in {2, 3, 4, 8}; d_in a multiple of 32; packed 4-byte aligned. */
int kronq_pack_codes(const uint8_t* codes, int64_t d_out, int64_t d_in, int64_t ldq, int bits,
                     uint32_t* packed, int64_t ldp, void* stream);

/* mul[j] = sign[j] / s[j] (a NULL sign or s counts as 1): the multipliers of the online
 * transforms, mul_in from (sx, sign_in) and mul_out from (sg, sign_out). mul: device fp32 [d],
 * 16-byte aligned. */
int kronq_online_factors(const float* s, const int8_t* sign, int64_t d, float* mul, void* stream);

/* y[b] = diag(mul_out) T_out W_hat' T_in diag(mul_in) x[b] for b < batch, where
 * T_in = V diag(sign_in)^-1 (the Hadamard factor (Q28_in (x) H) / sqrt(m), with KRONQ_ROT_IN) and
 * T_out = (Q28_out^T (x) H) / sqrt(m) (with KRONQ_ROT_OUT); with the factors of
 * kronq_online_factors this is S_G^-1 U^T W_hat' V S_X^-1 x. Other flag bits of KRONQ_BIIP are
 * accepted and ignored (the rescaling is inside mul_in, mul_out).
 *   packed  device uint32 [d_out x ldp] from kronq_pack_codes; 16-byte aligned, ldp % 4 == 0.
 *   scales, zeros  device fp32 [d_out x ldsz], one per row and group (group a multiple of 128
 *           dividing d_in; d_in: per-channel).
 *   mul_in [d_in], mul_out [d_out]  device fp32, 16-byte aligned, or NULL (1).
 *   q28_in, q28_out  as for kronq_rotate, required when that side rotates a 28 * 2^k dimension.
 *   x       device [batch x ldx], KRONQ_BF16 or KRONQ_FP32, 16-byte aligned rows.
 *   y       device fp32 [batch x ldy], 16-byte aligned, ldy % 4 == 0.
 *   1 <= batch <= 4, batch * d_in <= 32768, d_out <= 32768. Workspace: KRONQ_OP_ONLINE. */
int kronq_online_matvec(const uint32_t* packed, int64_t ldp, const float* scales,
                        const float* zeros, int64_t ldsz, int bits, int group, int64_t d_out,
                        int64_t d_in, const float* mul_in, const float* mul_out,
                        const float* q28_in, const float* q28_out, int flags, const void* x,
                        int x_dtype, int64_t ldx, int64_t batch, float* y, int64_t ldy, void* ws,
                        size_t ws_bytes, void* stream);

/* ---- 8. diagnostics of the incoherence processing ------------------------------------------
 * (Sec. 2.3 eq. incoherence_measure; Sec. 4.2 and Fig. 2; Prop. 2 eq. biip-bound, appendix A.3
 * and its optimality table.) Sums are taken in fp64; results land in device memory. */

/* out[5] = {max |M_ij|, ||M||_F^2, mu(M) = sqrt(rows cols) max |M_ij| / ||M||_F, CV_in, CV_out}:
 * CV_in and CV_out are the population coefficients of variation (std / mean) of the column
 * norms ||M_:,j|| and of the row norms ||M_i,:|| (Fig. 2b; the norms, not their squares).
 *   M    device [rows x ld], dtype KRONQ_BF16 or KRONQ_FP32, 4-byte aligned; rows, cols >= 1.
 *   out  device double[5]. Workspace: KRONQ_OP_STATS (rows as d_out, cols as d_in). */
int kronq_matrix_stats(const void* M, int dtype, int64_t rows, int64_t cols, int64_t ld,
                       double* out, void* ws, size_t ws_bytes, void* stream);

/* Eigendecomposition of the symmetric H (the eigenvector matrix Q of mu(H) = sqrt(d) max |Q_ij|,
 * eq. incoherence_measure) by block Jacobi in fp32: the order is padded to a multiple of 64
 * and split into blocks of 32 indices; a sweep visits every pair of blocks once (round-robin,
 * d/32 - 1 rounds of disjoint pairs), diagonalising the pair's 64 x 64 submatrix by one cyclic
 * sweep of scalar rotations (skipped once |a_pq| <= 1e-7 sqrt(|a_pp a_qq|)) and applying the
 * accumulated rotation to the whole matrix and to the eigenvectors.
 *   H      device fp32 [d x ldh], symmetric (read only; both triangles are read).
 *   sweeps 1..64 sweeps (about 12 reach the fp32 floor at d = 4096).
 *   evals  device fp32 [d]: the eigenvalues, unsorted; Q device fp32 [d x ldq], column k the
 *          unit eigenvector of evals[k]. Q must not overlap H.
 *   off    device double[1]: ||offdiag(Q^T H Q)||_F / ||H||_F after the last sweep, the
 *          convergence measure.
 *   1 <= d <= 16384. Workspace: KRONQ_OP_EIGH (d as d_in): three N x N fp32 matrices,
 *   N = d rounded up to a multiple of 64. */
int kronq_eigh(const float* H, int64_t d, int64_t ldh, int sweeps, float* evals, float* Q,
               int64_t ldq, double* off, void* ws, size_t ws_bytes, void* stream);

#define KRONQ_MAX_ALPHAS 16

/* The expected-loss factors of Prop. 2 and the optimality table, for h_i = [H_G]_ii and
 * a_i = ||W_i,:||^2 of the layer before BiIP, D_p = 1 / U_pp^2 the pivots the sweep divides by
 * (U the inverse-Cholesky factor of the damped post-BiIP H~, so D_p = 1 / [inv(H~[p:,p:])]_00):
 *   out[0] = (sum h)(sum a) tr(H~)       nearest rounding
 *   out[1] = (sum h)(sum a) tr(D)        GPTQ
 *   out[2] = (sum sqrt(h a))^2 tr(D)     KronQ
 *   out[3] = rho = (sum sqrt(h a))^2 / ((sum h)(sum a)),  out[4] = tr(D),  out[5] = tr(H~)
 *   out[6 + k] = (sum h / s^2)(sum s^2 a) tr(D) with s_i = (h_i / a_i)^alphas[k] (1 where
 *                h_i a_i = 0): the exponent sweep, minimal at alpha = 1/4.
 *   HG  device fp32 [d_out x ldg] (its diagonal is read); W device [d_out x ldw], w_dtype
 *       KRONQ_BF16 or KRONQ_FP32; Hd, U device fp32 [d_in x ldh], [d_in x ldu] (diagonals).
 *   alphas HOST double[n_alpha], 0 <= n_alpha <= KRONQ_MAX_ALPHAS; out device double[6 + n_alpha].
 *   Workspace: KRONQ_OP_PROXY (d_out, d_in). */
int kronq_proxy_loss_factors(const float* HG, int64_t d_out, int64_t ldg, const void* W,
                             int w_dtype, int64_t ldw, int64_t d_in, const float* Hd, int64_t ldh,
                             const float* U, int64_t ldu, const double* alphas, int n_alpha,
                             double* out, void* ws, size_t ws_bytes, void* stream);

/* ---- 6. K-FAC loss (Sec. 4.1 eq. kron_obj) -----------------------------------------------
 * loss = tr(H_G dW H_X dW^T) = sum_ij (H_G dW)_ij (dW H_X)_ij with dW = W - W_hat (W_hat NULL:
 * dW = W), fp32 products with fp32 accumulation and an fp64 final sum.
 *   W     device [d_out x ldw], w_dtype KRONQ_BF16 or KRONQ_FP32.
 *   W_hat device fp32 [d_out x ldwh] or NULL.
 *   HX, HG device fp32 (ldx, ldg). loss device double[1]. */
int kronq_layer_loss(const void* W, int w_dtype, int64_t ldw, const float* W_hat,
                     int64_t ldwh, int64_t d_out, int64_t d_in, const float* HX, int64_t ldx,
                     const float* HG, int64_t ldg, double* loss, void* ws, size_t ws_bytes,
                     void* stream);

/* ---- mixed-precision allocation (Sec. 4.3, Sec. 5.5) -------------------------------------
 * Host only. Chooses bits_out[l] in `choices` minimising sum_l scores[l] / (2^b_l - 1)^2
 * subject to sum_l weights[l] * b_l <= avg_bits * sum_l weights[l] (weights = parameter
 * counts for a parameter-weighted budget, or 1 for a count-weighted one), by exhaustive
 * search in lexicographic order of the sorted choices; ties keep the first (smallest) vector.
 * n_layers <= 12, n_choices <= 8. objective_out (nullable) receives the minimum. */
int kronq_allocate_bits(const double* scores, const int64_t* weights, int n_layers,
                        const int* choices, int n_choices, double avg_bits, int* bits_out,
                        double* objective_out);

/* ---- measured matrix-core ceiling (measurement support, not a step of the layer) ----------
 * The clock of the chip is power-limited under matrix-core load, and the limit depends on the
 * operand values; this measures the bf16 MFMA rate reachable on given data. Launches two
 * workgroups of 4 waves per compute unit; each wave runs `iters` iterations of 8 independent
 * v_mfma_f32_32x32x16_bf16 on 4 register fragments read once from `data`, with no memory
 * access inside the loop. Time the launch on the stream; it performs
 * (*workgroups) * 4 * iters * 8 * 32768 flops.
 *   data        device bf16 [>= 4096], 16-byte aligned (the operand values).
 *   iters       >= 1.
 *   out         device fp32 [out_len]: one checksum per workgroup (keeps the loop alive).
 *   workgroups  host int*, receives the workgroup count (2 x compute units); out_len must be at
 *               least that, else KRONQ_ERR_INVALID_ARG before any launch. */
int kronq_probe_mfma_bf16(const void* data, int iters, float* out, int64_t out_len,
                          int* workgroups, void* stream);

/* ---- profiler (hipEvent timing of every kernel launch, by kernel name) --------------------
 * While enabled, each launch is bracketed by two events on its stream. kronq_profile_read
 * synchronises the recorded events and returns the summed milliseconds and the launch count
 * of the named kernel (0 if never launched). Not thread-safe; meant for benchmarks. */
int kronq_profile_enable(int on);
/* Restrict the profiler to launches of the named kernels (one name or a comma-separated list;
 * NULL or "": every kernel), so that timing them adds no events around the others. */
int kronq_profile_only(const char* kernel);
void kronq_profile_reset(void);
int kronq_profile_read(const char* kernel, double* total_ms, int64_t* launches);
/* Names of the kernels recorded since the last reset, comma-separated, into buf (capacity
 * cap bytes, always NUL-terminated when cap > 0; truncated if short). Returns the length the
 * full list needs, without the terminator. */
int64_t kronq_profile_names(char* buf, size_t cap);

#ifdef __cplusplus
}
#endif

#endif /* KRONQ_H */
