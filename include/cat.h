/*
 * cat.h -- C ABI of the block Concentration-Alignment Transform (CAT)
 * W4A4 linear-layer library for MI355X (gfx950).
 *
 * Paper: "Dissecting Quantization Error: A Concentration-Alignment
 * Perspective" (Federici, van Breugel, Whatmough, Nagel).  The layer is
 * factored as Q(W T^-1) Q(T x) (Sec. 3, eq. 5), with T the block-diagonal
 * transform T_b = H_k M_b of Sec. 4, eq. 10, whose blocks M_b come from the
 * calibration second moment Sigma_x = E[x x^T] and Sigma_w = W^T W (eq. 7).
 * The quality measure is the output SQNR of Sec. 2, eq. 1.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Return value: CAT_OK (0) or a negative cat_status.  On failure
 *    cat_last_error() returns a thread-local message.  No C++ exception
 *    crosses this boundary.
 *  - Device calls (cov_accumulate, transform_quant, w4a4_linear, sqnr)
 *    take DEVICE pointers, validate their arguments on the host, enqueue
 *    kernels on `stream` (a hipStream_t passed as void*; NULL = the null
 *    stream) and return without synchronising.  Results are visible after
 *    the caller synchronises that stream.  Asynchronous faults surface at
 *    that synchronisation.  They never allocate: scratch memory comes from
 *    a caller-owned workspace whose size a *_workspace_bytes() query gives.
 *  - Host calls (build_transform, quantize_weights) take HOST pointers,
 *    run synchronously on the CPU in fp64 and touch no GPU.
 *  - Ownership: every buffer belongs to the caller; the library keeps no
 *    pointer after a call returns.
 *  - Layout: all matrices row-major and densely packed (leading dimension
 *    = row length).  Device pointers must be 16-byte aligned.
 *  - Packed INT4: byte j of a row holds element 2j in bits 0-3 and element
 *    2j+1 in bits 4-7, two's complement; codes lie in [-7, 7].
 *  - 6- and 8-bit codes (the W6A6 / W8A8 comparison widths): one int8 per
 *    element, codes in [-31, 31] or [-127, 127].
 *  - Calls are stateless and may be issued from several threads.
 *  - NaN / Inf inputs give undefined (but memory-safe) results.  So do
 *    rows the fp32 quantizer cannot represent: a token whose transformed
 *    values z all lie below qmax * 2^-128 in magnitude (about 2e-38 at 4
 *    bits; the reciprocal qmax / amax overflows) or whose z overflows fp32.
 */
#ifndef CAT_H
#define CAT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CAT_OK = 0,
    CAT_ERR_INVALID_ARG = -1,   /* null pointer, bad size, misalignment */
    CAT_ERR_UNSUPPORTED = -2,   /* valid but not implemented (e.g. bits) */
    CAT_ERR_WORKSPACE = -3,     /* workspace missing or too small */
    CAT_ERR_HIP = -4,           /* HIP runtime / launch failure */
    CAT_ERR_INTERNAL = -5,      /* anything else (e.g. host allocation) */
    CAT_ERR_TIMEOUT = -6        /* an exchange wait ran out (status queries) */
} cat_status;

typedef enum {
    CAT_F32 = 0,                /* IEEE binary32 */
    CAT_BF16 = 1                /* bfloat16 (upper half of a binary32) */
} cat_dtype;

/* cat_cov_accumulate modes */
#define CAT_COV_FULL 0          /* the whole d x d matrix */
#define CAT_COV_BLOCK_DIAG 1    /* only the d/k diagonal k x k blocks */

/* cat_build_transform flags */
#define CAT_BUILD_HADAMARD 1    /* left factor H_k (normalised Sylvester) */
#define CAT_BUILD_ALIGN 2       /* right factor M_b (alignment-optimal) */
#define CAT_BUILD_CAT (CAT_BUILD_HADAMARD | CAT_BUILD_ALIGN)

/* Largest supported d_in of cat_w4a4_linear: keeps the int32 accumulator
 * exact (49 * 256 * d_in < 2^31 with the in-register 16x code unpack). */
#define CAT_MAX_D_IN 131072
#define CAT_MAX_BLOCK 512

/* ------------------------------------------------------------------ (1)
 * Calibration second moment (Sec. 4: Sigma_x = E[x x^T], non-centred;
 * Sec. 6 "Calibration").
 *
 *   acc += X^T X        (an unnormalised sum; divide by the total token
 *                         count afterwards)
 *
 * X     device, [n x d] row-major, x_dtype (CAT_BF16 or CAT_F32).
 * n     tokens in this batch, n >= 1.  Calling again on the same acc
 *       continues the accumulation (split batches give the one-shot sum up
 *       to fp32 rounding).
 * d     channels, 1 <= d, d % k == 0.
 * mode  CAT_COV_FULL: acc is [d x d] fp32, both triangles written (the
 *       kernels compute the upper triangle and mirror it).
 *       CAT_COV_BLOCK_DIAG: acc is [d/k x k x k] fp32, block b holding
 *       X[:, bk:(b+1)k]^T X[:, bk:(b+1)k].
 * k     block size: power of two in [1, CAT_MAX_BLOCK] (only read in
 *       CAT_COV_BLOCK_DIAG mode).
 * acc   device fp32, caller-owned, read and written.  It must be symmetric
 *       on entry (zero, or the result of earlier calls): for matrices of
 *       256 channels or more the strictly lower triangle is rewritten as
 *       the transpose of the updated upper triangle.  Products are formed
 *       exactly (bf16) and summed in fp32 in register partials over at most
 *       8192 tokens, which are added into acc in a fixed order: results are
 *       deterministic for a given device.
 * workspace, workspace_bytes
 *       device scratch of at least cat_cov_workspace_bytes() bytes, 16-byte
 *       aligned, caller-owned (partial tiles of workgroups that share a
 *       tile); may be NULL when that size is 0.  One workspace must not be
 *       used by calls that run concurrently.
 * Errors: CAT_ERR_INVALID_ARG (NULL X/acc, bad sizes, mode, k, alignment),
 *       CAT_ERR_WORKSPACE (workspace missing or too small), CAT_ERR_HIP.
 */
/* Workspace size for cat_cov_accumulate with these arguments on the
 * current device (it scales with the device's CU count; 0 for
 * configurations that need none, or when the arguments are invalid or no
 * device is present). */
size_t cat_cov_workspace_bytes(int x_dtype, int64_t n, int64_t d, int mode, int64_t k);
int cat_cov_accumulate(const void* X, int x_dtype, int64_t n, int64_t d,
                       int mode, int64_t k, float* acc, void* workspace,
                       size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ (2)
 * Block transform fused with symmetric per-token quantization
 * (Sec. 3, eq. 5: Q(T x); Sec. 4, eq. 10: T = blockdiag(T_1..T_{d/k});
 * Lemma 2.2: symmetric range r(x) = 2 max|x_i|; Sec. 6: dynamic per-token
 * activation quantization).
 *
 * For every token t (row of X) and block b:
 *   z[t, bk+j] = sum_i T_b[j, i] * X[t, bk+i]        (fp32 accumulation)
 *   amax[t]    = max over the WHOLE row of |z[t, :]|
 *   s_x[t]     = amax / qmax,  qmax = 2^(bits-1) - 1    (fp32, rounded)
 *   inv        = qmax / amax                          (fp32, rounded)
 *   code       = clamp(rint(z * inv), -qmax, qmax)     (ties to even)
 * A row with amax == 0 gets s_x = 0 and all-zero codes.
 *
 * X        device [n x d], x_dtype.
 * T        device [d/k x k x k], t_dtype; block b row-major (row j = output j).
 * k        power of two in [1, CAT_MAX_BLOCK]; d % k == 0; d even.
 * bits     4, 6 or 8 (other widths return CAT_ERR_UNSUPPORTED).
 * codes    device, written: bits 4: uint8 [n x d/2] packed INT4;
 *          bits 6, 8: int8 [n x d], one code per byte.
 * s_x      device fp32 [n] (written).
 * workspace / workspace_bytes: device scratch of at least
 *          cat_transform_quant_workspace_bytes(n, d, k) bytes; its
 *          contents on entry are ignored and on exit undefined.  One
 *          workspace must not be used by calls that run concurrently.
 * Capture: the call may be captured into a HIP graph and replayed (it
 *          enqueues kernels only; a captured call also enqueues a one-thread
 *          kernel that renews the exchange tag for every replay).
 * The bf16 path with k = 128 and d = 2048, 4096 or 8192 runs one
 * persistent launch whose workgroups exchange row maxima through the
 * workspace with bounded waits.
 * Its grid never exceeds the device's resident capacity, so every wait ends
 * once the launch has the device; work from other streams that holds CUs
 * for seconds can still make a wait run out.  In particular, two such calls
 * (cat_transform_quant, _asym or _noalloc) must not run at the same time on
 * one device: each may hold CUs that the other's waiting workgroups need.
 * Issue them on one stream, or order them with events.  When a wait runs
 * out, the 32-bit word at byte offset cat_transform_quant_flag_offset(n, d,
 * k) of the workspace is set to a non-zero value, and the call's results
 * must be treated as invalid.
 * No wrong scale is ever used even then: every workgroup reads a token's
 * row maximum on its own and uses the exact value or NaN, so each
 * 128-channel block of a token's codes is exact or (where that block's
 * wait ran out) zero, and s_x is exact or NaN.  The library never clears
 * that word: a caller that wants to check it zeroes it before the call and
 * reads it after synchronising.
 */
size_t cat_transform_quant_workspace_bytes(int64_t n, int64_t d, int64_t k);
/* Byte offset, inside a workspace of cat_transform_quant_workspace_bytes
 * (n, d, k) bytes, of the exchange timeout word described above (0 when the
 * arguments are invalid). */
size_t cat_transform_quant_flag_offset(int64_t n, int64_t d, int64_t k);
/* Status query for the exchange timeout word (no passage of the paper: a
 * property of this library's single-pass exchange).  Waits for every call
 * issued to `stream` so far, reads the word at
 * cat_transform_quant_flag_offset(n, d, k) of `workspace` and clears it.
 * Returns CAT_OK when it was zero and CAT_ERR_TIMEOUT when a wait of a call
 * of that shape on this workspace ran out since the word was last cleared
 * (those calls' results are invalid, as described above).  workspace
 * device, at least cat_transform_quant_workspace_bytes(n, d, k) bytes (or
 * the asymmetric size, whose word lies at the same offset).  It
 * synchronises, so it must not be captured into a graph.  Errors:
 * CAT_ERR_INVALID_ARG (NULL workspace, n or d < 1), CAT_ERR_HIP. */
int cat_transform_quant_status(const void* workspace, int64_t n, int64_t d, int64_t k,
                               void* stream);
/* Testing hook (no passage of the paper): bounds the polls of every wait in
 * the single-pass exchange of later cat_transform_quant and
 * cat_transform_quant_asym calls, process-wide.  0 restores the default
 * (2^22, seconds of waiting); larger values are clamped to it.  A small
 * bound makes waits run out as described above, so that tests can check
 * that a timeout yields exact or NaN scales, exact or zero code blocks and
 * the flag word, with every kernel still finishing normally. */
void cat_set_exchange_spin_limit(uint32_t polls);
int cat_transform_quant(const void* X, int x_dtype, int64_t n, int64_t d,
                        const void* T, int t_dtype, int64_t k, int bits,
                        uint8_t* codes, float* s_x, void* workspace,
                        size_t workspace_bytes, void* stream);

/* Allocation-free cat_transform_quant, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, results and errors as
 * cat_transform_quant without the workspace: its scratch is a fixed array
 * of cat_transform_quant_noalloc_max_bytes() bytes (16 MiB) that the
 * library holds on each device it runs on, from its first use there until
 * the process ends.  The call allocates nothing and calls no allocating
 * routine.  A call whose cat_transform_quant_workspace_bytes(n, d, k)
 * exceeds that size returns CAT_ERR_UNSUPPORTED before touching the device
 * (8192 x 14336 and 16384 x 8192 bf16 inputs fit).  All calls on one GPU
 * share that GPU's array, which keeps the last call's contents; calls that
 * overlap on one GPU (other streams, other threads) race and must not be
 * issued.  The exchange timeout word lives in that array, at the offset
 * a workspace of the call's shape would hold it; a timed-out wait never
 * yields a wrong scale (zero code blocks, NaN scales), and
 * cat_transform_quant_noalloc_status reports it. */
size_t cat_transform_quant_noalloc_max_bytes(void);
int cat_transform_quant_noalloc(const void* X, int x_dtype, int64_t n, int64_t d,
                                const void* T, int t_dtype, int64_t k, int bits,
                                uint8_t* codes, float* s_x, void* stream);
/* cat_transform_quant_status for the current device's array of
 * cat_transform_quant_noalloc: the timeout word of calls of shape (n, d, k)
 * (each shape has its own word in the array; the array starts zeroed).
 * Same returns; CAT_ERR_UNSUPPORTED for a shape the array cannot hold. */
int cat_transform_quant_noalloc_status(int64_t n, int64_t d, int64_t k, void* stream);

/* ------------------------------------------------------------------ (3)
 * W4A4 integer GEMM with dequantization (Sec. 3, eq. 5:
 * Q(W T^-1) Q(T x)).
 *
 *   acc[t, o]     = sum_j qx[t, j] * qw[o, j]          (int32, exact)
 *   y_tilde[t, o] = fl32(fl32(acc) * s_x[t]) * s_w[o]  (fp32, in this order)
 *
 * codes_x  device uint8 [n x d_in/2] packed INT4, s_x device fp32 [n].
 * codes_w  device uint8 [d_out x d_in/2] packed INT4, s_w device fp32 [d_out].
 * n, d_out >= 1; d_in a multiple of 32 and <= CAT_MAX_D_IN.
 * Codes must lie in [-7, 7] (what cat_transform_quant and
 * cat_quantize_weights produce at 4 bits): every int32 sum is then exact
 * for d_in <= CAT_MAX_D_IN.  -8 is not checked; with -8 on both sides the
 * widened sum reaches 256 * 64 * d_in, which is 2^31 at CAT_MAX_D_IN.
 * y_tilde  device fp32 [n x d_out] (written).
 * acc_out  device int32 [n x d_out] or NULL (written when non-NULL).
 */
int cat_w4a4_linear(const uint8_t* codes_x, const float* s_x,
                    const uint8_t* codes_w, const float* s_w, int64_t n,
                    int64_t d_in, int64_t d_out, float* y_tilde,
                    int32_t* acc_out, void* stream);

/* The same product for codes stored one int8 per element: the W6A6 and
 * W8A8 layers the paper compares W4A4 against (Sec. 4 "CAT Block
 * Approximation" and the Fig. 6 caption; Sec. 3, eq. 5 at
 * those widths).  Same formula, arguments and errors as cat_w4a4_linear,
 * except:
 * codes_x  device int8 [n x d_in], s_x device fp32 [n].
 * codes_w  device int8 [d_out x d_in], s_w device fp32 [d_out].
 * Codes must lie in [-127, 127] (what cat_transform_quant and
 * cat_quantize_weights produce at 8 bits or fewer): with d_in <=
 * CAT_MAX_D_IN every int32 sum is then exact.  -128 is not checked. */
int cat_int8_linear(const int8_t* codes_x, const float* s_x,
                    const int8_t* codes_w, const float* s_w, int64_t n,
                    int64_t d_in, int64_t d_out, float* y_tilde,
                    int32_t* acc_out, void* stream);

/* ------------------------------------------------------------------
 * Asymmetric per-token activations (the paper's own set-up, Sec. 6:
 * activations per token, asymmetric; range r = max - min, Sec. 2 after
 * Lemma 2.2), INT4.
 *
 * cat_transform_quant_asym: z as in cat_transform_quant, then per token
 *   zmin = min z, r = fl(max z - zmin),
 *   s_x = fl(r / 15), inv = fl(15 / r)                 (both 0 if r == 0)
 *   q = clamp(rint(fl(fl(z - zmin) * inv)), 0, 15)     (ties to even)
 * so that z ~ s_x q + zmin.  codes hold q - 8 as packed INT4 (the layout
 * above, values in [-8, 7]); zmin_x device fp32 [n] (written).  Other
 * arguments and errors as cat_transform_quant (bits is 4).  The workspace
 * is at least cat_transform_quant_asym_workspace_bytes(n, d, k) bytes
 * (larger than the symmetric one: the single-pass path, bf16 with k = 128
 * and d = 2048, 4096 or 8192, exchanges a row minimum and maximum per
 * token); the exchange timeout word is at cat_transform_quant_flag_offset
 * as for the symmetric path; a timed-out wait never yields a wrong scale
 * (the blocks concerned are coded with a NaN range; where block 0's wait
 * ran out s_x = NaN, and zmin_x is exact or NaN).
 *
 * cat_w4a4_linear_asym: the product of those activations with symmetric
 * INT4 weights,
 *   acc[t, o] = sum_j q[t, j] qw[o, j] (q in [0, 15]; int32, exact)
 *   y_tilde   = fl(fl(fl(acc) s_x[t]) + fl(zmin_x[t] fl(rsum_w[o]))) s_w[o]
 * with rsum_w[o] = sum_j qw[o, j] (device int32 [d_out], from
 * cat_weight_code_sums).  acc_out, when non-NULL, receives acc.  Other
 * arguments and errors as cat_w4a4_linear.
 *
 * cat_weight_code_sums: host; rsum_out[o] = sum of row o's codes of the
 * packed INT4 [d_out x d_in/2] codes_w; d_in even.
 */
size_t cat_transform_quant_asym_workspace_bytes(int64_t n, int64_t d, int64_t k);
int cat_transform_quant_asym(const void* X, int x_dtype, int64_t n, int64_t d,
                             const void* T, int t_dtype, int64_t k,
                             uint8_t* codes, float* s_x, float* zmin_x,
                             void* workspace, size_t workspace_bytes,
                             void* stream);
int cat_w4a4_linear_asym(const uint8_t* codes_x, const float* s_x,
                         const float* zmin_x, const uint8_t* codes_w,
                         const float* s_w, const int32_t* rsum_w, int64_t n,
                         int64_t d_in, int64_t d_out, float* y_tilde,
                         int32_t* acc_out, void* stream);
int cat_weight_code_sums(const uint8_t* codes_w, int64_t d_out, int64_t d_in,
                         int32_t* rsum_out);

/* ------------------------------------------------------------------ (4)
 * SQNR reduction (Sec. 2, eq. 1: E||W x||^2 / E||W x - W~ x~||^2, with
 * the expectations replaced by sums over all tokens and outputs).
 *
 *   out[0] = sum y^2,  out[1] = sum (y - y_tilde)^2     (fp64 sums)
 *   out[2] = 10 log10(out[0] / out[1])   (+inf if out[1] == 0 < out[0];
 *                                          NaN if both are 0)
 *
 * y, y_tilde  device fp32 [count], count >= 1.
 * workspace   device, >= cat_sqnr_workspace_bytes(count) bytes.
 * out         device fp64 [3] (written).
 * The reduction order is fixed: repeated calls give identical bits.
 */
size_t cat_sqnr_workspace_bytes(int64_t count);
int cat_sqnr(const float* y, const float* y_tilde, int64_t count,
             void* workspace, size_t workspace_bytes, double* out,
             void* stream);

/* ------------------------------------------------------------ host side
 * Transform construction (Sec. 4, eq. 7 and eq. 10), on the CPU in fp64.
 *
 * For each block b of size k:
 *   Sigma_w,b = W[:, b]^T W[:, b]
 *   M_b       = (Sigma_w,b # Sigma_x,b^-1)^(1/2)        (if CAT_BUILD_ALIGN,
 *                                                       else I)
 *   T_b       = H_k M_b                                (if CAT_BUILD_HADAMARD,
 *                                                       else M_b)
 *   T_b is rounded to t_dtype; then W'[:, b] = W[:, b] T_b^-1 with the
 *   ROUNDED T_b, so W' T x = W x holds to fp64 accuracy.
 * Symmetric eigenproblems use cyclic Jacobi; eigenvalues below
 * 1e-12 * lambda_max are raised to that floor.
 *
 * sigma_x_blocks  host fp64 [d_in/k x k x k]: the diagonal blocks of
 *                 Sigma_x (already divided by the token count).
 * W               host fp32 [d_out x d_in].
 * k               power of two in [1, CAT_MAX_BLOCK], d_in % k == 0.
 * T_out           host [d_in/k x k x k] in t_dtype (bf16 as uint16 bits).
 * T_exact_out     host fp64 [d_in/k x k x k] before rounding, or NULL.
 * W_prime_out     host fp64 [d_out x d_in], or NULL.
 * n_threads       worker threads (<= 0: hardware concurrency).
 */
int cat_build_transform(const double* sigma_x_blocks, const float* W,
                        int64_t d_out, int64_t d_in, int64_t k, int flags,
                        int t_dtype, void* T_out, double* T_exact_out,
                        double* W_prime_out, int n_threads);

/* Per-output-channel symmetric weight quantization (Sec. 6: weights per
 * channel, symmetric, round to nearest), on fp32(W_prime) with exactly
 * the arithmetic of cat_transform_quant.
 * W_prime host fp64 [d_out x d_in]; s_w_out host fp32 [d_out]; d_in even.
 * bits 4: codes_w_out host uint8 [d_out x d_in/2], packed INT4;
 * bits 6, 8: codes_w_out host int8 [d_out x d_in] (as uint8 storage).
 * Other widths return CAT_ERR_UNSUPPORTED. */
int cat_quantize_weights(const double* W_prime, int64_t d_out, int64_t d_in,
                         int bits, uint8_t* codes_w_out, float* s_w_out);

/* ------------------------------------------------------------------
 * Full-dimension Hadamard (Sec. 4: T = H M with H over all d channels;
 * Sec. 3: Hadamard rotations).  H_d = H_m (x) H_k with m = d / k, so
 *   T = (H_m (x) I_k) / sqrt(m) . blockdiag(T_b),  T_b = H_k M_b / sqrt(k)
 * (the blocks cat_build_transform returns with CAT_BUILD_HADAMARD).  H_m is
 * Sylvester for m a power of two, else H_28 (x) Sylvester_(m/28), H_28 from
 * Paley's second construction with q = 13, rows split r = r1 (m/28) + r2.
 *
 * cat_transform_quant_full: z = blockdiag(T_b) x in fp32, z' =
 *   (H_m (x) I_k) z / sqrt(m) in fp32, then the per-token INT4 quantizer of
 *   cat_transform_quant on z'.  bf16 X and T, k = 128 or 256, m in {2, 4,
 *   8, 16, 32, 64, 28, 56, 112} (else CAT_ERR_UNSUPPORTED).  workspace:
 *   cat_transform_quant_full_workspace_bytes(n, d, k) bytes (z, fp32).
 *   Other arguments and errors as cat_transform_quant.
 * cat_full_hadamard_weights: host; W_full = W' (H_m (x) I_k)^T / sqrt(m)
 *   for W' = W blockdiag(T_b)^-1 (cat_build_transform's W_prime), so that
 *   W_full z' = W x.  fp64 [d_out x d_in] in and out (may not alias).
 */
size_t cat_transform_quant_full_workspace_bytes(int64_t n, int64_t d, int64_t k);
int cat_transform_quant_full(const void* X, int x_dtype, int64_t n, int64_t d,
                             const void* T, int t_dtype, int64_t k,
                             uint8_t* codes, float* s_x, void* workspace,
                             size_t workspace_bytes, void* stream);
int cat_full_hadamard_weights(const double* W_prime, int64_t d_out,
                              int64_t d_in, int64_t k, double* W_full_out);

/* The Theorem 2.4 decomposition of a quantized layer (Sec. 2: Lemmas 2.2,
 * 2.3, Theorem 2.4) from what the device calls produce, host side:
 *   C(x')  = E||x'||^2 / E[r(x')^2], x' = T x, r = 2 max|x'_i| = 2 qmax s_x
 *   C(W')  = sum_o ||w'_o||^2 / sum_o r(w'_o)^2
 *   A      = E||W' x'||^2 / (||W'||_F^2 E||x'||^2), E||W'x'||^2 = sum_y2 / n
 *   SQNR  ~= 12 (N(b_x)^2 C(x') || N(b_w)^2 C(W')) A,  N(b) = 2 qmax
 * with E||x'||^2 = (1/n) sum_b tr(T_b S_b T_b^T).
 * s_x              host fp32 [n]: cat_transform_quant's scales at bits_x.
 * sigma_sum_blocks host fp64 [d_in/k x k x k]: block sums X_b^T X_b over the
 *                  same n tokens (cat_cov_accumulate, BLOCK_DIAG, not
 *                  divided by n).
 * T                host [d_in/k x k x k] in t_dtype (bf16 as uint16 bits).
 * W_prime          host fp64 [d_out x d_in].
 * sum_y2           sum of y^2 over the batch (cat_sqnr's out[0]).
 * out              host fp64 [5]: C(x'), C(W'), A, predicted SQNR, in dB.
 * bits_x, bits_w in [2, 8]. */
int cat_sqnr_terms(const float* s_x, int64_t n, int bits_x,
                   const double* sigma_sum_blocks, int64_t d_in, int64_t k,
                   const void* T, int t_dtype, const double* W_prime,
                   int64_t d_out, int bits_w, double sum_y2, double* out);

/* Thread-local message describing the last non-OK return on this thread. */
const char* cat_last_error(void);

/* Library version string. */
const char* cat_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CAT_H */
