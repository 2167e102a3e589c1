/*
 * orbitquant.h -- C ABI of the OrbitQuant quantized-linear hot path on MI355X (gfx950).
 *
 * OrbitQuant (arXiv 2607.02461) quantizes a linear layer y = W x (Sec. 3.1, Eq. (1)) of a
 * diffusion transformer without calibration data.  Weights and activations are rotated by
 * the same randomized permuted block-Hadamard (RPBH) transform Pi_d (Sec. 4.4, Eq. (9)),
 * split into a norm and a unit direction, and the direction is encoded coordinate-wise
 * against one fixed Lloyd-Max codebook per (input dimension d, bit-width b) fitted to the
 * rotated-coordinate marginal f_d (Sec. 3.2, Eqs. (2)-(3)).  The rotation cancels inside
 * the product (Sec. 4.3), so the layer contracts the two code sets directly.
 *
 * Conventions shared by every call
 *   - Every function returns orbit_status; 0 is success.  Nothing throws across the ABI.
 *     On failure orbit_last_error() returns a message for the calling thread, valid until
 *     that thread's next call into the library.
 *   - BF16 values are passed as uint16_t bit patterns; fp32 as float.
 *   - Matrices are row-major with the reduction dimension K contiguous.
 *   - Packed codes: an LSB-first bit stream per row; the code of coordinate k occupies bits
 *     [k*b, k*b + b) of the row, so a row of K codes is K*b/8 bytes and rows are contiguous.
 *     A code is stored as the sign-magnitude label of its level: with levels ascending and
 *     antisymmetric (index c and 2^b - 1 - c are negatives of each other), level index
 *     c >= 2^(b-1) (a positive level) is stored as c - 2^(b-1) and index c < 2^(b-1) as
 *     2^b - 1 - c.  The label's top bit is the level's sign and its low b-1 bits rank the
 *     level's magnitude (0 = nearest zero); the labels are a storage format and change no
 *     nearest-level decision (Eq. (3)).
 *   - Device calls take device pointers the caller owns (e.g. torch tensors), only enqueue
 *     work on `stream` (a hipStream_t; NULL = the null stream) and return before it runs.
 *     They allocate no device memory for their operands.  Argument checks are synchronous
 *     and happen before any launch; a launch failure returns ORBIT_EHIP with HIP's message.
 *   - Handles are immutable after creation and may be used from several threads and streams
 *     at once.  A plan's permutation/sign tables (6 bytes per input) and a codebook's encoder
 *     table (at most 32 KB) live on each device that uses them.  They are copied there at set-up
 *     (hipMalloc + a synchronous copy): when the handle is created, to the device current on the
 *     creating thread if a HIP device is visible, and on other devices by rpbh_plan_upload /
 *     lloydmax_codebook_upload.  Device calls never allocate or copy: on a device without the
 *     handle's tables they return ORBIT_EINVAL.  So every device call, the first included, records
 *     only kernel launches and can be captured in a HIP graph and replayed.  The tables stay until
 *     the handle is destroyed; destroy a handle only after the work that uses it has finished.
 */
#ifndef ORBITQUANT_H
#define ORBITQUANT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ORBIT_OK = 0,
    ORBIT_EINVAL = 1,        /* an argument is invalid (null, out of range, inconsistent)     */
    ORBIT_EUNSUPPORTED = 2,  /* valid for the method, but outside what the kernels implement  */
    ORBIT_ENOMEM = 3,        /* host or device allocation failed                              */
    ORBIT_EHIP = 4,          /* a HIP runtime call or kernel launch failed                    */
    ORBIT_EINTERNAL = 5      /* a numerical routine failed to converge or a bug was detected  */
} orbit_status;

/* Message describing the calling thread's last failure ("" after a success). */
const char* orbit_last_error(void);

/* Library version string, e.g. "orbitquant-mi355x 0.1.0 gfx950". */
const char* orbit_version(void);

typedef struct orbit_plan_s* orbit_plan;
typedef struct orbit_codebook_s* orbit_codebook;

/* ------------------------------------------------------------------ host, offline stage */

/*
 * rpbh_plan -- draw the RPBH rotation Pi_d = blkdiag(H_h D_1, ..., H_h D_{d/h}) P_pi
 * (Sec. 4.4, Eq. (9); Alg. 1, offline stage), drawn on the host.
 *
 *   d     input dimension, >= 1
 *   h     Hadamard block size: a power of two dividing d; 0 selects the paper's rule,
 *         the largest power of two dividing d (Sec. 4.4).  The device kernels implement
 *         128 <= h <= 4096 (the rule gives 1024 for d = 3072 and 5120, 4096 for 12288 and
 *         512 for 13824); other sizes are valid plans for the host API only
 *   seed  generator seed.  pi and the signs are drawn from SplitMix64 (Steele, Lea &
 *         Flood 2014) started at state = seed: Fisher-Yates from the identity for
 *         j = d-1 .. 1 with k uniform in [0, j] (draw u until u >= 2^64 mod (j+1), take
 *         u mod (j+1)); then sign[j] = -1 when the top bit of the next output is 1.
 *   out   receives the new handle
 *
 * Conventions: (P_pi x)_j = x[perm[j]] (a gather) and sign[j] multiplies the j-th
 * post-permutation coordinate; H_h is the Sylvester-ordered Walsh-Hadamard matrix scaled
 * by 1/sqrt(h), so Pi_d is orthogonal.  With a HIP device visible, the plan's device tables are
 * copied to the current device before the call returns (see rpbh_plan_upload); without one the
 * plan is host-only.  Errors: ORBIT_EINVAL for d < 1, a bad h or a null `out`; ORBIT_ENOMEM;
 * ORBIT_EHIP when the copy to the device fails.
 */
orbit_status rpbh_plan(int64_t d, int32_t h, uint64_t seed, orbit_plan* out);

/*
 * rpbh_plan_from_arrays -- the same handle built from a caller-supplied permutation and
 * sign vector (host arrays, copied).  perm must be a permutation of 0..d-1, sign entries
 * must be +1 or -1.  Set-up and errors otherwise as for rpbh_plan; ORBIT_EINVAL for a bad
 * perm or sign.
 */
orbit_status rpbh_plan_from_arrays(int64_t d, int32_t h, const int32_t* perm, const int8_t* sign,
                                   orbit_plan* out);

/*
 * rpbh_plan_upload -- copy the plan's device tables (gather offsets with the signs folded in, and
 * the sign masks of the identity-permutation path: 6 bytes per input) to the current device, for
 * the device calls made there.  Creation already did this for the device current at the time;
 * another device needs this call once, before its first device call and outside stream capture
 * (it allocates and copies synchronously).  Repeated calls on a device return ORBIT_OK at once.
 * Errors: ORBIT_EINVAL (null plan); ORBIT_ENOMEM; ORBIT_EHIP (no device, or a failed copy).
 */
orbit_status rpbh_plan_upload(orbit_plan p);

/* Read back a plan.  Any output pointer may be NULL; perm and sign receive d entries. */
orbit_status rpbh_plan_get(orbit_plan p, int64_t* d, int32_t* h, int32_t* perm, int8_t* sign);

/* Free a plan (host arrays and every per-device copy).  NULL is ignored. */
void rpbh_plan_destroy(orbit_plan p);

/*
 * lloydmax_codebook -- the Lloyd-Max codebook C^(d,b) for the marginal
 * f_d(t) = Gamma(d/2) / (sqrt(pi) Gamma((d-1)/2)) (1 - t^2)^((d-3)/2) on [-1, 1]
 * (Sec. 3.2, Eqs. (2)-(3); Sec. 4.5; Alg. 1, offline stage), computed on the host.
 *
 *   bits  1..6 for the codebook itself; the quantizer accepts 2, 3, 4 and 6, the GEMM 2, 3, 4
 *         and 6 for activations and 2..4 for weights
 *   d     input dimension, >= 3
 *
 * Computed in fp64 by the fixed-point iteration of the midpoint and centroid conditions on
 * the exact f_d (not its Gaussian approximation).  The levels are exactly antisymmetric
 * and the thresholds are the midpoints of neighbouring levels, so the middle threshold is
 * exactly 0.  With a HIP device visible, the encoder table is copied to the current device
 * before the call returns (see lloydmax_codebook_upload).  Errors: ORBIT_EINVAL for bits or d
 * out of range; ORBIT_EINTERNAL if the iteration fails to converge; ORBIT_ENOMEM, ORBIT_EHIP
 * when the copy to the device fails.
 */
orbit_status lloydmax_codebook(int32_t bits, int64_t d, orbit_codebook* out);

/*
 * Read back a codebook: levels (2^b, ascending), thresholds (2^b - 1), and the bf16 image of
 * the levels that the GEMM decodes to (2^b bfloat16 bit patterns, the fp64 levels rounded once
 * to nearest, ties to even).  The paper dequantizes codes to BF16 and multiplies in BF16 (its
 * efficiency measurements and limitations section); the GEMM does the same with fp32
 * accumulation.  Any output pointer may be NULL.
 */
orbit_status lloydmax_codebook_get(orbit_codebook c, int32_t* bits, int64_t* d, double* levels,
                                   double* thresholds, uint16_t* lut_bf16);

/*
 * lloydmax_codebook_upload -- copy the codebook's encoder table (the quantizer's nearest-level
 * lookup, at most 8192 fp32 entries) to the current device; as rpbh_plan_upload.
 */
orbit_status lloydmax_codebook_upload(orbit_codebook c);

/* Free a codebook.  NULL is ignored. */
void lloydmax_codebook_destroy(orbit_codebook c);

/* ------------------------------------------------------------------ device, per call */

/*
 * quantize_weights_offline -- rotate, normalize and encode weight rows
 * (Sec. 4.2, Eqs. (4)-(6); Alg. 1, offline stage):
 *     w'_i = Pi_d w_i,  r'_i = ||w'_i||_2,  code_i = Q_{b_w}(w'_i / (r'_i + eps)),
 * with r' stored as BF16 (round-to-nearest-even of the fp32 norm).  The codes use the
 * fp32 norm; only the stored magnitude is rounded.
 *
 *   p       plan with plan.d == K
 *   cb_w    codebook with cb.d == K and cb.bits = b_w in {2, 3, 4, 6} (the GEMM takes 2..4)
 *   W       device, bf16 [N][ldw]; row i is w_i (the layout of nn.Linear.weight)
 *   N, K    rows and input dimension; N >= 0
 *   ldw     row stride of W in elements, >= K and a multiple of 8
 *   eps     guard added to the norm before dividing (1e-10 in the paper; a zero row gives
 *           r' = 0 and the middle code 2^(b-1) everywhere).  Finite and >= 0; the kernel
 *           floors r' + eps at 1e-30, which only matters for eps below that and rows whose
 *           norm is smaller still
 *   w_codes device, uint8 [N][K*b_w/8], packed as described above
 *   w_norm  device, bf16 [N]
 *   stream  hipStream_t
 *
 * Pointers: W and w_codes 16-byte aligned, w_norm 2-byte aligned.
 * Errors: ORBIT_EINVAL (null pointer, K mismatch, ldw, alignment, a plan or codebook without
 * tables on the current device); ORBIT_EUNSUPPORTED
 * (h outside 128..4096, K > 16384, bits not in {2, 3, 4, 6}, more than 2^31 - 1 rows, a row
 * stride ldw - K of 2^23 elements or more);
 * ORBIT_EHIP.  N = 0 returns at once.  Packing as above: at b = 6 every 4 codes fill 3 bytes.
 */
orbit_status quantize_weights_offline(orbit_plan p, orbit_codebook cb_w, const uint16_t* W, int64_t N,
                                      int64_t K, int64_t ldw, float eps, uint8_t* w_codes,
                                      uint16_t* w_norm, void* stream);

/*
 * rpbh_quantize_act -- online activation quantization, one fused kernel
 * (Sec. 4.3, Eqs. (7)-(8); Alg. 1, online stage):
 *     x'_n = Pi_d x_n,  s_n = ||x'_n||_2,  code_n = Q_{b_a}(x'_n / (s_n + eps)).
 *
 *   X       device, bf16 [M][ldx], tokens as rows
 *   M, K    tokens and input dimension; M >= 0
 *   ldx     row stride of X in elements, >= K and a multiple of 8
 *   eps     as above (1e-10 in the paper)
 *   x_codes device, uint8 [M][K*b_a/8]
 *   x_norm  device, fp32 [M]: s_n (the dequantized row is s_n * L_a[code_n])
 *
 * Pointers: X and x_codes 16-byte aligned, x_norm 4-byte aligned.
 * Errors and limits as for quantize_weights_offline.  M = 0 returns at once.  A row holding Inf
 * or NaN gets a non-finite norm and unspecified codes (both entry points); other rows are
 * unaffected.
 */
orbit_status rpbh_quantize_act(orbit_plan p, orbit_codebook cb_a, const uint16_t* X, int64_t M, int64_t K,
                               int64_t ldx, float eps, uint8_t* x_codes, float* x_norm, void* stream);

/*
 * orbit_qlinear -- the quantized layer on codes (Sec. 4.3: W'x' = W Pi^T Pi x = W x; the
 * codebook GEMM named as future work in the paper's limitations):
 *     Y[n][i] = x_norm[n] * w_norm[i] * sum_k L_a[x_code[n][k]] * L_w[w_code[i][k]],
 * where L_a, L_w are the bf16 images of the two codebooks' levels (codes dequantized to BF16
 * and multiplied in BF16, as the paper computes its layers).  Products are exact in fp32 and
 * accumulate in fp32 on the matrix cores.
 *
 *   cb_a, x_codes, x_norm   activation codebook (bits b_a) and the outputs of
 *                           rpbh_quantize_act for M rows
 *   cb_w, w_codes, w_norm   weight codebook (bits b_w) and the outputs of
 *                           quantize_weights_offline for N rows
 *   K                       input dimension; cb_a.d == cb_w.d == K, K a multiple of 64
 *   Y                       device, fp32 [M][ldy], ldy >= N
 *
 * Pointers: codes 16-byte aligned, x_norm 4-byte, w_norm 2-byte, Y 4-byte aligned (Y 16-byte
 * aligned with ldy % 4 == 0 and w_norm 8-byte aligned enable vector stores; other layouts are
 * handled element-wise).  The 4-bit decoder relies on the codebook's exact antisymmetry in
 * bf16 (L[15-c] = -L[c]), which lloydmax_codebook guarantees; ORBIT_EINTERNAL otherwise.
 * Errors: ORBIT_EINVAL (null pointer, dimension mismatch, ldy < N); ORBIT_EUNSUPPORTED
 * (activation bits not in {2, 3, 4, 6}, weight bits outside 2..4, K not a multiple of 64,
 * M or N above 2^31 - 1 or more than 2^27 output tiles of 256 x 256); ORBIT_EHIP.  M = 0 or
 * N = 0 returns at once.
 */
orbit_status orbit_qlinear(orbit_codebook cb_a, const uint8_t* x_codes, const float* x_norm, int64_t M,
                           orbit_codebook cb_w, const uint8_t* w_codes, const uint16_t* w_norm, int64_t N,
                           int64_t K, float* Y, int64_t ldy, void* stream);

/*
 * orbit_qlinear_ex -- orbit_qlinear with the rest of the layer fused into its epilogue, so the
 * output can feed the next layer's quantizer directly (the low-bit layer consumed natively, as
 * the paper's Limitations and Future Work section asks; the DiT MLP's two projections with the
 * GELU between them, Sec. 5's models):
 *     Y[n][i] = act(x_norm[n] * w_norm[i] * sum_k L_a[...] * L_w[...] + bias[i])
 *
 *   bias       device, bf16 [N], or NULL for none (Eq. (1) itself has no bias)
 *   act        ORBIT_ACT_NONE, or ORBIT_ACT_GELU: x * Phi(x), Phi the standard normal CDF from
 *              erfc to a fractional error below 1.2e-7 (Numerical Recipes' Chebyshev-fitted form)
 *   out_dtype  ORBIT_OUT_F32, or ORBIT_OUT_BF16 (round to nearest even), the input type of
 *              rpbh_quantize_act
 *   Y          device, [M][ldy] elements of out_dtype
 *   other arguments, limits and errors as for orbit_qlinear; ORBIT_EINVAL also for an unknown
 *   act or out_dtype, and Y must be aligned to its element size (bias to 2 bytes).
 * With bias = NULL, act = ORBIT_ACT_NONE and out_dtype = ORBIT_OUT_F32 this is orbit_qlinear.
 */
enum { ORBIT_ACT_NONE = 0, ORBIT_ACT_GELU = 1 };
enum { ORBIT_OUT_F32 = 0, ORBIT_OUT_BF16 = 1 };
orbit_status orbit_qlinear_ex(orbit_codebook cb_a, const uint8_t* x_codes, const float* x_norm, int64_t M,
                              orbit_codebook cb_w, const uint8_t* w_codes, const uint16_t* w_norm, int64_t N,
                              int64_t K, const uint16_t* bias, int32_t act, int32_t out_dtype, void* Y,
                              int64_t ldy, void* stream);

/*
 * orbit_qlinear_workspace_size -- bytes of device workspace with which orbit_qlinear_ws splits
 * the contraction over K for a layer of M x N outputs and K inputs on the current device; 0 when
 * it would not split.  A split pays where the grid of output tiles is too small to fill the
 * device: a layer of few tokens, or the rows of a large layer's last, partly filled round of
 * tiles.  Each split contracts a contiguous range of K, so every compute unit stays busy.
 *
 *   bytes  host, out: splits * (rows split) * N * 4 (fp32 partial sums), or 0
 *
 * Errors: ORBIT_EINVAL (null bytes, negative M or N, K not a positive multiple of 64 up to
 * 2^30); ORBIT_EHIP (no device).  M = 0 or N = 0 gives 0.
 */
orbit_status orbit_qlinear_workspace_size(int64_t M, int64_t N, int64_t K, size_t* bytes);

/*
 * orbit_qlinear_schedule -- how the layer kernels run an M x N x K layer on the current device:
 * output rows [0, rows_large) on the 256 x 256-tile kernel, rows [rows_large, M) on the
 * 128 x 128-tile kernel, the latter split over K into `splits` contiguous ranges (1 = unsplit)
 * when orbit_qlinear_ws has a workspace of orbit_qlinear_workspace_size(M, N, K) bytes.  For
 * profiling and for callers that time or place the two parts themselves; the layer calls make the
 * same choice internally.
 *   rows_large, splits  host, out
 * Errors: ORBIT_EINVAL (null outputs, negative M or N, K not a positive multiple of 64 up to
 * 2^30); ORBIT_EHIP (no device).  M = 0 or N = 0 gives 0 and 1.
 */
orbit_status orbit_qlinear_schedule(int64_t M, int64_t N, int64_t K, int64_t* rows_large, int32_t* splits);

/*
 * orbit_qlinear_ws -- orbit_qlinear_ex with a caller-owned device workspace.  With
 * workspace_bytes at least orbit_qlinear_workspace_size(M, N, K) on the same device (and the
 * workspace 16-byte aligned) the rows of a small grid run split over K: the splits' fp32 sums
 * are added in split order (deterministic for a given device) before the epilogue, so the result
 * differs from orbit_qlinear_ex's only in the fp32 rounding of the sum over K.  Otherwise (a
 * NULL or too small workspace, or a layer that does not split) it is orbit_qlinear_ex.  The
 * workspace's contents on entry do not matter.  The library does not keep the pointer; the
 * caller keeps the workspace alive and unused by other work until the call's work on `stream`
 * has finished, and gives concurrent calls separate workspaces.
 *   workspace        device, or NULL
 *   workspace_bytes  its size in bytes
 *   other arguments, limits and errors as for orbit_qlinear_ex.
 */
orbit_status orbit_qlinear_ws(orbit_codebook cb_a, const uint8_t* x_codes, const float* x_norm, int64_t M,
                              orbit_codebook cb_w, const uint8_t* w_codes, const uint16_t* w_norm, int64_t N,
                              int64_t K, const uint16_t* bias, int32_t act, int32_t out_dtype, void* Y,
                              int64_t ldy, void* workspace, size_t workspace_bytes, void* stream);

/*
 * orbit_qlinear_noalloc -- orbit_qlinear_ws for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the same layer,
 * split over K exactly as orbit_qlinear_ws splits it with a large enough workspace (so the same
 * bits), with the partial sums in a scratch array the library holds in device memory instead of a
 * caller workspace.  The call allocates nothing and calls no allocating routine.
 *   Limit: the scratch array is 32 MiB (33554432 bytes) per device, held by every device the
 *   library runs on until the process ends.  A layer whose split needs more
 *   (orbit_qlinear_workspace_size(M, N, K) > 32 MiB) returns ORBIT_EUNSUPPORTED; layers that do not
 *   split need none.
 *   Sharing: all calls on one device share its scratch array.  Calls that overlap in time on one
 *   device (on several streams, or from several threads without ordering) race on it and give
 *   undefined results; serialize them, e.g. on one stream.  The array keeps the last call's
 *   contents; nothing in it has to start at zero (every partial sum is written before it is read).
 *   Arguments, other limits and errors as for orbit_qlinear_ex.
 */
orbit_status orbit_qlinear_noalloc(orbit_codebook cb_a, const uint8_t* x_codes, const float* x_norm, int64_t M,
                                   orbit_codebook cb_w, const uint8_t* w_codes, const uint16_t* w_norm, int64_t N,
                                   int64_t K, const uint16_t* bias, int32_t act, int32_t out_dtype, void* Y,
                                   int64_t ldy, void* stream);

/*
 * adaln_int4_quantize_weights -- the offline pass of the adjacent layer type: the adaptive-layer-
 * norm modulation projections, which the paper keeps at INT4 weight round-to-nearest with group
 * size 64 and BF16 activations, unrotated (Sec. 5 setup; supplementary layer list; Sec. 6.2
 * ablates the bit-width).  Symmetric per group of 64 consecutive inputs:
 *     scale = fp16(min(absmax / 7, 65504)),  q = clamp(RNE(w / scale), -8, 7)
 * with both quotients formed in fp32 (IEEE, round to nearest even); a group whose scale is 0
 * has codes 0.
 *
 *   W       device, bf16 [N][ldw], the projection's weight rows
 *   N, K    rows and inputs; K a positive multiple of 64
 *   ldw     row stride of W in elements, >= K and a multiple of 8
 *   q       device, uint8 [N][K/2]: q + 8 (offset binary) per nibble, element 2j in the low
 *           nibble of byte j
 *   scales  device, fp16 [N][K/64]
 *   stream  hipStream_t
 *
 * Pointers: W and q 16-byte aligned, scales 2-byte aligned.  Errors: ORBIT_EINVAL (null pointer,
 * K, ldw, alignment); ORBIT_EUNSUPPORTED (N above 2^31 - 1 or K above 2^30); ORBIT_EHIP.
 * N = 0 returns at once.
 */
orbit_status adaln_int4_quantize_weights(const uint16_t* W, int64_t N, int64_t K, int64_t ldw, uint8_t* q,
                                         uint16_t* scales, void* stream);

/*
 * adaln_int4_linear -- the AdaLN modulation projection on its INT4 weights:
 *     Y[m][n] = sum_k X[m][k] * q[n][k] * scale[n][k/64] (+ bias[n])
 * Products of the BF16 activations with the codes are exact in fp32; each group's partial sum
 * accumulates in fp32 and is scaled before it joins the row total.  Built for the layer's shape:
 * a few conditioning tokens (M small) against many output rows, so it streams the weights once
 * and is bound by HBM.
 *
 *   X       device, bf16 [M][ldx]; ldx >= K and a multiple of 8; K <= 16384 (the tokens are
 *           staged in LDS)
 *   M       tokens; 0 <= M <= 131070 (rows are processed two at a time per weight pass)
 *   q, scales, N, K   as produced by adaln_int4_quantize_weights
 *   bias    device, bf16 [N], or NULL
 *   Y       device, fp32 [M][ldy], ldy >= N
 *   stream  hipStream_t
 *
 * Pointers: X and q 16-byte aligned; scales, bias 2-byte and Y 4-byte aligned.  Errors:
 * ORBIT_EINVAL (null pointer, K, strides, alignment); ORBIT_EUNSUPPORTED (sizes above the
 * limits); ORBIT_EHIP.  M = 0 or N = 0 returns at once.
 */
orbit_status adaln_int4_linear(const uint16_t* X, int64_t M, int64_t ldx, const uint8_t* q, const uint16_t* scales,
                               int64_t N, int64_t K, const uint16_t* bias, float* Y, int64_t ldy, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ORBITQUANT_H */
