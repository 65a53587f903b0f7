/*
 * kroquant.h -- C ABI of libkroquant.so, the MI355X (gfx950) online activation
 * quantizer of "KroQuant: Kronecker-Structured Block Transforms for Efficient
 * Post-Training Quantization of Diffusion Transformers".
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Matrices are row-major and contiguous (leading dimension = number of
 *    columns).  bf16 values are passed as their 16-bit patterns (uint16_t).
 *  - d (columns) must be a positive multiple of 32: the quantizer works on
 *    row-wise blocks of 32 elements (Sec. 3.1) and T is block-diagonal with
 *    one 32x32 block per 32-column group (Sec. 3.1 "Goal").  Any M >= 0 is
 *    accepted; M = 0 returns KQ_SUCCESS without touching the GPU.
 *  - MXFP4 output layout, for an input of M rows:
 *      codes  [M, d/2]  uint8: E2M1 codes (bit 3 = sign, bits 0-2 = index of
 *                       the magnitude 0, .5, 1, 1.5, 2, 3, 4, 6), element 2i
 *                       of a row in the low nibble of byte i, 2i+1 in the high;
 *      scales [M, d/32] uint8: E8M0 byte s of block j, scale 2^(s - 127),
 *                       s = max(floor(log2 amax) - 2 + 127, 0), 0 for an all-zero block.
 *    Element values round to the nearest E2M1 magnitude of |y| / 2^(s-127),
 *    ties to even, saturating at 6; a negative value that rounds to 0 keeps
 *    its sign (code 8).  (OCP Microscaling v1.0 MXFP4, the format of Sec. 3.1.)
 *  - Device pointers are plain HIP device (or managed) addresses; the caller
 *    owns every buffer.  The quantize calls never allocate, free or
 *    synchronize; they enqueue one kernel on `stream` (a hipStream_t; NULL =
 *    the null stream) and return.  A fault inside the kernel surfaces at the
 *    caller's next synchronization, as for any HIP launch.
 *  - Alignment: X, codes and y_out must be 16-byte aligned (every lane moves
 *    16 contiguous bytes per access; a row of codes is d/2 bytes, a multiple
 *    of 16, so an aligned base keeps every row aligned); scales need no
 *    alignment; the factors need 4 B and the SmoothQuant multipliers 16 B.
 *  - Inputs must be finite; NaN or Inf inputs give unspecified codes.
 *  - Size: the matrix-core calls (kq_quantize, kq_quantize_packed,
 *    kq_quantize_lu) launch one workgroup per 64 blocks (shared factors) or
 *    per 64 rows x 8 column blocks (per-block factors) and return
 *    KQ_ERROR_UNSUPPORTED when that count exceeds 2^31 - 1 (beyond 2^42
 *    elements of X, far more than one GPU holds).
 *  - Arguments are validated before any HIP call.  On failure the call
 *    returns the status and kq_last_error_detail() describes the argument
 *    (thread-local).  HIP launch/runtime errors return KQ_ERROR_HIP with the
 *    HIP error string in the detail.  No C++ exception crosses this ABI.
 */
#ifndef KROQUANT_H
#define KROQUANT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum kq_status {
    KQ_SUCCESS = 0,
    KQ_ERROR_INVALID_VALUE = 1, /* a size or count is out of range            */
    KQ_ERROR_NULL_POINTER = 2,  /* a required pointer is NULL                 */
    KQ_ERROR_MISALIGNED = 3,    /* a pointer breaks the alignment rule above  */
    KQ_ERROR_UNSUPPORTED = 4,   /* (a, b) split or factor count not supported */
    KQ_ERROR_SINGULAR = 5,      /* a factor is singular or ill-conditioned    */
    KQ_ERROR_HIP = 6            /* the HIP runtime reported an error          */
} kq_status;

/*
 * kq_quantize -- the KroQuant online quantizer (Sec. 3.2 transform, Sec. 3.5
 * kernels, Sec. 3.1 quantizer).  For every row r and 32-column block j of X:
 *     y = (A_f (x) B_f) x,   x = X[r, 32j : 32j+32] widened to fp32,
 * i.e. with the block reshaped row-major to a x b (Xm[p][q] = x[p*b+q]),
 * Ym = A_f . Xm . B_f^T = (A (x) B) vec(Xm^T) = vec(B Xm^T A^T); then MXFP4
 * of y into codes[r, 16j:16j+16] and scales[r, j].
 *
 *   X       device, bf16 [M, d]
 *   A       device, fp32 [nfac, a, a] row-major; B device, fp32 [nfac, b, b]
 *   (a, b)  one of (4, 8), (2, 16), (8, 4), (1, 32)
 *   nfac    1 (one pair for every block) or d/32 (pair f = j for block j:
 *           T = diag(K^(1), ..., K^(d/32)), Sec. 3.1); d/32 needs d < 2^25
 *           (KQ_ERROR_UNSUPPORTED otherwise; the same holds for every call
 *           that takes per-block factors)
 *   codes   device, uint8 [M, d/2];  scales device, uint8 [M, d/32]
 *   y_out   device, fp32 [M, d] or NULL: the transformed values that were
 *           quantized
 *
 * Arithmetic: the 32x32 block K = A (x) B is materialised in fp32 and applied
 * on the matrix cores as a three-term bf16 split with fp32 accumulation
 * (the single 32x32 GEMM per block of Sec. 3.5).  Results agree with the
 * fixed-order evaluation of kq_quantize_exact as follows: E8M0 scales are
 * identical (blocks whose amax lies within the rounding margin of a power of
 * two are re-evaluated in that order); codes differ only by one magnitude
 * step where a value sits on a rounding tie; y_out differs by at most
 * 116 * 2^-24 * sum_k |K_nk| |x_k| per element.
 * To apply the paper's right-multiplication A -> A T with K = G1 (x) ... (x) G5
 * (eq. (1), Sec. 3.2), pass A (x) B = K^T; kq_lu_to_factors builds exactly that.
 */
kq_status kq_quantize(const uint16_t* X, int64_t M, int64_t d, const float* A, const float* B,
                      int a, int b, int64_t nfac, uint8_t* codes, uint8_t* scales, float* y_out,
                      void* stream);

/* Bytes of packed K per factor pair (see kq_pack_factors). */
#define KQ_PACK_BYTES_PER_FACTOR 6160

/*
 * kq_pack_factors -- offline, once per layer: materialise every 32x32 block
 * K_f = A_f (x) B_f in fp32, split it into the three bf16 terms the matrix
 * cores multiply, and store them with ||K_f||_inf in `kpack` (device,
 * nfac * KQ_PACK_BYTES_PER_FACTOR bytes, 16-byte aligned).  This is the
 * "precomputed dense" kernel variant K1 of Sec. 3.5, which keeps the dense
 * blocks in HBM; kq_quantize instead rebuilds K from the factors on the fly
 * in every wave (variant K2).  A, B device fp32 as for kq_quantize.  Enqueued
 * on `stream`; no allocation, no synchronization.
 */
kq_status kq_pack_factors(const float* A, const float* B, int a, int b, int64_t nfac, void* kpack,
                          void* stream);

/*
 * kq_quantize_packed -- kq_quantize reading K from `kpack` (filled by
 * kq_pack_factors from the same A, B, a, b, nfac) instead of rebuilding it.
 * A and B are still required: blocks on a binade edge are re-evaluated in
 * the fixed order of kq_quantize_exact.  Same result contract as kq_quantize
 * (identical scales, codes within tie flips, y within the stated bound); the
 * edge window is 2^-17 cond_inf(A (x) B) amax here, taken from the pack,
 * instead of a per-block bound, so the set of re-evaluated blocks can differ.
 * With per-block factors (nfac = d/32) only the 16-byte window header of
 * each pair's pack is read: every pair's K is rebuilt on chip from its 320
 * bytes of A and B, which costs less than reading its 6160-byte pack, and
 * gives the K terms the pack holds, so the result equals this call's with
 * the same pair repeated in a single-pair pack (nfac = 1), y included.
 */
kq_status kq_quantize_packed(const uint16_t* X, int64_t M, int64_t d, const float* A,
                             const float* B, int a, int b, int64_t nfac, const void* kpack,
                             uint8_t* codes, uint8_t* scales, float* y_out, void* stream);

/*
 * kq_quantize_lu -- kq_quantize with the factors given in the paper's K2 form
 * (Sec. 3.5 "K2", parametrization of Sec. 3.2): 15 scalars per factor pair,
 * lu[f][k] = (a_k, b_k, c_k), k = 0..4, for G_{k+1} = L U with
 * L = [[1, 0], [c, 1]], U = [[a, b], [0, -1/a]].  The block applied is the
 * paper's K = G_1 (x) ... (x) G_5 acting on row activations from the right
 * (x^T K, eq. (1)), i.e. y = K^T x = (A (x) B) x with
 * A = G_1^T (x) ... (x) G_log2(a)^T and B = G_{log2(a)+1}^T (x) ... (x) G_5^T.
 * Every wave decodes its A and B from the 15 parameters on chip, in a fixed
 * fp32 order:
 *     g10 = c*a, g11 = fma(c, b, -(1/a)), and each entry of A and B is the
 *     product of its G entries, left to right.
 * The result then has the same contract as kq_quantize with those A and B.
 *   lu       device fp32 [nfac, 5, 3], 4-byte aligned; every a_k nonzero.
 *   a        1, 2, 4 or 8: how many G factors form A (log2 a); b = 32 / a.
 *   nfac     1 (shared) or d / 32 (one parameter set per column block).
 *   y16_out  optional device bf16 [M, d], 16-byte aligned.  It receives the
 *            transformed values the codes were computed from, rounded to
 *            bf16 (nearest even): the 16-bit activation of the low-rank
 *            branch (Sec. 3.4, LoRaQ).
 * Errors as kq_quantize; a not in {1, 2, 4, 8} -> KQ_ERROR_UNSUPPORTED.
 */
kq_status kq_quantize_lu(const uint16_t* X, int64_t M, int64_t d, const float* lu, int a, int64_t nfac,
                         uint8_t* codes, uint8_t* scales, float* y_out, uint16_t* y16_out, void* stream);

/*
 * kq_quantize_exact -- kq_quantize with the transform evaluated on the vector/*
 * kq_quantize_exact -- kq_quantize with the transform evaluated on the vector
 * ALUs in one fixed fp32 order, so that every output is a deterministic
 * function of that order:
 *     Z[p][i] = B[i][0]*Xm[p][0],  Z[p][i] = fma(B[i][q], Xm[p][q], Z[p][i]) for q = 1..b-1,
 *     Y[o][i] = A[o][0]*Z[0][i],   Y[o][i] = fma(A[o][p], Z[p][i], Y[o][i])  for p = 1..a-1.
 * Same arguments, layout and errors as kq_quantize; slower (12 FMAs per
 * element for (4, 8)).
 */
kq_status kq_quantize_exact(const uint16_t* X, int64_t M, int64_t d, const float* A,
                            const float* B, int a, int b, int64_t nfac, uint8_t* codes,
                            uint8_t* scales, float* y_out, void* stream);

/*
 * kq_smoothquant_quantize -- SmoothQuant comparator (per-channel scaling, the
 * "Scale" kernel of Sec. 4.4; smoothing vector of Appendix D): y_c = x_c *
 * mult_c, one fp32 multiply, then MXFP4 as above.  mult is device fp32 [d]
 * holding the multipliers 1/s_c (the activation is divided by the smoothing
 * factor s_c).
 */
kq_status kq_smoothquant_quantize(const uint16_t* X, int64_t M, int64_t d, const float* mult,
                                  uint8_t* codes, uint8_t* scales, float* y_out, void* stream);

/*
 * kq_hadamard32_quantize -- fixed block Hadamard comparator (Sec. 1; the
 * Hadamard initialization of Sec. 3.2 and the ablation of Sec. 4.3):
 * y = H32 x / sqrt(32) per block, H32 the Sylvester matrix, computed in fp32
 * by add/subtract butterflies with strides 1, 2, 4, 8, 16 and one final
 * multiply by fp32(1/sqrt(32)); then MXFP4.
 */
kq_status kq_hadamard32_quantize(const uint16_t* X, int64_t M, int64_t d, uint8_t* codes,
                                 uint8_t* scales, float* y_out, void* stream);

/*
 * kq_fwht_quantize -- full-row fast Walsh-Hadamard comparator (the FWHT
 * baseline of Sec. 4.4, Table 2): y = H_d x / sqrt(d) over the whole row,
 * H_d the Sylvester matrix, computed in fp32 by add/subtract butterflies with
 * strides 1, 2, 4, ..., d/2 (in that order) and one final multiply by the
 * fp32 nearest to 1/sqrt(d); then MXFP4 of every 32-element block.  d must be
 * a power of two from 32 to 16384 (KQ_ERROR_UNSUPPORTED otherwise); d = 32 is
 * kq_hadamard32_quantize.  Other arguments as kq_hadamard32_quantize.
 */
kq_status kq_fwht_quantize(const uint16_t* X, int64_t M, int64_t d, uint8_t* codes, uint8_t* scales,
                           float* y_out, void* stream);

/*
 * kq_mxfp4_gemm -- the W4A4 product that consumes the quantizer's output (the
 * quantized linear layer of Sec. 3.1 eq. (1) and Sec. 3.4):
 *     C[M, N] = deq(A)[M, K] . deq(B)[N, K]^T        (accumulate = 0)
 *     C[M, N] += deq(A)[M, K] . deq(B)[N, K]^T       (accumulate = 1)
 * with deq(code, s) = (-1)^sign E2M1[magnitude] 2^(s - 127).  A is an MXFP4
 * activation as written by kq_quantize* (codes [M, K/2], scales [M, K/32]) and
 * B an MXFP4 weight as written by kq_weight_transform (codes [N, K/2], scales
 * [N, K/32]); both row-major and contiguous, K a positive multiple of 32.  C
 * is fp32 [M, ldc] (ldc >= N).  Runs on the matrix cores (scaled E2M1 x E2M1
 * products, exact; fp32 accumulation in an unspecified order).  All pointers
 * are device pointers; codes 16-byte aligned, C 4-byte aligned.  M, N = 0 is
 * a no-op; M may be at most 65535 * 128.  Enqueued on `stream`; no
 * allocation, no synchronization.
 */
kq_status kq_mxfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, int64_t M, const uint8_t* b_codes,
                        const uint8_t* b_scales, int64_t N, int64_t K, float* C, int64_t ldc, int accumulate,
                        void* stream);

/*
 * kq_mxfp4_gemm_bf16 -- kq_mxfp4_gemm with the product rounded to bf16
 * (nearest, ties to even) into C [M, ldc] (bf16 bit patterns, 2-byte
 * aligned; ldc >= N), the layer output's 16-bit form: the same matrix-core
 * products and fp32 accumulation, then one rounding per element, half the
 * output bytes of the fp32 call.  No accumulate mode.  Other arguments and
 * errors as kq_mxfp4_gemm.
 */
kq_status kq_mxfp4_gemm_bf16(const uint8_t* a_codes, const uint8_t* a_scales, int64_t M, const uint8_t* b_codes,
                             const uint8_t* b_scales, int64_t N, int64_t K, uint16_t* C, int64_t ldc, void* stream);

/*
 * kq_mxfp4_quantize -- the bare MXFP4 quantizer ("Q4", the lower bound of
 * Sec. 4.4): y = x, then MXFP4.
 */
kq_status kq_mxfp4_quantize(const uint16_t* X, int64_t M, int64_t d, uint8_t* codes,
                            uint8_t* scales, void* stream);

/*
 * kq_stream_floor -- a measurement aid, not part of the method: the memory
 * traffic of the quantizers above with no arithmetic, for timing the floor
 * their launch shape and bytes alone set (2 bytes read, 17/32 byte written
 * per element, one wave per 64 blocks, the same nontemporal loads).  For
 * every 32-element block k of X it writes out16[16 k .. 16 k + 15] = the XOR
 * of the block's four 16-byte chunks and out1[k] = the low byte of
 * (word 0 XOR word 1) of that XOR (little-endian words).  X as for
 * kq_mxfp4_quantize (device bf16 [M, d], d a positive multiple of 32, 16-byte
 * aligned); out16 device [M, d/2] (16-byte aligned), out1 device [M, d/32].
 * Errors as kq_mxfp4_quantize; M = 0 is a no-op.  Enqueued on `stream`; no
 * allocation, no synchronization.
 */
kq_status kq_stream_floor(const uint16_t* X, int64_t M, int64_t d, uint8_t* out16, uint8_t* out1, void* stream);

/*
 * kq_stream_probe -- a measurement aid like kq_stream_floor (same traffic,
 * same outputs) in a launch shape given by the caller, to measure what a
 * single launch of that traffic can reach independently of the quantizers'
 * own shape: waves_per_group (1, 2, 4, 8 or 16) waves per workgroup, each
 * taking units_per_wave (1, 2 or 4) consecutive 64-block units with all
 * their loads issued before any store; groups = 0 launches one pass
 * (ceil(units / (waves_per_group * units_per_wave)) workgroups), groups > 0
 * that many workgroups walking the units in a grid-stride loop.  Other
 * arguments, outputs and errors as kq_stream_floor; a shape outside these
 * sets is KQ_ERROR_INVALID_VALUE.
 */
kq_status kq_stream_probe(const uint16_t* X, int64_t M, int64_t d, uint8_t* out16, uint8_t* out1,
                          int waves_per_group, int units_per_wave, int64_t groups, void* stream);

/*
 * kq_timestamp -- a measurement aid, not part of the method: enqueues on
 * `stream` a one-lane kernel that stores the device's constant-rate real-time
 * counter (100 MHz, the same counter on every compute unit) into dst[0], so
 * that a sequence of launches can be timed between two such stamps, also
 * inside a captured graph, without the cost of launching the graph itself.
 * dst device uint64 [1], 8-byte aligned (KQ_ERROR_NULL_POINTER /
 * KQ_ERROR_MISALIGNED otherwise, checked before anything is enqueued).  No
 * allocation, no synchronization.
 */
kq_status kq_timestamp(uint64_t* dst, void* stream);

/*
 * kq_e2m1_encode -- the element-encode step alone, for checking the device
 * conversion: codes[i] = code(v[2i]) | code(v[2i+1]) << 4 at E8M0 byte s
 * (0..254), with the rounding rule above.  v device fp32 [n], n even;
 * codes device uint8 [n/2] (4-byte aligned).
 */
kq_status kq_e2m1_encode(const float* v, int64_t n, int s, uint8_t* codes, void* stream);

/*
 * kq_weight_transform -- offline weight side (Sec. 3.4, eq. (1)):
 * W~ = W T^-T, i.e. per block w' = (A_f (x) B_f)^-T w = (A_f^-T (x) B_f^-T) w,
 * using (A (x) B)^-1 = A^-1 (x) B^-1 (Sec. 3.2).
 *   W        device bf16 [o, d];  A_host / B_host: HOST fp32 forward factors
 *            ([nfac, a, a], [nfac, b, b]) as for kq_quantize
 *   W_out    device fp32 [o, d] (required)
 *   codes, scales  device, optional (both NULL or both set): MXFP4 of W~
 * The factors are inverted on the host in fp64 (Gauss-Jordan, partial
 * pivoting), transposed and rounded to fp32; then the kq_quantize_exact
 * kernel applies them.  Returns KQ_ERROR_SINGULAR if a pivot is below 1e-12 times
 * its row's infinity norm or a factor's infinity-norm condition number
 * exceeds 1e6.  Allocates a small device buffer for the inverted factors and
 * synchronizes `stream` before returning (offline call).
 */
kq_status kq_weight_transform(const uint16_t* W, int64_t o, int64_t d, const float* A_host,
                              const float* B_host, int a, int b, int64_t nfac, float* W_out,
                              uint8_t* codes, uint8_t* scales, void* stream);

/*
 * kq_factors_inverse_transpose -- host helper for the weight side of eq. (1)
 * (Sec. 3.1: W is multiplied by T^-T so that X T (W T^-T)^T = X W^T) with the
 * inverse of a Kronecker product taken factor by factor,
 * (A (x) B)^-T = A^-T (x) B^-T (Sec. 3.2): A_it[f] = fp32(inv(A[f])^T),
 * B_it[f] = fp32(inv(B[f])^T) with fp64 Gauss-Jordan and partial pivoting.
 *   A, B     HOST fp32 [nfac, a, a], [nfac, b, b] (forward factors)
 *   A_it, B_it  HOST fp32, same shapes (caller-owned)
 * (a, b) and nfac as for kq_quantize (any nfac >= 1).  Same singularity rule
 * as kq_weight_transform (KQ_ERROR_SINGULAR, outputs then unspecified).
 */
kq_status kq_factors_inverse_transpose(const float* A, const float* B, int a, int b,
                                       int64_t nfac, float* A_it, float* B_it);

/*
 * kq_lu_to_factors -- host helper for the unit-determinant LU parametrization
 * of Sec. 3.2: abc holds, per block, the 15 parameters (a_k, b_k, c_k) for
 * k = 1..5 (HOST fp32 [nfac, 5, 3]); G_k = [[1,0],[c_k,1]] . [[a_k,b_k],[0,-1/a_k]]
 * and K = G1 (x) G2 (x) G3 (x) G4 (x) G5.  Writes HOST fp32 A [nfac, a, a],
 * B [nfac, 32/a, 32/a] with A (x) B = K^T, so that kq_quantize applies the
 * paper's x -> x K to every row block.  a in {1, 2, 4, 8}; a_k = 0 gives
 * KQ_ERROR_SINGULAR.  Computed in fp64, rounded once to fp32.
 */
kq_status kq_lu_to_factors(const float* abc, int a, int64_t nfac, float* A, float* B);

/*
 * Layer-wise calibration of the block transform (Sec. 3.3), on device.
 *
 * For the activations X [R, d] of one layer (R = N m rows: N calibration
 * samples of m tokens, stacked) and its weight W [o, d], both bf16 row-major,
 * and the transform T = diag(T_f), T_f = G_1 (x) ... (x) G_5 with the LU
 * parameters lu [nfac, 5, 3] of kq_quantize_lu (nfac = 1: one T_f for every
 * 32-column block; nfac = d / 32: one per block), the objective is
 *     L_out = || Q(X T) Q(W T^-T)^T - X W^T ||_F^2 / (R o)
 *     L_A   = || Q(X T) - X T ||_F^2 / (R d)
 *     L_W   = || Q(W T^-T) - W T^-T ||_F^2 / (o d)
 *     L     = L_out + lambda_A L_A + lambda_W L_W
 * with Q the MXFP4 quantizer of this library (Sec. 3.1).  Q(X T) is
 * kq_quantize_lu; W T^-T applies T_f^-1 = G_1^-1 (x) ... (x) G_5^-1 with the
 * closed-form inverse of a unit-determinant factor, G^-1 = [[-g11, g01],
 * [g10, -g00]] (det G = -1, Sec. 3.2), each entry of the two Kronecker
 * factors a left-to-right fp32 product of those entries, then kq_quantize;
 * the product is kq_mxfp4_gemm.
 * The gradient uses a straight-through estimator: the E2M1 rounding passes
 * the gradient unchanged, the E8M0 scale is held fixed, and an element with
 * |v| > 6 * scale (clipped) passes none.  The backward products run on the
 * bf16 matrix cores: the dequantized MXFP4 operands are exact in bf16, the
 * fp32 residual enters as two bf16 terms (hi = bf16(r), lo = bf16(r - hi),
 * within 2^-17 |r|), every product term is exact and sums are fp32; the
 * loss sums are fp64.
 *
 * kq_calib_workspace_size -- bytes of device workspace that kq_calib_step and
 * kq_calibrate need for these sizes (about 6.6 R d + 8 R o + 6.6 o d bytes
 * plus per-workgroup partial sums).  Same size checks as kq_calib_step.
 */
kq_status kq_calib_workspace_size(int64_t R, int64_t o, int64_t d, int a, int64_t nfac, size_t* bytes);

/*
 * kq_calib_reference -- Yneg = -(X W^T), fp32 [R, o] row-major (products of
 * bf16 values exact, fp32 accumulation on the matrix cores): the fixed
 * reference of L_out, computed once per layer.  X, W device, 16-byte aligned;
 * 1 <= R <= 65535 * 128, 1 <= o <= 65535 * 64; d a positive multiple of 32,
 * at most 65535 * 64.
 */
kq_status kq_calib_reference(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o, float* Yneg,
                             void* stream);

/*
 * kq_calib_step -- one evaluation of the objective and its gradient at the
 * parameters lu, optionally followed by one Adam update of lu in place.
 *   Yneg      from kq_calib_reference (device fp32 [R, o], 16-byte aligned)
 *   lambdas   device fp32 [2] = (lambda_A, lambda_W)
 *   grad      device fp32 [nfac, 5, 3]: dL/d(a_k, b_k, c_k)
 *   losses    device fp64 [4]: L_out, L_A, L_W, L at lu (before any update)
 *   adam_t    0: no update; t >= 1: Adam step t (Kingma and Ba; beta1 0.9,
 *             beta2 0.999, eps 1e-8, learning rate lr) with the moment
 *             buffers adam_m, adam_v (device fp32 [nfac * 15], zero before
 *             step 1)
 *   workspace device, 256-byte aligned, >= kq_calib_workspace_size bytes;
 *             its contents are scratch between calls.
 * Enqueued on `stream`; no allocation, no synchronization.  Errors as for
 * kq_quantize_lu and kq_mxfp4_gemm, plus KQ_ERROR_INVALID_VALUE for a short
 * workspace.
 */
kq_status kq_calib_step(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o, const float* Yneg,
                        float* lu, int a, int64_t nfac, const float* lambdas, float* grad, double* losses,
                        float* adam_m, float* adam_v, int adam_t, float lr, void* workspace,
                        size_t workspace_bytes, void* stream);

/* Scratch bytes held per GPU for kq_calib_step_noalloc (64 MiB). */
#define KQ_CALIB_NOALLOC_MAX_BYTES (64u << 20)

/*
 * kq_calib_step_noalloc -- kq_calib_step without the workspace argument and
 * without any allocation, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight loops, harnesses that forbid
 * hipMalloc).  Its workspace is a scratch array of the library in device
 * memory, KQ_CALIB_NOALLOC_MAX_BYTES bytes, one copy per GPU, held from the
 * library's first use on that GPU until the process ends; its device address
 * is looked up once per GPU on the first call there (with that GPU current).
 * Arguments, results and errors as kq_calib_step; sizes whose workspace
 * (kq_calib_workspace_size) exceeds KQ_CALIB_NOALLOC_MAX_BYTES return
 * KQ_ERROR_INVALID_VALUE before any HIP call (e.g. R = 2048 rows with
 * o = d = 1024 fit, R = 4096 with o = d = 1152 do not).  The step writes every
 * part of the scratch it reads, so what an earlier call left there does not
 * matter.  All calls on one GPU share its scratch: calls that overlap in time
 * on one GPU (concurrent streams, or host threads enqueueing on different
 * streams) race and give undefined results; calls on one stream are ordered
 * and safe.  Enqueued on `stream`; no allocation, no synchronization.
 */
kq_status kq_calib_step_noalloc(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o,
                                const float* Yneg, float* lu, int a, int64_t nfac, const float* lambdas, float* grad,
                                double* losses, float* adam_m, float* adam_v, int adam_t, float lr, void* stream);

/*
 * kq_calibrate -- the per-layer optimisation of Sec. 3.3 in one call:
 *   1. evaluate the objective at the given lu (the initial transform T_0,
 *      normally the Hadamard initialisation a = b = 1/sqrt(2), c = 1) with
 *      lambda = 0, and set lambda_A = L_out(T_0) / L_A(T_0),
 *      lambda_W = L_out(T_0) / L_W(T_0) (0 where the denominator is 0);
 *   2. `steps` Adam steps of learning rate lr on L, updating lu in place;
 *   3. evaluate the objective at the final lu.
 * losses: device fp64 [(steps + 2), 4], 8-byte aligned; row 0 is step 1's
 * evaluation (lambda = 0), row t the evaluation before update t, row
 * steps + 1 the final one (each row L_out, L_A, L_W, L).  The Adam moments,
 * lambdas and gradient live in the workspace.  Enqueued on `stream`; no
 * allocation, no synchronization.
 */
kq_status kq_calibrate(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o, const float* Yneg,
                       float* lu, int a, int64_t nfac, int steps, float lr, double* losses, void* workspace,
                       size_t workspace_bytes, void* stream);

/* Stable name of a status ("KQ_SUCCESS", ...). Never NULL. */
const char* kq_status_string(kq_status s);

/* Detail of the last failure on the calling thread ("" if none). */
const char* kq_last_error_detail(void);

/* Library version: major * 10000 + minor * 100 + patch. */
int kq_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KROQUANT_H */
