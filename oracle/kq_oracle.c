/*
 * KroQuant CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * This file is the plain, slow, obviously-correct reference for the online
 * activation quantizer of "KroQuant: Kronecker-Structured Block Transforms for
 * Efficient Post-Training Quantization of Diffusion Transformers".  Only the
 * test suite, the smoke check and the benchmark's CPU-baseline leg may load it.
 * It shares no code, header, table or constant with the HIP library: every
 * rule below is written out again from the paper and from the OCP
 * Microscaling (MX) v1.0 format that the paper quantizes to.
 *
 * Build (see oracle/__init__.py):  gcc -O2 -ffp-contract=off -fopenmp -shared -fPIC
 * -ffp-contract=off keeps the compiler from fusing a*b+c on its own; every
 * fused multiply-add below is an explicit fmaf() and every other product and
 * sum is rounded to fp32 on its own.
 *
 * What is computed, per row r of X[M, d] (bf16) and per column block j of 32
 * elements (Sec. 3.1 "Quantization setup": row-wise blocks of n = 32 sharing
 * one scale; block-diagonal T = diag(K^(1), ..., K^(d/32)), Sec. 3.1 "Goal"):
 *
 *   1. x = the 32 bf16 values widened to fp32 (exact).
 *   2. y = (A (x) B) x, the Kronecker-structured block transform of Sec. 3.2,
 *      evaluated through the identity (A (x) B) vec(X) = vec(B X A^T) on the
 *      block reshaped row-major to a x b (Xm[p][q] = x[p*b+q]), i.e.
 *      Ym = A . Xm . B^T.  Evaluation order (the canonical fp32 order):
 *        Z[p][i] = B[i][0]*Xm[p][0];  Z[p][i] = fmaf(B[i][q], Xm[p][q], Z[p][i]), q = 1..b-1
 *        Y[o][i] = A[o][0]*Z[0][i];   Y[o][i] = fmaf(A[o][p], Z[p][i],  Y[o][i]), p = 1..a-1
 *        y[o*b+i] = Y[o][i].
 *      The paper leaves the fp32 order open (Sec. 3.5 only says fp32
 *      accumulation); this order is the reading adopted for parity.
 *   3. MXFP4 encode of the fp32 y (Sec. 3.1; format per OCP MX v1.0, which
 *      the paper cites for MXFP4):
 *        shared exponent E = floor(log2(max_k |y_k|)) - 2   (2 = emax of E2M1)
 *        stored E8M0 byte  s = clamp(E + 127, 0, 254);  s = 0 for an all-zero block
 *        element code      = sign bit (bit 3) | index of the E2M1 magnitude
 *                            {0, .5, 1, 1.5, 2, 3, 4, 6} nearest to |y_k| / 2^(s-127),
 *                            ties to the even index, saturating at 6.
 *        packing           codes[r, 16j + i] = code(2i) | code(2i+1) << 4.
 *
 * Comparators (Sec. 4.4 and the ablation of Sec. 4.3):
 *   SmoothQuant   y_c = x_c * m_c (per-channel multiplier m = 1/s, Appendix D "Smoothing").
 *   Hadamard-32   y = H32 x / sqrt(32), H32 the Sylvester matrix = H2 (x) ... (x) H2 (Sec. 3.2
 *                 "Hadamard initialization"), evaluated by add/subtract butterflies with
 *                 strides 1, 2, 4, 8, 16 followed by one multiply by fp32(1/sqrt(32)).
 *   plain MXFP4   y = x (the bare quantizer, "Q4" of Sec. 4.4).
 *
 * Every entry point returns 0 on success and a negative value on a bad
 * argument; it never allocates beyond the stack.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define BLK 32

/* --- bf16 -> fp32: the bf16 bit pattern is the upper half of the fp32 one. */
static float bf16_to_f32(uint16_t h) {
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* --- E8M0 shared scale of one block (OCP MX v1.0; Sec. 3.1 shared scale s).
 * floor(log2(amax)) comes from frexp, which returns amax = m * 2^e with
 * m in [0.5, 1), so floor(log2(amax)) = e - 1 for every finite amax > 0,
 * subnormals included. */
static int e8m0_scale(float amax) {
    if (!(amax > 0.0f)) return 0;              /* all-zero block: smallest scale */
    int e;
    (void)frexp((double)amax, &e);
    int shared = (e - 1) - 2;                  /* floor(log2 amax) - emax(E2M1) */
    int s = shared + 127;
    if (s < 0) s = 0;
    if (s > 254) s = 254;
    return s;
}

/* --- E2M1 element code (OCP MX v1.0 FP4 E2M1: 1 sign, 2 exponent, 1 mantissa
 * bit; magnitudes indexed by the 3 low code bits).  Brute-force nearest over
 * the eight magnitudes, exact in double; on a tie the even index wins (round
 * half to even on the code).  Values above 6 pick 6 (saturation). */
static const double kE2M1[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};

static int e2m1_code(float y, int s) {
    double v = ldexp(fabs((double)y), 127 - s); /* exact: a power-of-two rescale in double */
    int best = 0;
    double bestd = fabs(v - kE2M1[0]);
    for (int k = 1; k < 8; ++k) {
        double dk = fabs(v - kE2M1[k]);
        if (dk < bestd || (dk == bestd && (k % 2 == 0) && (best % 2 == 1))) {
            best = k;
            bestd = dk;
        }
    }
    return best | (signbit(y) ? 8 : 0);
}

/* --- encode one block of 32 fp32 values: scale byte + 16 packed bytes. */
static void encode_block(const float* y, uint8_t* codes16, uint8_t* scale) {
    float amax = 0.0f;
    for (int k = 0; k < BLK; ++k) {
        float a = fabsf(y[k]);
        if (a > amax) amax = a;
    }
    int s = e8m0_scale(amax);
    *scale = (uint8_t)s;
    for (int i = 0; i < BLK / 2; ++i) {
        int lo = e2m1_code(y[2 * i], s);
        int hi = e2m1_code(y[2 * i + 1], s);
        codes16[i] = (uint8_t)(lo | (hi << 4));
    }
}

/* --- y = (A (x) B) x for one block, canonical order (see header). */
static void kron_block(const float* x, const float* A, const float* B, int a, int b, float* y) {
    float Z[BLK];
    for (int p = 0; p < a; ++p) {
        for (int i = 0; i < b; ++i) {
            float z = B[i * b + 0] * x[p * b + 0];
            for (int q = 1; q < b; ++q) z = fmaf(B[i * b + q], x[p * b + q], z);
            Z[p * b + i] = z;
        }
    }
    for (int o = 0; o < a; ++o) {
        for (int i = 0; i < b; ++i) {
            float acc = A[o * a + 0] * Z[0 * b + i];
            for (int p = 1; p < a; ++p) acc = fmaf(A[o * a + p], Z[p * b + i], acc);
            y[o * b + i] = acc;
        }
    }
}

/* --- Hadamard-32 of one block: Sylvester butterflies, then 1/sqrt(32). */
static void hadamard32_block(const float* x, float* y) {
    float u[BLK];
    for (int k = 0; k < BLK; ++k) u[k] = x[k];
    for (int h = 1; h < BLK; h <<= 1) {
        for (int i = 0; i < BLK; ++i) {
            if (i & h) continue;
            float s0 = u[i] + u[i + h];
            float s1 = u[i] - u[i + h];
            u[i] = s0;
            u[i + h] = s1;
        }
    }
    const float inv_sqrt32 = (float)(1.0 / sqrt(32.0)); /* nearest fp32 to 1/sqrt(32) */
    for (int k = 0; k < BLK; ++k) y[k] = u[k] * inv_sqrt32;
}

static int valid_ab(int a, int b) {
    return (a == 4 && b == 8) || (a == 2 && b == 16) || (a == 8 && b == 4) || (a == 1 && b == 32);
}

enum { KIND_KRON = 0, KIND_SMOOTH = 1, KIND_HAD = 2, KIND_PLAIN = 3, KIND_KRON_F32IN = 4 };

/* Shared driver: rows in parallel; each output element is produced by
 * exactly one iteration and its value does not depend on the thread count. */
static int run(int kind, const void* Xv, int64_t M, int64_t d, const float* A, const float* B,
               int a, int b, int64_t nfac, const float* mult, uint8_t* codes, uint8_t* scales,
               float* yout) {
    if (M < 0 || d <= 0 || d % BLK != 0) return -1;
    if (!Xv || !codes || !scales) return -2;
    int64_t nb = d / BLK;
    if (kind == KIND_KRON || kind == KIND_KRON_F32IN) {
        if (!A || !B) return -2;
        if (!valid_ab(a, b)) return -3;
        if (nfac != 1 && nfac != nb) return -4;
    }
    if (kind == KIND_SMOOTH && !mult) return -2;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < M; ++r) {
        float x[BLK], y[BLK];
        for (int64_t j = 0; j < nb; ++j) {
            int64_t base = r * d + j * BLK;
            for (int k = 0; k < BLK; ++k) {
                if (kind == KIND_KRON_F32IN)
                    x[k] = ((const float*)Xv)[base + k];
                else
                    x[k] = bf16_to_f32(((const uint16_t*)Xv)[base + k]);
            }
            switch (kind) {
                case KIND_KRON:
                case KIND_KRON_F32IN: {
                    int64_t f = (nfac == 1) ? 0 : j;
                    kron_block(x, A + f * a * a, B + f * b * b, a, b, y);
                    break;
                }
                case KIND_SMOOTH:
                    for (int k = 0; k < BLK; ++k) y[k] = x[k] * mult[j * BLK + k];
                    break;
                case KIND_HAD:
                    hadamard32_block(x, y);
                    break;
                default:
                    for (int k = 0; k < BLK; ++k) y[k] = x[k];
                    break;
            }
            encode_block(y, codes + r * (d / 2) + j * (BLK / 2), scales + r * nb + j);
            if (yout)
                for (int k = 0; k < BLK; ++k) yout[base + k] = y[k];
        }
    }
    return 0;
}

/* KroQuant quantizer: per block y = (A (x) B) x, then MXFP4 (Sec. 3.2, 3.5).
 * A: [nfac, a, a], B: [nfac, b, b] fp32 row-major; nfac = 1 (shared) or d/32. */
int kqo_quantize(const uint16_t* X, int64_t M, int64_t d, const float* A, const float* B, int a,
                 int b, int64_t nfac, uint8_t* codes, uint8_t* scales, float* yout) {
    return run(KIND_KRON, X, M, d, A, B, a, b, nfac, NULL, codes, scales, yout);
}

/* Same transform on fp32 input rows (used for the weight side, Sec. 3.4, and
 * for round-trip checks). */
int kqo_quantize_f32(const float* X, int64_t M, int64_t d, const float* A, const float* B, int a,
                     int b, int64_t nfac, uint8_t* codes, uint8_t* scales, float* yout) {
    return run(KIND_KRON_F32IN, X, M, d, A, B, a, b, nfac, NULL, codes, scales, yout);
}

/* SmoothQuant comparator: y_c = x_c * mult_c, then MXFP4 (Sec. 4.4 "Scale"). */
int kqo_smoothquant(const uint16_t* X, int64_t M, int64_t d, const float* mult, uint8_t* codes,
                    uint8_t* scales, float* yout) {
    return run(KIND_SMOOTH, X, M, d, NULL, NULL, 0, 0, 1, mult, codes, scales, yout);
}

/* Hadamard-32 comparator: y = H32 x / sqrt(32), then MXFP4 (Sec. 1, Sec. 4.3). */
int kqo_hadamard32(const uint16_t* X, int64_t M, int64_t d, uint8_t* codes, uint8_t* scales,
                   float* yout) {
    return run(KIND_HAD, X, M, d, NULL, NULL, 0, 0, 1, NULL, codes, scales, yout);
}

/* Plain MXFP4 of the bf16 input ("Q4", Sec. 4.4). */
int kqo_mxfp4(const uint16_t* X, int64_t M, int64_t d, uint8_t* codes, uint8_t* scales) {
    return run(KIND_PLAIN, X, M, d, NULL, NULL, 0, 0, 1, NULL, codes, scales, NULL);
}

/* Element encode alone: one unpacked code per value at E8M0 byte s. */
int kqo_e2m1_codes(const float* v, int64_t n, int s, uint8_t* out) {
    if (n < 0 || s < 0 || s > 254) return -1;
    if (n > 0 && (!v || !out)) return -2;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = (uint8_t)e2m1_code(v[i], s);
    return 0;
}

/* Scale rule alone: E8M0 byte of each block maximum. */
int kqo_e8m0_scales(const float* amax, int64_t n, uint8_t* out) {
    if (n < 0) return -1;
    if (n > 0 && (!amax || !out)) return -2;
    for (int64_t i = 0; i < n; ++i) out[i] = (uint8_t)e8m0_scale(amax[i]);
    return 0;
}

/* Full-row fast Walsh-Hadamard transform comparator (the FWHT column of
 * Sec. 4.4, Table 2; Hadamard rotations of the whole hidden dimension, Sec. 1
 * and 2): for d = 2^n, y = H_d x / sqrt(d) with H_d the Sylvester matrix
 * H_2 (x) ... (x) H_2, evaluated by butterflies
 *     (u_i, u_{i+h}) <- (u_i + u_{i+h}, u_i - u_{i+h}),  h = 1, 2, 4, ..., d/2,
 * in fp32, then one multiply by the fp32 nearest to 1/sqrt(d); then MXFP4 of
 * every 32-element block of the transformed row.  For d = 32 this is exactly
 * the Hadamard-32 comparator.  Returns -1 (nothing written) unless d is a
 * power of two from 32 to 2^16. */
int kqo_fwht(const uint16_t* X, int64_t M, int64_t d, uint8_t* codes, uint8_t* scales, float* yout) {
    /* d a power of two from 32 up to the row buffer below (2^16 elements) */
    if (M < 0 || d < BLK || d > (1 << 16) || (d & (d - 1)) != 0) return -1;
    if (!X || !codes || !scales) return -2;
    const float inv_sqrt_d = (float)(1.0 / sqrt((double)d));
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < M; ++r) {
        float u[1 << 16];
        for (int64_t k = 0; k < d; ++k) u[k] = bf16_to_f32(X[r * d + k]);
        for (int64_t h = 1; h < d; h <<= 1) {
            for (int64_t i = 0; i < d; ++i) {
                if (i & h) continue;
                float s0 = u[i] + u[i + h];
                float s1 = u[i] - u[i + h];
                u[i] = s0;
                u[i + h] = s1;
            }
        }
        for (int64_t k = 0; k < d; ++k) u[k] = u[k] * inv_sqrt_d;
        for (int64_t j = 0; j < d / BLK; ++j)
            encode_block(u + j * BLK, codes + r * (d / 2) + j * (BLK / 2), scales + r * (d / BLK) + j);
        if (yout)
            for (int64_t k = 0; k < d; ++k) yout[r * d + k] = u[k];
    }
    return 0;
}

/* Factors of the on-the-fly variant K2 from the paper's LU parameters (Sec. 3.2
 * "Parametrization", Sec. 3.5 "K2").  For each factor pair f, lu[f][k] =
 * (a_k, b_k, c_k), k = 0..4, parametrize the 2x2 factor G_{k+1} = L U with
 * L = [[1, 0], [c, 1]] and U = [[a, b], [0, -1/a]], so
 *     G = [[a, b], [c a, c b - 1/a]]   (det G = -1).
 * The paper's block K = G_1 (x) ... (x) G_5 multiplies row activations from the
 * right (x^T K, eq. (1)), i.e. y = K^T x per block, and
 * K^T = A (x) B with A = G_1^T (x) ... (x) G_na^T (a x a, na = log2 a) and
 * B = G_{na+1}^T (x) ... (x) G_5^T (b x b): entrywise (Kronecker index order,
 * most significant index bit with the first factor)
 *     A[o][p] = prod_{k<na}  G_k[bit(p, na-1-k)][bit(o, na-1-k)]
 *     B[i][q] = prod_{k>=na} G_k[bit(q, 4-k)][bit(i, 4-k)]
 * (an empty product, A for a = 1, is 1).  fp32 order (the reading adopted for
 * parity; the paper does not fix it): g10 = c*a, g11 = fmaf(c, b, -(1/a)) with
 * 1/a correctly rounded, and each product left to right with one rounding per
 * multiply.  a_k must be nonzero.  Output A [nfac, a, a], B [nfac, b, b]. */
static float lu_entry(const float* g /* [5][2][2] */, int k0, int k1, int top, int row, int col) {
    float v = 1.0f;
    int first = 1;
    for (int k = k0; k < k1; ++k) {
        int sh = top - (k - k0);
        float e = g[k * 4 + ((row >> sh) & 1) * 2 + ((col >> sh) & 1)];
        v = first ? e : v * e;
        first = 0;
    }
    return v;
}

int kqo_lu_factors(const float* lu, int a, int64_t nfac, float* A, float* B) {
    int na = a == 1 ? 0 : a == 2 ? 1 : a == 4 ? 2 : a == 8 ? 3 : -1;
    if (na < 0 || nfac < 1) return -3;
    if (!lu || !A || !B) return -2;
    int b = BLK / a;
    for (int64_t f = 0; f < nfac; ++f) {
        float g[5 * 4];
        for (int k = 0; k < 5; ++k) {
            float pa = lu[f * 15 + 3 * k], pb = lu[f * 15 + 3 * k + 1], pc = lu[f * 15 + 3 * k + 2];
            if (pa == 0.0f) return -5;
            float inv = 1.0f / pa;
            g[k * 4 + 0] = pa;
            g[k * 4 + 1] = pb;
            g[k * 4 + 2] = pc * pa;
            g[k * 4 + 3] = fmaf(pc, pb, -inv);
        }
        /* A^T of the first na factors: entry (o, p) reads G[bit of p][bit of o] */
        for (int o = 0; o < a; ++o)
            for (int p = 0; p < a; ++p) A[f * a * a + o * a + p] = lu_entry(g, 0, na, na - 1, p, o);
        for (int i = 0; i < b; ++i)
            for (int q = 0; q < b; ++q) B[f * b * b + i * b + q] = lu_entry(g, na, 5, 4 - na, q, i);
    }
    return 0;
}

/* Weight-side factors for the same parameters (Sec. 3.2, Sec. 3.4): the
 * weight is multiplied by T^-T, i.e. every block row w^T becomes w^T K^-T, so
 * as a column map w -> K^-1 w with K^-1 = G1^-1 (x) ... (x) G5^-1 (the inverse
 * of a Kronecker product is the product of the inverses).  A unit-determinant
 * factor has det G = -1, so G^-1 = -adj(G) = [[-g11, g01], [g10, -g00]].
 * Writes A' (x) B' = K^-1: A'[o][p] = prod over the first na factors of
 * G_k^-1[bit of o][bit of p], B' likewise over the rest, fp32 products left to
 * right from the fp32 g entries of kqo_lu_factors. */
int kqo_lu_inverse_factors(const float* lu, int a, int64_t nfac, float* A, float* B) {
    int na = a == 1 ? 0 : a == 2 ? 1 : a == 4 ? 2 : a == 8 ? 3 : -1;
    if (na < 0 || nfac < 1) return -3;
    if (!lu || !A || !B) return -2;
    int b = BLK / a;
    for (int64_t f = 0; f < nfac; ++f) {
        float gi[5 * 4];
        for (int k = 0; k < 5; ++k) {
            float pa = lu[f * 15 + 3 * k], pb = lu[f * 15 + 3 * k + 1], pc = lu[f * 15 + 3 * k + 2];
            if (pa == 0.0f) return -5;
            float g00 = pa, g01 = pb, g10 = pc * pa, g11 = fmaf(pc, pb, -(1.0f / pa));
            gi[k * 4 + 0] = -g11;
            gi[k * 4 + 1] = g01;
            gi[k * 4 + 2] = g10;
            gi[k * 4 + 3] = -g00;
        }
        for (int o = 0; o < a; ++o)
            for (int p = 0; p < a; ++p) A[f * a * a + o * a + p] = lu_entry(gi, 0, na, na - 1, o, p);
        for (int i = 0; i < b; ++i)
            for (int q = 0; q < b; ++q) B[f * b * b + i * b + q] = lu_entry(gi, na, 5, 4 - na, i, q);
    }
    return 0;
}

/* fp32 -> bf16, round to nearest, ties to the even bf16 (the 16-bit output of
 * the transformed activation): the two bf16 neighbours of v are its 16-bit
 * truncation toward zero and the next one away from zero; the nearer one
 * wins, a tie goes to the one whose last mantissa bit is 0.  Finite inputs. */
int kqo_f32_to_bf16(const float* v, int64_t n, uint16_t* out) {
    if (n < 0) return -1;
    if (n > 0 && (!v || !out)) return -2;
    for (int64_t i = 0; i < n; ++i) {
        uint32_t u;
        memcpy(&u, &v[i], 4);
        uint32_t lo = u & 0xFFFF0000u, hi = lo + 0x10000u;
        float flo, fhi;
        memcpy(&flo, &lo, 4);
        memcpy(&fhi, &hi, 4);
        double dl = fabs((double)v[i] - (double)flo), dh = fabs((double)fhi - (double)v[i]);
        uint32_t pick = (dl < dh) ? lo : (dh < dl) ? hi : (((lo >> 16) & 1u) ? hi : lo);
        out[i] = (uint16_t)(pick >> 16);
    }
    return 0;
}

/* Number of OpenMP threads a parallel region would use (for reporting). */
#ifdef _OPENMP
#include <omp.h>
int kqo_num_threads(void) { return omp_get_max_threads(); }
void kqo_set_num_threads(int n) { omp_set_num_threads(n); }
#else
int kqo_num_threads(void) { return 1; }
void kqo_set_num_threads(int n) { (void)n; }
#endif
