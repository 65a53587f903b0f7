// Layer-wise calibration of the block transform (Sec. 3.3).
//
// One step evaluates, for the activations X [R, d] and weight W [o, d] of a
// layer and the transform T = diag(T_f), T_f = G_1 (x) ... (x) G_5 (Sec. 3.2),
//   L_out = ||Q(X T) Q(W T^-T)^T - X W^T||^2 / (R o)
//   L_A   = ||Q(X T) - X T||^2 / (R d),   L_W = ||Q(W T^-T) - W T^-T||^2 / (o d)
//   L     = L_out + lambda_A L_A + lambda_W L_W
// and its gradient with respect to the 15 LU parameters of every block,
// with a straight-through estimator for Q: the E2M1 rounding passes the
// gradient unchanged, the E8M0 scale (a step function of the block maximum)
// is held fixed, and an element clipped at +-6 * scale passes none.  The
// forward products come from the quantizers and the W4A4 GEMM of the
// library; this file holds the backward pass:
//   * calib_gemm_kernel: fp32 matrix-core GEMM (v_mfma_f32_32x32x2_f32,
//     128 x 128 workgroup tile, 16-deep K stages double-buffered in LDS) with
//     two epilogues -- the reference product X W^T, and the fused gradient
//     epilogue that turns a tile of dL/dQ into dL/d(transformed operand)
//     (mask, regulariser term) and contracts it at once with the untransformed
//     operand into 32 x 32 per-block sums  sum_rows left^T g  on the matrix
//     cores, so the R x d gradient never reaches memory;
//   * gram_reduce_kernel: fixed-order sum of the per-workgroup block sums;
//   * lu_grad_kernel: chain rule through T^-T and the Kronecker product to the
//     2 x 2 factors and their (a, b, c), the losses, and the Adam update.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "kq_calib.h"

namespace kq {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int CT = 128;      // C tile edge of a workgroup (rows and columns)
constexpr int CK = 16;       // K rows per LDS stage
constexpr int CS = CT + 4;   // LDS row stride (floats): the two MFMA k-halves read rows 8 apart,
                             // 8 * 132 = 32 (mod 64) banks apart
constexpr int kSumParts = 1024;  // partial sums of the residual's squares
constexpr int kTargetWg = 2048;  // workgroups the backward GEMMs aim for

__device__ __forceinline__ float bf16f(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }

// Value of an E2M1 code at E8M0 scale byte s (OCP MX v1.0), exact in fp32.
__device__ __forceinline__ float mx_value(uint32_t nib, uint32_t s) {
    const uint32_t m = nib & 7u;
    const uint32_t bits = m >= 2 ? (((126u + (m >> 1)) << 23) | ((m & 1u) << 22)) : (m == 1 ? (126u << 23) : 0u);
    const float scale = s ? __uint_as_float(s << 23) : __uint_as_float(0x00400000u);
    const float v = __uint_as_float(bits) * scale;
    return (nib & 8u) ? -v : v;
}

__device__ __forceinline__ float scale_value(uint32_t s) {
    return s ? __uint_as_float(s << 23) : __uint_as_float(0x00400000u);
}

__device__ __forceinline__ f32x16 mfma32(float a, float b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------- loaders
// Each loader stages a CK x CT slab of one operand (K rows, 128 M or N
// columns) into an LDS buffer laid out [k][col] with stride CS; load() reads
// global memory into registers (rows/cols beyond the matrix and k >= kend
// read as 0), store() writes them to LDS.

// fp32 row-major [rows][ld], K contiguous (the residual read along o).
struct LoadRowF32 {
    const float* src;
    int64_t rows, ld;
    bool vec;
    float4 v[2];
    __device__ void load(int64_t r0, int64_t k0, int64_t kend, int t) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int64_t gr = r0 + t / 4 + 64 * i;
            const int64_t gk = k0 + 4 * (t % 4);
            float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
            if (gr < rows) {
                const float* p = src + gr * ld + gk;
                if (vec && gk + 3 < kend) {
                    x = *reinterpret_cast<const float4*>(p);
                } else {
                    if (gk < kend) x.x = p[0];
                    if (gk + 1 < kend) x.y = p[1];
                    if (gk + 2 < kend) x.z = p[2];
                    if (gk + 3 < kend) x.w = p[3];
                }
            }
            v[i] = x;
        }
    }
    __device__ void store(float* lds, int t) const {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int row = t / 4 + 64 * i, k = 4 * (t % 4);
            lds[(k + 0) * CS + row] = v[i].x;
            lds[(k + 1) * CS + row] = v[i].y;
            lds[(k + 2) * CS + row] = v[i].z;
            lds[(k + 3) * CS + row] = v[i].w;
        }
    }
};

// bf16 row-major [rows][ld], K contiguous (X and W of the reference product).
struct LoadRowBF16 {
    const uint16_t* src;
    int64_t rows, ld;
    bool vec;
    uint16_t v[8];
    __device__ void load(int64_t r0, int64_t k0, int64_t kend, int t) {
        const int64_t gr = r0 + t / 2;
        const int64_t gk = k0 + 8 * (t % 2);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0;
        if (gr < rows) {
            const uint16_t* p = src + gr * ld + gk;
            if (vec && gk + 7 < kend) {
                const uint4 x = *reinterpret_cast<const uint4*>(p);
                const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = uint16_t(w[e / 2] >> (16 * (e % 2)));
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (gk + e < kend) v[e] = p[e];
            }
        }
    }
    __device__ void store(float* lds, int t) const {
        const int row = t / 2, k = 8 * (t % 2);
#pragma unroll
        for (int e = 0; e < 8; ++e) lds[(k + e) * CS + row] = bf16f(v[e]);
    }
};

// fp32 [K][ld] with the M index contiguous (the residual read as its transpose).
struct LoadColF32 {
    const float* src;
    int64_t cols, ld;  // cols: extent of the contiguous index
    bool vec;
    float4 v[2];
    __device__ void load(int64_t m0, int64_t k0, int64_t kend, int t) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int64_t gk = k0 + t / 32 + 8 * i;
            const int64_t gm = m0 + 4 * (t % 32);
            float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
            if (gk < kend) {
                const float* p = src + gk * ld + gm;
                if (vec && gm + 3 < cols) {
                    x = *reinterpret_cast<const float4*>(p);
                } else {
                    if (gm < cols) x.x = p[0];
                    if (gm + 1 < cols) x.y = p[1];
                    if (gm + 2 < cols) x.z = p[2];
                    if (gm + 3 < cols) x.w = p[3];
                }
            }
            v[i] = x;
        }
    }
    __device__ void store(float* lds, int t) const {
#pragma unroll
        for (int i = 0; i < 2; ++i)
            *reinterpret_cast<float4*>(&lds[(t / 32 + 8 * i) * CS + 4 * (t % 32)]) = v[i];
    }
};

// MXFP4 matrix [K][N] as the quantizer writes it (codes [K][N/2], two per
// byte, low nibble first; scales [K][N/32]); N a multiple of 32.  Decoded to
// exact fp32 values.
struct LoadMx {
    const uint8_t* codes;
    const uint8_t* scales;
    int64_t N;
    uint32_t c, s;
    __device__ void load(int64_t n0, int64_t k0, int64_t kend, int t) {
        const int64_t gk = k0 + t / 16;
        const int64_t gn = n0 + 8 * (t % 16);
        c = 0;
        s = 127;
        if (gk < kend && gn < N) {
            c = *reinterpret_cast<const uint32_t*>(codes + gk * (N / 2) + gn / 2);
            s = scales[gk * (N / 32) + gn / 32];
        }
    }
    __device__ void store(float* lds, int t) const {
        float4 lo, hi;
        lo.x = mx_value(c, s);
        lo.y = mx_value(c >> 4, s);
        lo.z = mx_value(c >> 8, s);
        lo.w = mx_value(c >> 12, s);
        hi.x = mx_value(c >> 16, s);
        hi.y = mx_value(c >> 20, s);
        hi.z = mx_value(c >> 24, s);
        hi.w = mx_value(c >> 28, s);
        float* p = &lds[(t / 16) * CS + 8 * (t % 16)];
        *reinterpret_cast<float4*>(p) = lo;
        *reinterpret_cast<float4*>(p + 4) = hi;
    }
};

// --------------------------------------------------------------- epilogues
// The accumulator of a 32 x 32 MFMA tile holds, in lane l (h = l / 32) and
// register 4q + r, element (row 8q + 4h + r, column l % 32).

// Yneg = -acc (the reference product of the loss).
struct EpiStoreNeg {
    float* out;
    int64_t M, N, ld;
    static constexpr bool kGram = false;
    __device__ void tile(const f32x16 (&acc)[2][2], int64_t m0, int64_t n0, int64_t, int wm, int wn, int lane,
                         f32x16 (&)[2], double&) const {
        const int h = lane >> 5, l32 = lane & 31;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int jj = 0; jj < 2; ++jj) {
                const int64_t col = n0 + wn * 64 + 32 * jj + l32;
                if (col >= N) continue;
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int64_t row = m0 + wm * 64 + 32 * i + 8 * (e / 4) + 4 * h + (e % 4);
                    if (row < M) out[row * ld + col] = -acc[i][jj][e];
                }
            }
    }
};

// Gradient epilogue.  acc holds a tile of  P = dL_out/dQ * (R o) / 2  for the
// quantized operand Q [M, d] (exact up to the split of K, which is linear).
// With y the operand before quantization (fp32 from the quantizer) and
// m = [|y| <= 6 * scale] the straight-through mask,
//   g = c1 * P * m + [ks == 0] * c2 * (Q - y) * (m - 1)
// is the tile of dL/dy (c1 = 2 / (R o), c2 = lambda * 2 / (rows d)); the
// per-block sums  S_j += left_j^T g_j  (left = the operand before the
// transform, bf16) run on the matrix cores with the rows as the K index,
// taking g straight from the accumulator registers.  [ks == 0] tiles also add
// (Q - y)^2 to the regulariser sum.
struct EpiGram {
    const uint16_t* left;   // [M, d] bf16
    const float* y;         // [M, d]
    const uint8_t* codes;   // [M, d / 2]
    const uint8_t* scales;  // [M, d / 32]
    int64_t M, d;
    float c1;
    const float* lambdas;
    int lam_index;
    float c2_unit;          // 2 / (rows d); c2 = lambda * c2_unit
    float* partial;         // [chunks, d / 32, 32, 32]
    double* sq_partial;     // [chunks, ntn]
    static constexpr bool kGram = true;
    __device__ void tile(const f32x16 (&acc)[2][2], int64_t m0, int64_t n0, int64_t ks, int wm, int wn, int lane,
                         f32x16 (&gram)[2], double& sq) const {
        const int h = lane >> 5, l32 = lane & 31;
        const float c2 = lambdas[lam_index] * c2_unit;
        const int64_t nb = d / 32;
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
            const int64_t blk = (n0 + wn * 64 + 32 * jj) / 32;
            if (blk >= nb) continue;
            const int64_t col = blk * 32 + l32;
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int64_t rbase = m0 + wm * 64 + 32 * i;
                if (rbase >= M) continue;
                f32x16 g;
                float lv[16];
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int64_t row = rbase + 8 * (e / 4) + 4 * h + (e % 4);
                    float gv = 0.f, lf = 0.f;
                    if (row < M) {
                        const float yv = y[row * d + col];
                        const uint32_t byte = codes[row * (d / 2) + col / 2];
                        const uint32_t sb = scales[row * nb + blk];
                        const float qv = mx_value((col & 1) ? byte >> 4 : byte, sb);
                        const bool pass = fabsf(yv) <= 6.0f * scale_value(sb);
                        gv = pass ? c1 * acc[i][jj][e] : 0.f;
                        if (ks == 0) {
                            const float diff = qv - yv;
                            if (!pass) gv -= c2 * diff;
                            sq += double(diff) * double(diff);
                        }
                        lf = bf16f(left[row * d + col]);
                    }
                    g[e] = gv;
                    lv[e] = lf;
                }
#pragma unroll
                for (int e = 0; e < 16; ++e) gram[jj] = mfma32(lv[e], g[e], gram[jj]);
            }
        }
    }
};

struct GemmGrid {
    int64_t M, N, K;
    int64_t m_tiles, ks, kchunk, chunks;
};

template <class LA, class LB, class EPI>
__global__ __launch_bounds__(256) void calib_gemm_kernel(LA la, LB lb, const EPI epi, const GemmGrid g) {
    __shared__ float lds[2][2][CK * CS];
    __shared__ double sq_lds[4];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int h = lane >> 5, l32 = lane & 31;
    const int64_t tn = blockIdx.x, c = blockIdx.y;
    const int64_t n0 = tn * CT;

    f32x16 gram[2];
    gram[0] = f32x16{};
    gram[1] = f32x16{};
    double sq = 0.0;

    for (int64_t it = c; it < g.m_tiles * g.ks; it += g.chunks) {
        const int64_t mt = it / g.ks, ks = it % g.ks;
        const int64_t m0 = mt * CT;
        const int64_t k_lo = ks * g.kchunk, k_hi = std::min(g.K, k_lo + g.kchunk);
        f32x16 acc[2][2];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

        if (k_lo < k_hi) {
            la.load(m0, k_lo, k_hi, t);
            lb.load(n0, k_lo, k_hi, t);
            la.store(lds[0][0], t);
            lb.store(lds[0][1], t);
            __syncthreads();
            int buf = 0;
            for (int64_t k0 = k_lo; k0 < k_hi; k0 += CK) {
                const bool more = k0 + CK < k_hi;
                if (more) {
                    la.load(m0, k0 + CK, k_hi, t);
                    lb.load(n0, k0 + CK, k_hi, t);
                }
                const float* As = lds[buf][0];
                const float* Bs = lds[buf][1];
#pragma unroll
                for (int s = 0; s < CK / 2; ++s) {
                    const int kr = s + (CK / 2) * h;
                    const float a0 = As[kr * CS + wm * 64 + l32], a1 = As[kr * CS + wm * 64 + 32 + l32];
                    const float b0 = Bs[kr * CS + wn * 64 + l32], b1 = Bs[kr * CS + wn * 64 + 32 + l32];
                    acc[0][0] = mfma32(a0, b0, acc[0][0]);
                    acc[0][1] = mfma32(a0, b1, acc[0][1]);
                    acc[1][0] = mfma32(a1, b0, acc[1][0]);
                    acc[1][1] = mfma32(a1, b1, acc[1][1]);
                }
                if (more) {
                    la.store(lds[buf ^ 1][0], t);
                    lb.store(lds[buf ^ 1][1], t);
                }
                __syncthreads();
                buf ^= 1;
            }
        }
        epi.tile(acc, m0, n0, ks, wm, wn, lane, gram, sq);
    }

    if constexpr (EPI::kGram) {
        // rows 64..127 of the tile (wm = 1) join rows 0..63, then one write per block
        float* red = &lds[0][0][0];
        if (wm == 1) {
#pragma unroll
            for (int jj = 0; jj < 2; ++jj)
#pragma unroll
                for (int e = 0; e < 16; ++e) red[((wn * 2 + jj) * 16 + e) * 64 + lane] = gram[jj][e];
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) sq += __shfl_xor(sq, off);
        if (lane == 0) sq_lds[wave] = sq;
        __syncthreads();
        if (wm == 0) {
            const int64_t nb = epi.d / 32;
#pragma unroll
            for (int jj = 0; jj < 2; ++jj) {
                const int64_t blk = (n0 + wn * 64 + 32 * jj) / 32;
                if (blk >= nb) continue;
                float* dst = epi.partial + (c * nb + blk) * 1024;
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int p = 8 * (e / 4) + 4 * h + (e % 4);
                    dst[p * 32 + l32] = gram[jj][e] + red[((wn * 2 + jj) * 16 + e) * 64 + lane];
                }
            }
        }
        if (t == 0) epi.sq_partial[c * gridDim.x + tn] = ((sq_lds[0] + sq_lds[1]) + sq_lds[2]) + sq_lds[3];
    }
}

// ------------------------------------------------------------ small kernels

// sum of squares of v[0 .. n) into partial[blockIdx.x] (grid-stride, fp64).
__global__ __launch_bounds__(256) void sumsq_kernel(const float* v, int64_t n, double* partial) {
    __shared__ double red[4];
    double s = 0.0;
    const int64_t n4 = n / 4;
    const float4* v4 = reinterpret_cast<const float4*>(v);
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n4; i += int64_t(gridDim.x) * 256) {
        const float4 x = v4[i];
        s += double(x.x) * x.x + double(x.y) * x.y + double(x.z) * x.z + double(x.w) * x.w;
    }
    if (blockIdx.x == 0 && threadIdx.x < n - 4 * n4) {
        const double x = v[4 * n4 + threadIdx.x];
        s += x * x;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) partial[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

// out[f][e] = sum over chunks c and the blocks j of factor f of partial[c][j][e];
// one factor per block j (nfac = nb) or one for all (nfac = 1).  Fixed order.
__global__ __launch_bounds__(256) void gram_reduce_kernel(const float* partial, int64_t chunks, int64_t nb,
                                                          int64_t nfac, float* out) {
    const int64_t f = blockIdx.x;
    const int e = blockIdx.y * 256 + threadIdx.x;
    const int64_t j0 = nfac == 1 ? 0 : f, j1 = nfac == 1 ? nb : f + 1;
    double s = 0.0;
    for (int64_t j = j0; j < j1; ++j)
        for (int64_t c = 0; c < chunks; ++c) s += partial[(c * nb + j) * 1024 + e];
    out[f * 1024 + e] = float(s);
}

__device__ __forceinline__ void decode_g(const float* lu, float (&g)[5][4]) {
#pragma unroll
    for (int k = 0; k < 5; ++k) {
        const float pa = lu[3 * k], pb = lu[3 * k + 1], pc = lu[3 * k + 2];
        g[k][0] = pa;
        g[k][1] = pb;
        g[k][2] = pc * pa;
        g[k][3] = __builtin_fmaf(pc, pb, -(1.0f / pa));
    }
}

// Factors of T_f^-1 in the layout kq_quantize applies (y = (A (x) B) x per
// block, so A (x) B = T^-1 gives the weight side's w -> w T^-T).  With
// det G = -1, G^-1 = [[-g11, g01], [g10, -g00]]; every entry of A and B is the
// product of its G^-1 entries, left to right, in fp32.
__global__ __launch_bounds__(64) void inverse_factors_kernel(const float* lu, int na, float* Ainv, float* Binv) {
    const int64_t f = blockIdx.x;
    const int a = 1 << na, b = 32 >> na;
    float g[5][4];
    decode_g(lu + f * 15, g);
    float gi[5][4];
#pragma unroll
    for (int k = 0; k < 5; ++k) {
        gi[k][0] = -g[k][3];
        gi[k][1] = g[k][1];
        gi[k][2] = g[k][2];
        gi[k][3] = -g[k][0];
    }
    for (int idx = threadIdx.x; idx < a * a + b * b; idx += 64) {
        const bool in_a = idx < a * a;
        const int row = in_a ? idx / a : (idx - a * a) / b;
        const int col = in_a ? idx % a : (idx - a * a) % b;
        float v = 1.0f;
        bool first = true;
#pragma unroll
        for (int k = 0; k < 5; ++k) {
            if ((k < na) != in_a) continue;
            const int sh = in_a ? na - 1 - k : 4 - k;
            const int e = 2 * ((row >> sh) & 1) + ((col >> sh) & 1);
            const float ge = e == 0 ? gi[k][0] : e == 1 ? gi[k][1] : e == 2 ? gi[k][2] : gi[k][3];
            v = first ? ge : v * ge;
            first = false;
        }
        if (in_a) Ainv[f * a * a + idx] = v;
        else Binv[f * b * b + idx - a * a] = v;
    }
}

__device__ __forceinline__ double block_sum256(double v, double* red) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    return ((red[0] + red[1]) + red[2]) + red[3];
}

struct LuGradArgs {
    const float* lu;
    const float* ga;   // [nfac, 32, 32]  dL/dT_f from the activation side
    const float* gw;   // [nfac, 32, 32]  dL/dU_f, U_f = T_f^-T, from the weight side
    float* grad;       // [nfac, 15]
    float* lu_out;
    float* adam_m;
    float* adam_v;
    int adam_t;
    float lr;
    // losses (block 0)
    const double* sr;
    int64_t nsr;
    const double* sqa;
    int64_t nsqa;
    const double* sqw;
    int64_t nsqw;
    double n_out, n_a, n_w;  // R o, R d, o d
    const float* lambdas;
    double* losses;
};

// dL/dT_f = GA_f - U GW_f^T U (U = T_f^-T; d(T^-T) = -U dT^T U), then for
// every factor G_k of T_f = G_1 (x) ... (x) G_5:
//   dL/dG_k[u][v] = sum_{p, q: bit_k(p) = u, bit_k(q) = v} dT[p][q] prod_{l != k} G_l[bit_l(p)][bit_l(q)]
// (bit_1 the most significant of the 5-bit index), and for G = [[a, b], [c a, c b - 1/a]]:
//   dL/da = dG00 + c dG10 + dG11 / a^2,  dL/db = dG01 + c dG11,  dL/dc = a dG10 + b dG11.
__global__ __launch_bounds__(256) void lu_grad_kernel(const LuGradArgs p) {
    __shared__ float sU[32][33];
    __shared__ float sGW[32][33];
    __shared__ float sV[32][33];
    __shared__ double red[4];
    __shared__ float gsum[5][4];
    const int64_t f = blockIdx.x;
    const int t = threadIdx.x;
    float g[5][4];
    decode_g(p.lu + f * 15, g);
    // (G^-1)^T = [[-g11, g10], [g01, -g00]]
    float git[5][4];
#pragma unroll
    for (int k = 0; k < 5; ++k) {
        git[k][0] = -g[k][3];
        git[k][1] = g[k][2];
        git[k][2] = g[k][1];
        git[k][3] = -g[k][0];
    }
    for (int e = t; e < 1024; e += 256) {
        const int r = e / 32, q = e % 32;
        float u = 1.0f;
#pragma unroll
        for (int k = 0; k < 5; ++k) {
            const int ee = 2 * ((r >> (4 - k)) & 1) + ((q >> (4 - k)) & 1);
            u *= ee == 0 ? git[k][0] : ee == 1 ? git[k][1] : ee == 2 ? git[k][2] : git[k][3];
        }
        sU[r][q] = u;
        sGW[r][q] = p.gw[f * 1024 + e];
    }
    __syncthreads();
    // V = GW^T U
    for (int e = t; e < 1024; e += 256) {
        const int r = e / 32, q = e % 32;
        float s = 0.f;
        for (int x = 0; x < 32; ++x) s = __builtin_fmaf(sGW[x][r], sU[x][q], s);
        sV[r][q] = s;
    }
    __syncthreads();
    double dg[5][4];
#pragma unroll
    for (int k = 0; k < 5; ++k)
#pragma unroll
        for (int e = 0; e < 4; ++e) dg[k][e] = 0.0;
    for (int e = t; e < 1024; e += 256) {
        const int r = e / 32, q = e % 32;
        float s = 0.f;
        for (int x = 0; x < 32; ++x) s = __builtin_fmaf(sU[r][x], sV[x][q], s);
        const float dT = p.ga[f * 1024 + e] - s;
        float ge[5];
#pragma unroll
        for (int k = 0; k < 5; ++k) {
            const int ee = 2 * ((r >> (4 - k)) & 1) + ((q >> (4 - k)) & 1);
            ge[k] = ee == 0 ? g[k][0] : ee == 1 ? g[k][1] : ee == 2 ? g[k][2] : g[k][3];
        }
#pragma unroll
        for (int k = 0; k < 5; ++k) {
            double others = dT;
#pragma unroll
            for (int l = 0; l < 5; ++l)
                if (l != k) others *= ge[l];
            const int ee = 2 * ((r >> (4 - k)) & 1) + ((q >> (4 - k)) & 1);
#pragma unroll
            for (int x = 0; x < 4; ++x) dg[k][x] += (x == ee) ? others : 0.0;
        }
    }
#pragma unroll
    for (int k = 0; k < 5; ++k)
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            const double s = block_sum256(dg[k][x], red);
            if (t == 0) gsum[k][x] = float(s);
        }
    __syncthreads();
    if (t < 5) {
        const int k = t;
        const float pa = p.lu[f * 15 + 3 * k], pb = p.lu[f * 15 + 3 * k + 1], pc = p.lu[f * 15 + 3 * k + 2];
        const float d00 = gsum[k][0], d01 = gsum[k][1], d10 = gsum[k][2], d11 = gsum[k][3];
        float gr[3];
        gr[0] = d00 + pc * d10 + d11 / (pa * pa);
        gr[1] = d01 + pc * d11;
        gr[2] = pa * d10 + pb * d11;
        const float par[3] = {pa, pb, pc};
#pragma unroll
        for (int x = 0; x < 3; ++x) {
            const int64_t i = f * 15 + 3 * k + x;
            p.grad[i] = gr[x];
            if (p.adam_t > 0) {
                // Adam (Kingma and Ba), beta1 0.9, beta2 0.999, eps 1e-8
                const float m = 0.9f * p.adam_m[i] + 0.1f * gr[x];
                const float v = 0.999f * p.adam_v[i] + 0.001f * gr[x] * gr[x];
                p.adam_m[i] = m;
                p.adam_v[i] = v;
                const float bc1 = 1.0f - powf(0.9f, float(p.adam_t));
                const float bc2 = 1.0f - powf(0.999f, float(p.adam_t));
                p.lu_out[i] = par[x] - p.lr * (m / bc1) / (sqrtf(v / bc2) + 1e-8f);
            }
        }
    }
    if (f == 0) {
        double s = 0.0;
        for (int64_t i = t; i < p.nsr; i += 256) s += p.sr[i];
        const double sr = block_sum256(s, red);
        s = 0.0;
        for (int64_t i = t; i < p.nsqa; i += 256) s += p.sqa[i];
        const double sa = block_sum256(s, red);
        s = 0.0;
        for (int64_t i = t; i < p.nsqw; i += 256) s += p.sqw[i];
        const double sw = block_sum256(s, red);
        if (t == 0) {
            const double lo = sr / p.n_out, la = sa / p.n_a, lw = sw / p.n_w;
            p.losses[0] = lo;
            p.losses[1] = la;
            p.losses[2] = lw;
            p.losses[3] = lo + double(p.lambdas[0]) * la + double(p.lambdas[1]) * lw;
        }
    }
}

__global__ void init_kernel(float* m, float* v, int64_t n, float* lambdas) {
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x) {
        m[i] = 0.f;
        v[i] = 0.f;
    }
    if (blockIdx.x == 0 && threadIdx.x < 2) lambdas[threadIdx.x] = 0.f;
}

// lambda_A = L_out / L_A, lambda_W = L_out / L_W at the initial transform (0 if the denominator is 0).
__global__ void set_lambdas_kernel(const double* losses, float* lambdas) {
    if (threadIdx.x == 0) {
        lambdas[0] = losses[1] > 0.0 ? float(losses[0] / losses[1]) : 0.f;
        lambdas[1] = losses[2] > 0.0 ? float(losses[0] / losses[2]) : 0.f;
    }
}

__global__ __launch_bounds__(256) void copy_kernel(const float4* src, float4* dst, int64_t n4, const float* s1,
                                                   float* d1, int64_t tail) {
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n4; i += int64_t(gridDim.x) * 256) dst[i] = src[i];
    if (blockIdx.x == 0 && threadIdx.x < tail) d1[threadIdx.x] = s1[threadIdx.x];
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

CalibPlan calib_plan(int64_t R, int64_t o, int64_t d, int a, int64_t nfac) {
    CalibPlan pl;
    pl.R = R;
    pl.o = o;
    pl.d = d;
    pl.nb = d / 32;
    pl.a = a;
    pl.nfac = nfac;
    pl.ntn = cdiv(d, CT);
    pl.act_mt = cdiv(R, CT);
    pl.act_chunks = std::max<int64_t>(1, std::min(pl.act_mt, cdiv(kTargetWg, pl.ntn)));
    pl.w_mt = cdiv(o, CT);
    const int64_t stages = std::max<int64_t>(1, cdiv(R, CK));
    pl.w_ks = std::max<int64_t>(1, std::min(cdiv(kTargetWg, pl.ntn * pl.w_mt), cdiv(stages, 8)));
    pl.w_kchunk = cdiv(cdiv(std::max<int64_t>(R, 1), pl.w_ks), CK) * CK;
    pl.w_ks = std::max<int64_t>(1, cdiv(std::max<int64_t>(R, 1), pl.w_kchunk));
    pl.w_chunks = pl.w_mt * pl.w_ks;
    pl.nsum = kSumParts;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = align256(off + bytes);
        return at;
    };
    const int b = 32 / a;
    pl.yA = take(size_t(R) * d * 4);
    pl.cA = take(size_t(R) * d / 2);
    pl.sA = take(size_t(R) * (d / 32));
    pl.yW = take(size_t(o) * d * 4);
    pl.cW = take(size_t(o) * d / 2);
    pl.sW = take(size_t(o) * (d / 32));
    pl.res = take(size_t(R) * o * 4);
    pl.fa = take(size_t(nfac) * a * a * 4);
    pl.fb = take(size_t(nfac) * b * b * 4);
    pl.gpa = take(size_t(pl.act_chunks) * pl.nb * 1024 * 4);
    pl.gpw = take(size_t(pl.w_chunks) * pl.nb * 1024 * 4);
    pl.sqa = take(size_t(pl.act_chunks) * pl.ntn * 8);
    pl.sqw = take(size_t(pl.w_chunks) * pl.ntn * 8);
    pl.sr = take(size_t(pl.nsum) * 8);
    pl.ga = take(size_t(nfac) * 1024 * 4);
    pl.gw = take(size_t(nfac) * 1024 * 4);
    pl.grad = take(size_t(nfac) * 15 * 4);
    pl.am = take(size_t(nfac) * 15 * 4);
    pl.av = take(size_t(nfac) * 15 * 4);
    pl.lam = take(2 * 4);
    pl.total = off;
    return pl;
}

hipError_t launch_calib_reference(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o,
                                  float* Yneg, hipStream_t st) {
    if (R == 0 || o == 0) return hipSuccess;
    const bool vec = d % 8 == 0;
    LoadRowBF16 la{X, R, d, vec, {}};
    LoadRowBF16 lb{W, o, d, vec, {}};
    EpiStoreNeg epi{Yneg, R, o, o};
    GemmGrid g{R, o, d, cdiv(R, CT), 1, cdiv(d, CK) * CK, cdiv(R, CT)};
    dim3 grid(unsigned(cdiv(o, CT)), unsigned(g.chunks));
    calib_gemm_kernel<<<grid, 256, 0, st>>>(la, lb, epi, g);
    return hipGetLastError();
}

hipError_t launch_calib_inverse_factors(const float* lu, int a, int64_t nfac, float* Ainv, float* Binv,
                                        hipStream_t st) {
    const int na = a == 1 ? 0 : a == 2 ? 1 : a == 4 ? 2 : 3;
    inverse_factors_kernel<<<unsigned(nfac), 64, 0, st>>>(lu, na, Ainv, Binv);
    return hipGetLastError();
}

hipError_t launch_calib_backward(const CalibPlan& pl, const CalibStepArgs& s, hipStream_t st) {
    unsigned char* ws = s.ws;
    float* yA = reinterpret_cast<float*>(ws + pl.yA);
    const uint8_t* cA = ws + pl.cA;
    const uint8_t* sA = ws + pl.sA;
    float* yW = reinterpret_cast<float*>(ws + pl.yW);
    const uint8_t* cW = ws + pl.cW;
    const uint8_t* sW = ws + pl.sW;
    float* res = reinterpret_cast<float*>(ws + pl.res);
    float* gpa = reinterpret_cast<float*>(ws + pl.gpa);
    float* gpw = reinterpret_cast<float*>(ws + pl.gpw);
    double* sqa = reinterpret_cast<double*>(ws + pl.sqa);
    double* sqw = reinterpret_cast<double*>(ws + pl.sqw);
    double* sr = reinterpret_cast<double*>(ws + pl.sr);
    float* ga = reinterpret_cast<float*>(ws + pl.ga);
    float* gw = reinterpret_cast<float*>(ws + pl.gw);
    const int64_t R = pl.R, o = pl.o, d = pl.d;

    sumsq_kernel<<<kSumParts, 256, 0, st>>>(res, R * o, sr);
    const float c1 = float(2.0 / (double(R) * double(o)));
    // activation side: P = res . What  (M = R, N = d, K = o)
    {
        LoadRowF32 la{res, R, o, o % 4 == 0, {}};
        LoadMx lb{cW, sW, d, 0, 0};
        EpiGram epi{s.X, yA, cA, sA, R, d, c1, s.lambdas, 0, float(2.0 / (double(R) * double(d))), gpa, sqa};
        GemmGrid g{R, d, o, pl.act_mt, 1, cdiv(o, CK) * CK, pl.act_chunks};
        dim3 grid(unsigned(pl.ntn), unsigned(pl.act_chunks));
        calib_gemm_kernel<<<grid, 256, 0, st>>>(la, lb, epi, g);
    }
    // weight side: P = res^T . Ahat  (M = o, N = d, K = R)
    {
        LoadColF32 la{res, o, o, o % 4 == 0, {}};
        LoadMx lb{cA, sA, d, 0, 0};
        EpiGram epi{s.W, yW, cW, sW, o, d, c1, s.lambdas, 1, float(2.0 / (double(o) * double(d))), gpw, sqw};
        GemmGrid g{o, d, R, pl.w_mt, pl.w_ks, pl.w_kchunk, pl.w_chunks};
        dim3 grid(unsigned(pl.ntn), unsigned(pl.w_chunks));
        calib_gemm_kernel<<<grid, 256, 0, st>>>(la, lb, epi, g);
    }
    gram_reduce_kernel<<<dim3(unsigned(pl.nfac), 4), 256, 0, st>>>(gpa, pl.act_chunks, pl.nb, pl.nfac, ga);
    gram_reduce_kernel<<<dim3(unsigned(pl.nfac), 4), 256, 0, st>>>(gpw, pl.w_chunks, pl.nb, pl.nfac, gw);
    LuGradArgs la{};
    la.lu = s.lu;
    la.ga = ga;
    la.gw = gw;
    la.grad = s.grad;
    la.lu_out = s.lu_out;
    la.adam_m = s.adam_m;
    la.adam_v = s.adam_v;
    la.adam_t = s.adam_t;
    la.lr = s.lr;
    la.sr = sr;
    la.nsr = kSumParts;
    la.sqa = sqa;
    la.nsqa = pl.act_chunks * pl.ntn;
    la.sqw = sqw;
    la.nsqw = pl.w_chunks * pl.ntn;
    la.n_out = double(R) * double(o);
    la.n_a = double(R) * double(d);
    la.n_w = double(o) * double(d);
    la.lambdas = s.lambdas;
    la.losses = s.losses;
    lu_grad_kernel<<<unsigned(pl.nfac), 256, 0, st>>>(la);
    return hipGetLastError();
}

hipError_t launch_calib_init(float* adam_m, float* adam_v, int64_t n, float* lambdas, hipStream_t st) {
    init_kernel<<<1, 256, 0, st>>>(adam_m, adam_v, n, lambdas);
    return hipGetLastError();
}

hipError_t launch_calib_set_lambdas(const double* losses, float* lambdas, hipStream_t st) {
    set_lambdas_kernel<<<1, 64, 0, st>>>(losses, lambdas);
    return hipGetLastError();
}

hipError_t launch_calib_copy(const float* src, float* dst, int64_t n, hipStream_t st) {
    const int64_t n4 = n / 4;
    const unsigned grid = unsigned(std::max<int64_t>(1, std::min<int64_t>(cdiv(n4, 256), 4096)));
    copy_kernel<<<grid, 256, 0, st>>>(reinterpret_cast<const float4*>(src), reinterpret_cast<float4*>(dst), n4,
                                      src + 4 * n4, dst + 4 * n4, n - 4 * n4);
    return hipGetLastError();
}

}  // namespace kq
