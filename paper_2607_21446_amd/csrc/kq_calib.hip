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
//   * calib_gemm_kernel: bf16 matrix-core GEMM (v_mfma_f32_32x32x16_bf16,
//     128 x 256 workgroup tile for the backward products, 128 x 128 for the
//     reference product, 32-deep K stages loaded straight into three LDS
//     buffers, two in flight) on operands stored K-contiguous.  The dequantized MXFP4 operands are exact
//     in bf16; the fp32 residual enters as two bf16 terms (hi = bf16(r),
//     lo = bf16(r - hi), |r - hi - lo| <= 2^-17 |r|), so every product term
//     is exact and sums run in fp32.  Two epilogues: the reference product
//     X W^T, and the fused gradient epilogue that turns a tile of dL/dQ into
//     dL/d(transformed operand) (mask, regulariser term) and contracts it at
//     once with the untransformed operand into 32 x 32 per-block sums
//     sum_rows left^T g (fp32 matrix cores), so the R x d gradient never
//     reaches memory;
//   * residual_prep_kernel / decode_t_kernel: the residual as its two bf16
//     terms (in its own layout and transposed, plus its sum of squares) and
//     the dequantized operands laid out K-contiguous for the products;
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
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int CT = 128;          // C tile rows of a workgroup
constexpr int BK = 32;           // K per LDS stage (bf16 elements; 64-byte rows)
constexpr int kTargetWg = 2048;  // workgroups the backward GEMMs aim for
// Workgroup shapes: 2 x WN waves of 64 x 64, a C tile of 128 x 64 WN.  The
// backward GEMMs take WN = 4 (eight waves, 128 x 256: a stage's bytes then
// carry 1.5 times the matrix-core work of the 128 x 128 tile, as A has two
// terms), the reference product WN = 2.
constexpr int kWnBackward = 4;
constexpr int kWnReference = 2;

__device__ __forceinline__ float bf16f(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }

// bf16 nearest-even of a finite fp32 value.
__device__ __forceinline__ uint32_t bf16_rne(float x) {
    const uint32_t u = __float_as_uint(x);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Value of an E2M1 code at E8M0 scale byte s (OCP MX v1.0), exact in fp32 (and in bf16).
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

// LDS stage of one operand: 128 rows x 32 bf16 (four 16-byte chunks per
// row); chunk c of row r sits at slot c ^ ((r >> 2) & 3), so the 16 lanes of
// a ds_read_b128 phase (rows r .. r + 15, one chunk each) cover all banks.
__device__ __forceinline__ int lds_off(int r, int c) { return r * 64 + 16 * (c ^ ((r >> 2) & 3)); }

// ---------------------------------------------------------------- operands
// A GEMM operand: bf16 [rows][ld], K contiguous, K extent a multiple of 32
// (zero padded by the producer), 16-byte aligned rows.  Stages of 32 K
// columns x 128 rows go straight from global memory into LDS
// (global_load_lds: lane l's 16 bytes land at the wave-uniform LDS address
// + 16 l); one instruction fills 16 rows, lane l taking row l / 4 and the
// chunk whose swizzled slot is l % 4.  Rows past the matrix load its last row
// (their products land in rows or columns the epilogues never use).
struct Opnd {
    const uint8_t* p;
    int64_t rows, ld;  // ld in bytes
};

__device__ __forceinline__ void lds_load16(const uint8_t* src, void* lds_base) {
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                     (__attribute__((address_space(3))) void*)lds_base, 16, 0, 0);
}

template <int TA, int WN>
struct StageBuf {
    uint4 a[TA][512];   // 128 rows x 4 slots of 16 bytes, slot lds_off(r, c) / 16
    uint4 b[256 * WN];  // 64 WN rows, the same layout
};

// Loads of one stage per wave (one instruction = 16 rows x 64 bytes): of
// each A term the GA = 4 / WN groups of 16 rows GA wave .. GA wave + GA - 1,
// of B the groups 2 wave and 2 wave + 1; TA GA + 2 instructions in all.
template <int TA, int WN>
constexpr int stage_loads() { return TA * (4 / WN) + 2; }

template <int TA, int WN>
__device__ __forceinline__ void stage_issue(const Opnd (&A)[TA], const Opnd& B, StageBuf<TA, WN>& sb, int wave,
                                            int lane, int64_t m0, int64_t n0, int64_t k0) {
    constexpr int GA = 4 / WN;
    const int q = lane >> 2;
    const int blk = (lane & 3) ^ ((q >> 2) & 3);
    const int64_t kb = k0 * 2 + 16 * blk;
#pragma unroll
    for (int gr = 0; gr < 2; ++gr) {
        if (gr < GA) {
            const int grp = GA * wave + gr;
#pragma unroll
            for (int x = 0; x < TA; ++x) {
                const int64_t m = min(m0 + 16 * grp + q, A[x].rows - 1);
                lds_load16(A[x].p + m * A[x].ld + kb, &sb.a[x][64 * grp]);
            }
        }
        const int grp = 2 * wave + gr;
        const int64_t n = min(n0 + 16 * grp + q, B.rows - 1);
        lds_load16(B.p + n * B.ld + kb, &sb.b[64 * grp]);
    }
}

template <int TA>
struct Frags {
    bf16x8 a[2][TA][2], b[2][2];  // [k half s][term][tile]
};

// this wave's fragments of one stage (all LDS reads of the stage, before any
// later stage is issued)
template <int TA, int WN>
__device__ __forceinline__ void stage_frags(const StageBuf<TA, WN>& sb, int h, int wm, int wn, int l32,
                                            Frags<TA>& f) {
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int i = 0; i < 2; ++i) {
#pragma unroll
            for (int x = 0; x < TA; ++x)
                f.a[s][x][i] = __builtin_bit_cast(bf16x8, sb.a[x][lds_off(wm * 64 + 32 * i + l32, 2 * h + s) / 16]);
            f.b[s][i] = __builtin_bit_cast(bf16x8, sb.b[lds_off(wn * 64 + 32 * i + l32, 2 * h + s) / 16]);
        }
}

template <int TA>
__device__ __forceinline__ void stage_mfma(const Frags<TA>& f, f32x16 (&acc)[2][2]) {
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int x = 0; x < TA; ++x)
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[s][x][i], f.b[s][j], acc[i][j], 0, 0, 0);
}

// Before stage st is used (buffer st % 3; stage st + 2 is then issued into
// buffer (st + 2) % 3, which every wave finished reading before the barrier)
// each wave waits until only its loads of stage st + 1 are outstanding, then
// a bare s_barrier (a fenced barrier would drain the loads in flight).
template <int TA, int WN>
__device__ __forceinline__ void pipe_wait(int64_t st, int64_t nst) {
    constexpr int kLoads = stage_loads<TA, WN>();
    if (st + 1 < nst)
        __builtin_amdgcn_s_waitcnt((kLoads & 15) | (7 << 4) | (15 << 8));  // vmcnt(kLoads)
    else
        __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
    __builtin_amdgcn_s_barrier();
}

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
                // per half of the 16 rows: all loads first (rows past M read row M - 1 and are
                // masked), then the arithmetic
                f32x16 g;
                float lv[16];
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    float yv[8];
                    uint32_t byte[8], sbyte[8], lraw[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        const int e = 8 * half + u;
                        const int64_t row = min(rbase + 8 * (e / 4) + 4 * h + (e % 4), M - 1);
                        yv[u] = y[row * d + col];
                        byte[u] = codes[row * (d / 2) + col / 2];
                        sbyte[u] = scales[row * nb + blk];
                        lraw[u] = left[row * d + col];
                    }
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        const int e = 8 * half + u;
                        const bool valid = rbase + 8 * (e / 4) + 4 * h + (e % 4) < M;
                        const float qv = mx_value((col & 1) ? byte[u] >> 4 : byte[u], sbyte[u]);
                        const bool pass = fabsf(yv[u]) <= 6.0f * scale_value(sbyte[u]);
                        float gv = pass ? c1 * acc[i][jj][e] : 0.f;
                        if (ks == 0) {
                            const float diff = qv - yv[u];
                            if (!pass) gv -= c2 * diff;
                            if (valid) sq += double(diff) * double(diff);
                        }
                        g[e] = valid ? gv : 0.f;
                        lv[e] = valid ? bf16f(uint16_t(lraw[u])) : 0.f;
                    }
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
    int xcd;  // 1: the column tiles of one chunk on one XCD (see calib_gemm_kernel)
};

template <int TA, class EPI>
struct GemmArgs {
    Opnd A[TA];
    Opnd B;
    EPI epi;
    GemmGrid g;
};

// C tile = sum_k A[m][k] B[n][k] over the work items (m tile, K split) of
// this workgroup, each handed to the epilogue; A has TA bf16 terms.  Three
// stage buffers, two stages in flight.
template <int TA, int WN, class EPI>
__global__ __launch_bounds__(128 * WN) void calib_gemm_kernel(const GemmArgs<TA, EPI> args) {
    __shared__ StageBuf<TA, WN> sb0, sb1, sb2;
    __shared__ double sq_lds[2 * WN];
    const GemmGrid& g = args.g;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int h = lane >> 5, l32 = lane & 31;
    // work (chunk c, column tile tn).  xcd: workgroup L of the dispatch order
    // runs on XCD L % 8, and each XCD takes a contiguous range of the works
    // (column tile fastest), so the column tiles of a chunk, which read the
    // same A rows at the same pace, share one L2
    int64_t tn = blockIdx.x, c = blockIdx.y;
    if (g.xcd) {
        const int64_t G = int64_t(gridDim.x) * gridDim.y, L = blockIdx.x + int64_t(gridDim.x) * blockIdx.y;
        const int64_t q = G >> 3, r = G & 7, x = L & 7;
        const int64_t wk = x * q + (x < r ? x : r) + (L >> 3);
        tn = wk % gridDim.x;
        c = wk / gridDim.x;
    }
    const int64_t n0 = tn * (64 * WN);

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
        const int64_t nst = k_hi > k_lo ? (k_hi - k_lo) / BK : 0;
        if (nst > 0) {
            // every wave is done with the buffers (and its earlier memory operations) before they refill
            __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));
            __syncthreads();
            stage_issue<TA, WN>(args.A, args.B, sb0, wave, lane, m0, n0, k_lo);
            if (nst > 1) stage_issue<TA, WN>(args.A, args.B, sb1, wave, lane, m0, n0, k_lo + BK);
            Frags<TA> f;
            for (int64_t st = 0; st < nst; st += 3) {
                pipe_wait<TA, WN>(st, nst);
                stage_frags<TA, WN>(sb0, h, wm, wn, l32, f);
                if (st + 2 < nst) stage_issue<TA, WN>(args.A, args.B, sb2, wave, lane, m0, n0, k_lo + (st + 2) * BK);
                stage_mfma<TA>(f, acc);
                if (st + 1 < nst) {
                    pipe_wait<TA, WN>(st + 1, nst);
                    stage_frags<TA, WN>(sb1, h, wm, wn, l32, f);
                    if (st + 3 < nst) stage_issue<TA, WN>(args.A, args.B, sb0, wave, lane, m0, n0, k_lo + (st + 3) * BK);
                    stage_mfma<TA>(f, acc);
                }
                if (st + 2 < nst) {
                    pipe_wait<TA, WN>(st + 2, nst);
                    stage_frags<TA, WN>(sb2, h, wm, wn, l32, f);
                    if (st + 4 < nst) stage_issue<TA, WN>(args.A, args.B, sb1, wave, lane, m0, n0, k_lo + (st + 4) * BK);
                    stage_mfma<TA>(f, acc);
                }
            }
        }
        args.epi.tile(acc, m0, n0, ks, wm, wn, lane, gram, sq);
    }

    if constexpr (EPI::kGram) {
        // rows 64..127 of the tile (wm = 1) join rows 0..63, then one write per block
        __syncthreads();
        float* red = reinterpret_cast<float*>(&sb0);
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
        const EPI& epi = args.epi;
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
        if (t == 0) {
            double tot = sq_lds[0];
#pragma unroll
            for (int i = 1; i < 2 * WN; ++i) tot += sq_lds[i];
            epi.sq_partial[c * gridDim.x + tn] = tot;
        }
    }
}

// One pass over the residual res [R, o] (fp32): its bf16 terms hi = bf16(r),
// lo = bf16(r - hi) both as [R, op] (K = o contiguous, zero for columns
// o .. op) and transposed as [o, Rp] (K = rows contiguous, zero for rows
// R .. Rp), and the sum of its squares per workgroup (fp64) into
// partial[blockIdx.y * gridDim.x + blockIdx.x].  Grid: 64-row x 64-column tiles.
__global__ __launch_bounds__(256) void residual_prep_kernel(const float* res, int64_t rows, int64_t cols, int64_t op,
                                                            int64_t Rp, uint16_t* nh, uint16_t* nl, uint16_t* th,
                                                            uint16_t* tl, double* partial) {
    __shared__ float tile[64][65];
    __shared__ double red[4];
    const int t = threadIdx.x;
    const int64_t r0 = int64_t(blockIdx.x) * 64, c0 = int64_t(blockIdx.y) * 64;
    double sq = 0.0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int rl = t / 16 + 16 * i, cl = 4 * (t % 16);
        const int64_t r = r0 + rl, cc = c0 + cl;
        float e[4] = {0.f, 0.f, 0.f, 0.f};
        if (r < rows) {
            const float* p = res + r * cols + cc;
            if (cols % 4 == 0 && cc + 3 < cols) {
                const float4 x = *reinterpret_cast<const float4*>(p);
                e[0] = x.x;
                e[1] = x.y;
                e[2] = x.z;
                e[3] = x.w;
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (cc + j < cols) e[j] = p[j];
            }
        }
        uint32_t hb[4], lb[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            tile[rl][cl + j] = e[j];
            sq += double(e[j]) * double(e[j]);
            hb[j] = bf16_rne(e[j]);
            lb[j] = bf16_rne(e[j] - __uint_as_float(hb[j] << 16));
        }
        // natural layout [R, op]: 4 columns (8 bytes) per thread; zero beyond o, up to op
        if (r < rows && cc < op) {
            *reinterpret_cast<uint2*>(nh + r * op + cc) = make_uint2(hb[0] | (hb[1] << 16), hb[2] | (hb[3] << 16));
            *reinterpret_cast<uint2*>(nl + r * op + cc) = make_uint2(lb[0] | (lb[1] << 16), lb[2] | (lb[3] << 16));
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sq += __shfl_xor(sq, off);
    if ((t & 63) == 0) red[t >> 6] = sq;
    __syncthreads();
    if (t == 0) partial[int64_t(blockIdx.y) * gridDim.x + blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
    const int cl = t / 4, seg = t % 4;
    const int64_t cc = c0 + cl, rr = r0 + 16 * seg;
    if (cc >= cols || rr >= Rp) return;
    uint32_t h[8], l[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float x0 = tile[16 * seg + 2 * j][cl], x1 = tile[16 * seg + 2 * j + 1][cl];
        const uint32_t h0 = bf16_rne(x0), h1 = bf16_rne(x1);
        const uint32_t l0 = bf16_rne(x0 - __uint_as_float(h0 << 16)), l1 = bf16_rne(x1 - __uint_as_float(h1 << 16));
        h[j] = h0 | (h1 << 16);
        l[j] = l0 | (l1 << 16);
    }
    uint4* ph = reinterpret_cast<uint4*>(th + cc * Rp + rr);
    uint4* pl = reinterpret_cast<uint4*>(tl + cc * Rp + rr);
    ph[0] = make_uint4(h[0], h[1], h[2], h[3]);
    ph[1] = make_uint4(h[4], h[5], h[6], h[7]);
    pl[0] = make_uint4(l[0], l[1], l[2], l[3]);
    pl[1] = make_uint4(l[4], l[5], l[6], l[7]);
}

// out[c][r] = bf16 of the dequantized MXFP4 value (r, c) (exact), c < d,
// r < ldo, zero for r >= rows: an MXFP4 matrix [rows, d] as its transpose.
__global__ __launch_bounds__(256) void decode_t_kernel(const uint8_t* codes, const uint8_t* scales, int64_t rows,
                                                       int64_t d, uint16_t* out, int64_t ldo) {
    __shared__ uint16_t tile[64][66];
    const int t = threadIdx.x;
    const int64_t r0 = int64_t(blockIdx.x) * 64, c0 = int64_t(blockIdx.y) * 64;
    {
        const int rl = t / 4, cq = t % 4;
        const int64_t r = r0 + rl, cc = c0 + 16 * cq;
        uint2 cw = make_uint2(0, 0);
        uint32_t s = 127;
        if (r < rows && cc < d) {
            cw = *reinterpret_cast<const uint2*>(codes + r * (d / 2) + cc / 2);
            s = scales[r * (d / 32) + cc / 32];
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const uint32_t w = j < 8 ? cw.x : cw.y;
            tile[rl][16 * cq + j] = uint16_t(__float_as_uint(mx_value(w >> (4 * (j % 8)), s)) >> 16);
        }
    }
    __syncthreads();
    const int cl = t / 4, seg = t % 4;
    const int64_t cc = c0 + cl, rr = r0 + 16 * seg;
    if (cc >= d || rr >= ldo) return;
    uint32_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = uint32_t(tile[16 * seg + 2 * j][cl]) | (uint32_t(tile[16 * seg + 2 * j + 1][cl]) << 16);
    uint4* p = reinterpret_cast<uint4*>(out + cc * ldo + rr);
    p[0] = make_uint4(v[0], v[1], v[2], v[3]);
    p[1] = make_uint4(v[4], v[5], v[6], v[7]);
}

// ------------------------------------------------------------ small kernels

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
    pl.ntn = cdiv(d, 64 * kWnBackward);
    pl.act_mt = cdiv(R, CT);
    pl.act_chunks = std::max<int64_t>(1, std::min(pl.act_mt, cdiv(kTargetWg, pl.ntn)));
    pl.w_mt = cdiv(o, CT);
    pl.Rp = cdiv(std::max<int64_t>(R, 1), BK) * BK;
    pl.op = cdiv(o, BK) * BK;
    const int64_t stages = pl.Rp / BK;
    pl.w_ks = std::max<int64_t>(1, std::min(cdiv(kTargetWg, pl.ntn * pl.w_mt), cdiv(stages, 8)));
    pl.w_kchunk = cdiv(cdiv(pl.Rp, pl.w_ks), BK) * BK;
    pl.w_ks = std::max<int64_t>(1, cdiv(pl.Rp, pl.w_kchunk));
    pl.w_chunks = pl.w_mt * pl.w_ks;
    pl.nsum = cdiv(pl.Rp, 64) * cdiv(o, 64);
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
    pl.rnh = take(size_t(R) * pl.op * 2);
    pl.rnl = take(size_t(R) * pl.op * 2);
    pl.rth = take(size_t(o) * pl.Rp * 2);
    pl.rtl = take(size_t(o) * pl.Rp * 2);
    pl.aht = take(size_t(d) * pl.Rp * 2);
    pl.wht = take(size_t(d) * pl.op * 2);
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
    GemmArgs<1, EpiStoreNeg> args{{{reinterpret_cast<const uint8_t*>(X), R, d * 2}},
                                  {reinterpret_cast<const uint8_t*>(W), o, d * 2},
                                  {Yneg, R, o, o},
                                  {R, o, d, cdiv(R, CT), 1, d, cdiv(R, CT), 0}};
    dim3 grid(unsigned(cdiv(o, 64 * kWnReference)), unsigned(args.g.chunks));
    calib_gemm_kernel<1, kWnReference><<<grid, 128 * kWnReference, 0, st>>>(args);
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
    uint16_t* rnh = reinterpret_cast<uint16_t*>(ws + pl.rnh);
    uint16_t* rnl = reinterpret_cast<uint16_t*>(ws + pl.rnl);
    uint16_t* rth = reinterpret_cast<uint16_t*>(ws + pl.rth);
    uint16_t* rtl = reinterpret_cast<uint16_t*>(ws + pl.rtl);
    uint16_t* aht = reinterpret_cast<uint16_t*>(ws + pl.aht);
    uint16_t* wht = reinterpret_cast<uint16_t*>(ws + pl.wht);
    float* gpa = reinterpret_cast<float*>(ws + pl.gpa);
    float* gpw = reinterpret_cast<float*>(ws + pl.gpw);
    double* sqa = reinterpret_cast<double*>(ws + pl.sqa);
    double* sqw = reinterpret_cast<double*>(ws + pl.sqw);
    double* sr = reinterpret_cast<double*>(ws + pl.sr);
    float* ga = reinterpret_cast<float*>(ws + pl.ga);
    float* gw = reinterpret_cast<float*>(ws + pl.gw);
    const int64_t R = pl.R, o = pl.o, d = pl.d;

    const float c1 = float(2.0 / (double(R) * double(o)));
    // K-contiguous operands: What^T [d, op], Ahat^T [d, Rp], res as bf16 hi / lo [R, op] and [o, Rp]
    decode_t_kernel<<<dim3(unsigned(cdiv(pl.op, 64)), unsigned(cdiv(d, 64))), 256, 0, st>>>(cW, sW, o, d, wht, pl.op);
    decode_t_kernel<<<dim3(unsigned(cdiv(pl.Rp, 64)), unsigned(cdiv(d, 64))), 256, 0, st>>>(cA, sA, R, d, aht, pl.Rp);
    residual_prep_kernel<<<dim3(unsigned(cdiv(pl.Rp, 64)), unsigned(cdiv(o, 64))), 256, 0, st>>>(
        res, R, o, pl.op, pl.Rp, rnh, rnl, rth, rtl, sr);
    // activation side: P = res . What  (M = R, N = d, K = o)
    {
        GemmArgs<2, EpiGram> args{
            {{reinterpret_cast<const uint8_t*>(rnh), R, pl.op * 2}, {reinterpret_cast<const uint8_t*>(rnl), R, pl.op * 2}},
            {reinterpret_cast<const uint8_t*>(wht), d, pl.op * 2},
            {s.X, yA, cA, sA, R, d, c1, s.lambdas, 0, float(2.0 / (double(R) * double(d))), gpa, sqa},
            {R, d, pl.op, pl.act_mt, 1, pl.op, pl.act_chunks, 1}};
        dim3 grid(unsigned(pl.ntn), unsigned(pl.act_chunks));
        calib_gemm_kernel<2, kWnBackward><<<grid, 128 * kWnBackward, 0, st>>>(args);
    }
    // weight side: P = res^T . Ahat  (M = o, N = d, K = R)
    {
        GemmArgs<2, EpiGram> args{
            {{reinterpret_cast<const uint8_t*>(rth), o, pl.Rp * 2}, {reinterpret_cast<const uint8_t*>(rtl), o, pl.Rp * 2}},
            {reinterpret_cast<const uint8_t*>(aht), d, pl.Rp * 2},
            {s.W, yW, cW, sW, o, d, c1, s.lambdas, 1, float(2.0 / (double(o) * double(d))), gpw, sqw},
            {o, d, pl.Rp, pl.w_mt, pl.w_ks, pl.w_kchunk, pl.w_chunks, 1}};
        dim3 grid(unsigned(pl.ntn), unsigned(pl.w_chunks));
        calib_gemm_kernel<2, kWnBackward><<<grid, 128 * kWnBackward, 0, st>>>(args);
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
    la.nsr = pl.nsum;
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

}  // namespace kq
