// KroQuant online activation quantizer: HIP kernels for gfx950 (MI355X).
//
// One lane owns one whole 32-element block (Sec. 3.1: row-wise blocks of 32
// sharing one E8M0 scale).  The block's 64 input bytes, its 32 transformed
// fp32 values, its amax, scale and 16 code bytes all stay in that lane's
// registers, so the transform, the amax and the encode need no cross-lane
// traffic.  Factors are wave-uniform and are read with scalar loads.
//
// Two lane -> block mappings:
//   FLAT    the blocks of the matrix are one flat array (rows are contiguous);
//           lane l of sub-tile k of wave unit u owns block (u*U + k)*64 + l.
//           Stores of one sub-tile are 1 KiB of codes and 64 B of scales,
//           both contiguous.  Used when every block has the same factors.
//   COLUMN  wave unit u owns column block j = u % nb over 64*U consecutive
//           rows (lane = row), so per-block factors K^(j) (T = diag(K^(1..d/32)),
//           Sec. 3.1) are uniform across the wave.
//
// Arithmetic contract (kept bit-identical to the reference evaluation order):
//   Kronecker  Z[p][i] = B[i][0]*Xm[p][0], then fma(B[i][q], Xm[p][q], .) for q = 1..b-1;
//              Y[o][i] = A[o][0]*Z[0][i],  then fma(A[o][p], Z[p][i], .)  for p = 1..a-1;
//              Xm[p][q] = x[p*b+q], y[o*b+i] = Y[o][i]            (Sec. 3.2, Sec. 3.5)
//   Hadamard   butterflies (u_i, u_i+h) <- (u_i + u_i+h, u_i - u_i+h), h = 1, 2, 4, 8, 16,
//              then * fp32(1/sqrt(32))                              (Sec. 1, Sec. 3.2)
//   Smooth     y_c = x_c * m_c                                      (Sec. 4.4, Appendix D)
//   MXFP4      s = max(biased_exp(amax) - 2, 0); code = RNE_sat(|y| / 2^(s-127)) | sign
//              via the gfx950 scaled FP4 convert, whose scale operand is the float
//              with exponent field s (mantissa ignored by the hardware).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kq_kernels.h"

namespace kq {

// ------------------------------------------------------------------ helpers
__device__ __forceinline__ void unpack8(const uint4 r, float* x) {
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
}

__device__ __forceinline__ void load_block(const uint16_t* __restrict__ X, int64_t blk, uint4 (&r)[4]) {
    const uint4* p = reinterpret_cast<const uint4*>(X) + blk * 4;
#pragma unroll
    for (int m = 0; m < 4; ++m) r[m] = p[m];
}

// Wave-uniform read-only loads through the constant address space: the
// compiler then uses scalar loads (SGPR results) instead of one vector load
// per lane of the same address.
typedef const __attribute__((address_space(4))) float* const_f32_ptr;
__device__ __forceinline__ float ld_uniform(const float* base, int64_t idx) {
    return ((const_f32_ptr)base)[idx];
}

// E8M0 byte of a block maximum (amax >= 0, finite): biased exponent - 2, at least 0.
__device__ __forceinline__ uint32_t e8m0_byte(float amax) {
    const uint32_t e = __float_as_uint(amax) >> 23;
    return e > 2u ? e - 2u : 0u;
}

// Encode 32 fp32 values: returns the scale byte, writes 4 dwords of packed codes.
__device__ __forceinline__ uint32_t encode32(const float (&y)[32], uint32_t (&w)[4]) {
    float amax = 0.0f;
#pragma unroll
    for (int k = 0; k < 32; ++k) amax = fmaxf(amax, fabsf(y[k]));
    const uint32_t s = e8m0_byte(amax);
    const float sc = __uint_as_float(s << 23);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t acc = 0;
        acc = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(acc, y[8 * i + 0], y[8 * i + 1], sc, 0);
        acc = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(acc, y[8 * i + 2], y[8 * i + 3], sc, 1);
        acc = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(acc, y[8 * i + 4], y[8 * i + 5], sc, 2);
        acc = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(acc, y[8 * i + 6], y[8 * i + 7], sc, 3);
        w[i] = acc;
    }
    return s;
}

// ------------------------------------------------------------------ transforms
// Each op: setup(f) with f the factor index (uniform in the COLUMN mapping,
// 0 for shared factors), apply(x, y).
struct PlainOp {
    __device__ __forceinline__ void setup(const Params&, int64_t) {}
    __device__ __forceinline__ void apply(const float (&x)[32], float (&y)[32], int64_t) const {
#pragma unroll
        for (int k = 0; k < 32; ++k) y[k] = x[k];
    }
};

// COLUMN mapping: the wave's column block is uniform, multipliers come in
// through scalar loads.
struct SmoothUniformOp {
    const float* m;
    __device__ __forceinline__ void setup(const Params& p, int64_t j) { m = p.mult + j * 32; }
    __device__ __forceinline__ void apply(const float (&x)[32], float (&y)[32], int64_t) const {
#pragma unroll
        for (int k = 0; k < 32; ++k) y[k] = x[k] * ld_uniform(m, k);
    }
};

// FLAT mapping: every lane has its own column block, multipliers come in
// through per-lane vector loads (the [d] array stays cache resident).
struct SmoothLaneOp {
    const float* m;
    __device__ __forceinline__ void setup(const Params& p, int64_t) { m = p.mult; }
    __device__ __forceinline__ void apply(const float (&x)[32], float (&y)[32], int64_t col) const {
        const float4* mv = reinterpret_cast<const float4*>(m + col * 32);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const float4 f = mv[k];
            y[4 * k + 0] = x[4 * k + 0] * f.x;
            y[4 * k + 1] = x[4 * k + 1] * f.y;
            y[4 * k + 2] = x[4 * k + 2] * f.z;
            y[4 * k + 3] = x[4 * k + 3] * f.w;
        }
    }
};

struct HadamardOp {
    __device__ __forceinline__ void setup(const Params&, int64_t) {}
    __device__ __forceinline__ void apply(const float (&x)[32], float (&y)[32], int64_t) const {
        float u[32];
#pragma unroll
        for (int k = 0; k < 32; ++k) u[k] = x[k];
#pragma unroll
        for (int h = 1; h < 32; h <<= 1) {
#pragma unroll
            for (int i = 0; i < 32; ++i) {
                if (i & h) continue;
                const float s0 = u[i] + u[i + h];
                const float s1 = u[i] - u[i + h];
                u[i] = s0;
                u[i + h] = s1;
            }
        }
        const float r = 0x1.6a09e6p-3f;  // fp32 nearest to 1/sqrt(32), 0x3E3504F3
#pragma unroll
        for (int k = 0; k < 32; ++k) y[k] = u[k] * r;
    }
};

template <int NA, int NB>
struct KronOp {
    static_assert(NA * NB == 32, "a*b must be 32");
    const float* A;
    const float* B;
    // f: factor pair of this wave (0 when every block shares one pair)
    __device__ __forceinline__ void setup(const Params& p, int64_t f) {
        const int64_t g = p.nfac == 1 ? 0 : f;
        A = p.A + g * (NA * NA);
        B = p.B + g * (NB * NB);
    }
    __device__ __forceinline__ void apply(const float (&x)[32], float (&y)[32], int64_t) const {
        float z[32];
#pragma unroll
        for (int i = 0; i < NB; ++i) {
#pragma unroll
            for (int pr = 0; pr < NA; ++pr) {
                float acc = ld_uniform(B, i * NB) * x[pr * NB];
#pragma unroll
                for (int q = 1; q < NB; ++q) acc = __builtin_fmaf(ld_uniform(B, i * NB + q), x[pr * NB + q], acc);
                z[pr * NB + i] = acc;
            }
        }
#pragma unroll
        for (int o = 0; o < NA; ++o) {
#pragma unroll
            for (int i = 0; i < NB; ++i) {
                float acc = ld_uniform(A, o * NA) * z[i];
#pragma unroll
                for (int pr = 1; pr < NA; ++pr) acc = __builtin_fmaf(ld_uniform(A, o * NA + pr), z[pr * NB + i], acc);
                y[o * NB + i] = acc;
            }
        }
    }
};

// ------------------------------------------------------------------ kernels
template <int U>
struct Tile {
    uint4 raw[U][4];
};

// per-block body shared by both mappings
template <class Op>
__device__ __forceinline__ void process_block(const Op& op, const uint4 (&raw)[4], const Params& p,
                                              int64_t blk, int64_t col) {
    const int64_t codes_off = blk * 16, scale_off = blk, y_off = blk * 32;
    float x[32], y[32];
#pragma unroll
    for (int m = 0; m < 4; ++m) unpack8(raw[m], x + 8 * m);
    op.apply(x, y, col);
    uint32_t w[4];
    const uint32_t s = encode32(y, w);
    if (p.codes) {
        *reinterpret_cast<uint4*>(p.codes + codes_off) = make_uint4(w[0], w[1], w[2], w[3]);
        p.scales[scale_off] = (uint8_t)s;
    }
    if (p.y) {
        float4* dst = reinterpret_cast<float4*>(p.y + y_off);
#pragma unroll
        for (int m = 0; m < 8; ++m)
            dst[m] = make_float4(y[4 * m], y[4 * m + 1], y[4 * m + 2], y[4 * m + 3]);
    }
}

template <int U, class Op>
__global__ __launch_bounds__(kThreads) void flat_kernel(const Params p) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t stride = (int64_t)gridDim.x * (kThreads / 64);
    Op op;
    op.setup(p, 0);
    for (int64_t u = (int64_t)blockIdx.x * (kThreads / 64) + wave; u < p.units; u += stride) {
        Tile<U> t;
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t blk = (u * U + k) * 64 + lane;
            if (blk < p.nblocks) load_block(p.X, blk, t.raw[k]);
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t blk = (u * U + k) * 64 + lane;
            if (blk < p.nblocks) process_block(op, t.raw[k], p, blk, blk % p.nb);
        }
    }
}

template <int U, class Op>
__global__ __launch_bounds__(kThreads) void column_kernel(const Params p) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t stride = (int64_t)gridDim.x * (kThreads / 64);
    for (int64_t u = (int64_t)blockIdx.x * (kThreads / 64) + wave; u < p.units; u += stride) {
        const int64_t j = u % p.nb;
        const int64_t row0 = (u / p.nb) * (64 * U);
        Op op;
        op.setup(p, j);
        Tile<U> t;
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t r = row0 + k * 64 + lane;
            if (r < p.M) load_block(p.X, r * p.nb + j, t.raw[k]);
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t r = row0 + k * 64 + lane;
            if (r < p.M) {
                const int64_t blk = r * p.nb + j;
                process_block(op, t.raw[k], p, blk, j);
            }
        }
    }
}

// element encode alone (checks of the device conversion)
__global__ __launch_bounds__(kThreads) void e2m1_kernel(const float* __restrict__ v, int64_t npairs,
                                                       uint32_t s, uint8_t* __restrict__ codes) {
    const float sc = __uint_as_float(s << 23);
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < npairs; i += stride) {
        const uint32_t c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, v[2 * i], v[2 * i + 1], sc, 0);
        codes[i] = (uint8_t)(c & 0xFFu);
    }
}

// ------------------------------------------------------------------ launchers
namespace {
int grid_for(int64_t units, int max_blocks) {
    const int64_t waves_per_block = kThreads / 64;
    int64_t g = (units + waves_per_block - 1) / waves_per_block;
    if (g > max_blocks) g = max_blocks;
    if (g < 1) g = 1;
    return (int)g;
}
}  // namespace

template <int U, class Op>
static hipError_t launch_flat(Params p, hipStream_t st, int max_blocks) {
    p.units = (p.nblocks + 64 * U - 1) / (64 * U);
    hipLaunchKernelGGL((flat_kernel<U, Op>), dim3(grid_for(p.units, max_blocks)), dim3(kThreads), 0, st, p);
    return hipGetLastError();
}

template <int U, class Op>
static hipError_t launch_column(Params p, hipStream_t st, int max_blocks) {
    const int64_t row_tiles = (p.M + 64 * U - 1) / (64 * U);
    p.units = row_tiles * p.nb;
    hipLaunchKernelGGL((column_kernel<U, Op>), dim3(grid_for(p.units, max_blocks)), dim3(kThreads), 0, st, p);
    return hipGetLastError();
}

template <class Op>
static hipError_t launch_op(const Params& p, Mapping map, hipStream_t st, const LaunchConfig& cfg) {
    if (map == Mapping::Flat) {
        if (cfg.blocks_per_lane == 2) return launch_flat<2, Op>(p, st, cfg.max_blocks);
        return launch_flat<1, Op>(p, st, cfg.max_blocks);
    }
    if (cfg.blocks_per_lane == 2) return launch_column<2, Op>(p, st, cfg.max_blocks);
    return launch_column<1, Op>(p, st, cfg.max_blocks);
}

hipError_t launch(Kind kind, int a, const Params& p, Mapping map, hipStream_t st, const LaunchConfig& cfg) {
    switch (kind) {
        case Kind::Plain: return launch_op<PlainOp>(p, map, st, cfg);
        case Kind::Smooth:
            if (map == Mapping::Flat) return launch_op<SmoothLaneOp>(p, map, st, cfg);
            return launch_op<SmoothUniformOp>(p, map, st, cfg);
        case Kind::Hadamard: return launch_op<HadamardOp>(p, map, st, cfg);
        case Kind::Kron:
            switch (a) {
                case 4: return launch_op<KronOp<4, 8>>(p, map, st, cfg);
                case 2: return launch_op<KronOp<2, 16>>(p, map, st, cfg);
                case 8: return launch_op<KronOp<8, 4>>(p, map, st, cfg);
                case 1: return launch_op<KronOp<1, 32>>(p, map, st, cfg);
                default: return hipErrorInvalidValue;
            }
    }
    return hipErrorInvalidValue;
}

hipError_t launch_e2m1(const float* v, int64_t npairs, uint32_t s, uint8_t* codes, hipStream_t st) {
    int64_t g = (npairs + kThreads - 1) / kThreads;
    if (g > 65536) g = 65536;
    if (g < 1) g = 1;
    hipLaunchKernelGGL(e2m1_kernel, dim3((unsigned)g), dim3(kThreads), 0, st, v, npairs, s, codes);
    return hipGetLastError();
}

}  // namespace kq
