// W4A4 MXFP4 GEMM: the consumer of the quantizer's output (Sec. 3.1 eq. (1),
// Sec. 3.4): C[M, N] (+)= deq(Xq)[M, K] . deq(Wq)[N, K]^T, both operands in
// the MXFP4 layout the quantizer writes -- codes [rows, K/2] (element 2i in
// the low nibble of byte i) and E8M0 scales [rows, K/32] -- so activations
// from kq_quantize* and weights from kq_weight_transform feed it unchanged.
//
// Matrix cores: v_mfma_scale_f32_32x32x64_f8f6f4 with both operands E2M1.  In
// that instruction lane l supplies row (A) or column (B) l % 32 and the 32
// K-values 32 (l / 32) .. 32 (l / 32) + 31 of the 64-wide K step, 16 bytes,
// plus one E8M0 byte for them: exactly one 32-element block and its scale in
// the quantizer's layout, so fragments are plain 16-byte loads and no
// re-layout or pre-shuffle of codes or scales is needed.  Products of E2M1
// values times the two scales are exact in fp32; the sum over K is
// accumulated in fp32 (order not specified).
//
// Tiling: a 256-thread workgroup owns a 128 x 128 tile of C; its four waves
// own 64 x 64 quadrants, 2 x 2 instruction tiles of 32 x 32 each (four fp32
// accumulators).  Fragments are loaded straight from global memory (the
// workgroup's two waves per row/column quadrant share them through L1/L2),
// with the next K step's fragments in flight while the current step's four
// instructions run.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kq_kernels.h"

namespace kq {

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16g __attribute__((ext_vector_type(16)));

namespace {

// One lane's share of a K step: the 16 code bytes of one block (as the low
// half of the 8-dword operand; E2M1 uses 4 dwords) and its scale byte.
struct Frag {
    uint4 codes;
    uint32_t scale;
};

__device__ __forceinline__ Frag load_frag(const uint8_t* __restrict__ codes, const uint8_t* __restrict__ scales,
                                          int64_t row, int64_t nrows, int64_t kb, int64_t nkb, int64_t row_bytes) {
    Frag f;
    if (row < nrows && kb < nkb) {
        f.codes = *reinterpret_cast<const uint4*>(codes + row * row_bytes + kb * 16);
        f.scale = scales[row * nkb + kb];
    } else {
        f.codes = make_uint4(0u, 0u, 0u, 0u);  // zero codes contribute 0 whatever the scale
        f.scale = 127u;
    }
    return f;
}

__device__ __forceinline__ i32x8 operand(const Frag& f) {
    i32x8 v = {(int)f.codes.x, (int)f.codes.y, (int)f.codes.z, (int)f.codes.w, 0, 0, 0, 0};
    return v;
}

}  // namespace

__global__ __launch_bounds__(256) void mxfp4_gemm_kernel(const GemmParams g) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int r = lane & 31, h = lane >> 5;
    const int64_t m0 = (int64_t)blockIdx.y * 128 + (wave >> 1) * 64;
    const int64_t n0 = (int64_t)blockIdx.x * 128 + (wave & 1) * 64;
    const int64_t nkb = g.K / 32;                // 32-element blocks along K
    const int64_t row_bytes = g.K / 2;           // code bytes per row
    const int64_t nsteps = (nkb + 1) / 2;        // 64-wide K steps
    f32x16g acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16g{};
    Frag fa[2], fb[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        fa[i] = load_frag(g.a_codes, g.a_scales, m0 + 32 * i + r, g.M, h, nkb, row_bytes);
        fb[i] = load_frag(g.b_codes, g.b_scales, n0 + 32 * i + r, g.N, h, nkb, row_bytes);
    }
    for (int64_t s = 0; s < nsteps; ++s) {
        Frag na[2], nbf[2];
        const int64_t kb = 2 * (s + 1) + h;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            na[i] = load_frag(g.a_codes, g.a_scales, m0 + 32 * i + r, g.M, kb, nkb, row_bytes);
            nbf[i] = load_frag(g.b_codes, g.b_scales, n0 + 32 * i + r, g.N, kb, nkb, row_bytes);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                    operand(fa[i]), operand(fb[j]), acc[i][j], 4, 4, 0, (int)fa[i].scale, 0, (int)fb[j].scale);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            fa[i] = na[i];
            fb[i] = nbf[i];
        }
    }
    // acc[i][j][4q + e] = C[m0 + 32 i + 8 q + 4 h + e][n0 + 32 j + r]
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t col = n0 + 32 * j + r;
            if (col >= g.N) continue;
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int64_t row = m0 + 32 * i + 8 * q + 4 * h + e;
                    if (row >= g.M) continue;
                    float* dst = g.C + row * g.ldc_out + col;
                    *dst = g.accumulate ? *dst + acc[i][j][4 * q + e] : acc[i][j][4 * q + e];
                }
        }
}

hipError_t launch_mxfp4_gemm(const GemmParams& g, hipStream_t st) {
    const dim3 grid((unsigned)((g.N + 127) / 128), (unsigned)((g.M + 127) / 128));
    hipLaunchKernelGGL(mxfp4_gemm_kernel, grid, dim3(256), 0, st, g);
    return hipGetLastError();
}

}  // namespace kq
