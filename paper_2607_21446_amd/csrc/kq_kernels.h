// Internal interface between the C-ABI layer (kq_api.hip) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kq {

constexpr int kThreads = 256;  // workgroup size of the element-encode kernel
constexpr int64_t kPackBytes = 6 * 64 * 16 + 16;  // packed K per factor pair

enum class Kind { Plain, Smooth, Hadamard, Kron, KronMfma, KronLU };
enum class Mapping { Flat, Column };

// Everything a launch needs; sizes already validated by the caller.
struct Params {
    const uint16_t* X;   // [M, d] bf16 bits
    int64_t M;
    int64_t d;
    int64_t nb;          // d / 32
    int64_t nblocks;     // M * nb
    int64_t nfac;        // 1 or nb
    const float* A;      // [nfac, a, a]
    const float* B;      // [nfac, b, b]
    const float* mult;   // [d] SmoothQuant multipliers
    uint8_t* codes;      // [M, d/2] or null (then scales is null too)
    uint8_t* scales;     // [M, nb]
    float* y;            // [M, d] or null
    const uint8_t* kpack;  // [nfac, kPackBytes] materialised K terms, or null
    const float* lu;       // [nfac, 5, 3] LU parameters of G_1..G_5 (KronLU), or null
    uint16_t* y16;         // [M, d] bf16 of the transformed values, or null (KronLU)
    int64_t units;       // wave units, filled in by the launcher
};

// Launch shapes.
constexpr int64_t kMaxGridStride = int64_t(1) << 30;  // workgroup cap of the grid-stride kernels
constexpr int64_t kInterleaveMaxUnits = 4096;         // packed K: interleave both tiles up to this many units
constexpr int64_t kSmoothWaves = 2048;                // target workgroups of the column-stationary SmoothQuant
// Largest one-workgroup-per-unit grid (units of 64 blocks, or tiles of the
// per-block kernel): launches beyond it are refused by the API layer.
constexpr int64_t kMaxUnitGrid = (int64_t(1) << 31) - 1;

// W4A4 MXFP4 GEMM C[M, N] (+)= deq(A)[M, K] . deq(B)[N, K]^T (kq_gemm.hip).
struct GemmParams {
    const uint8_t* a_codes;   // [M, K/2]
    const uint8_t* a_scales;  // [M, K/32]
    int64_t M;
    const uint8_t* b_codes;   // [N, K/2]
    const uint8_t* b_scales;  // [N, K/32]
    int64_t N;
    int64_t K;                // multiple of 32
    float* C;                 // [M, ldc_out]
    int64_t ldc_out;
    int accumulate;           // 1: C += product, 0: C = product
    const float* bias = nullptr;  // if set: C = bias + product (bias [M, ldc_out], vec rule as C)
    uint16_t* C16 = nullptr;      // if set: bf16 output [M, ldc_out] instead of C (no bias, no accumulate)
    int vec_ok;               // C 16-byte (C16 8-byte) aligned and ldc_out a multiple of 4
    int scales_aligned;       // both scale arrays 4-byte aligned
};

hipError_t launch(Kind kind, int a, const Params& p, Mapping map, hipStream_t st);
hipError_t launch_mxfp4_gemm(const GemmParams& g, hipStream_t st);
hipError_t launch_pack(int a, const float* A, const float* B, int64_t nfac, uint8_t* kpack, hipStream_t st);
hipError_t launch_e2m1(const float* v, int64_t npairs, uint32_t s, uint8_t* codes, hipStream_t st);
hipError_t launch_fwht(const Params& p, hipStream_t st);  // d a power of two, 32 .. 16384
hipError_t launch_stream_floor(const Params& p, hipStream_t st);  // traffic of the quantizers, no arithmetic
// the same traffic in another launch shape: waves per workgroup (1, 2, 4, 8, 16), units per wave (1, 2, 4),
// groups > 0: that many workgroups in a grid-stride loop, else one pass
hipError_t launch_stream_probe(const Params& p, int waves, int units, int64_t groups, hipStream_t st);
hipError_t launch_timestamp(uint64_t* dst, hipStream_t st);  // the 100 MHz real-time counter into dst[0]

}  // namespace kq
