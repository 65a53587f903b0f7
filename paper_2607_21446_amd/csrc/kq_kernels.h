// Internal interface between the C-ABI layer (kq_api.hip) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kq {

constexpr int kThreads = 256;  // 4 wave64 per workgroup

enum class Kind { Plain, Smooth, Hadamard, Kron };
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
    int64_t units;       // wave units, filled in by the launcher
};

struct LaunchConfig {
    int blocks_per_lane = 1;   // U: 32-element blocks a lane holds per wave unit
    int max_blocks = 1 << 20;  // cap on the workgroup count (grid-stride beyond it)
};

hipError_t launch(Kind kind, int a, const Params& p, Mapping map, hipStream_t st, const LaunchConfig& cfg);
hipError_t launch_e2m1(const float* v, int64_t npairs, uint32_t s, uint8_t* codes, hipStream_t st);

}  // namespace kq
