// KroQuant online activation quantizer: HIP kernels for gfx950 (MI355X).
//
// Two implementations of the Kronecker block transform y = (A (x) B) x
// (Sec. 3.2) feed the same MXFP4 encoder (Sec. 3.1: row-wise blocks of 32
// sharing one E8M0 scale):
//
//  * exact (VALU, quant_kernel): one lane owns one whole 32-element block.
//    The block's input, its 32 transformed fp32 values, its amax, scale and
//    16 code bytes stay in that lane's registers, and the separable product
//    is evaluated with fp32 FMAs in the fixed order below, so every output
//    is bit-identical to that order.  Factors are wave-uniform scalar loads.
//    12 FMAs per element make it bound by VALU issue, not by HBM.
//  * matrix-core (MFMA; kron_mfma_unit_kernel with K from the pack,
//    kron_build_unit_kernel with K built on chip, kron_tile_kernel for
//    per-block factors): the materialised 32x32 block
//    K = A (x) B, rounded to fp32 and split into three bf16 terms
//    (hi + mid + lo), multiplies 32 blocks at a time with
//    v_mfma_f32_32x32x16_bf16 (the bf16 input is the B operand as loaded),
//    accumulating in fp32 -- the "single 32x32 tensor-core GEMM per block"
//    of Sec. 3.5 done in enough precision for fp32 parity.  Its rounding
//    differs from the exact order by at most 116 u S, S = sum_k |K_nk||x_k|
//    (u = 2^-24), which can move a code only next to a rounding tie: the
//    fixed order is within (a + b) u S <= 33 u S of the exact product, the
//    rounded and split K within 2 u |K|, the bf16 products are exact, and the
//    accumulation rounds at most 16 times per instruction with relative error
//    <= 2 u each (nearest or truncating, any internal order), on partial sums
//    below S for the two hi-term instructions and below 2^-7 S for the other
//    four: <= 66 u S; 33 + 2 + 66 <= 116.  The E8M0 scale depends on amax only
//    through its binade; whenever a block's amax lies within 2^-17 ||K||_inf
//    max|x| of a power of two (128 u) that block is recomputed on the exact
//    path, so scales are always those of the exact order and each block's
//    outputs depend on that block alone.
//
// Two unit -> block mappings (a unit is the 64 blocks of one wave):
//   FLAT    the blocks of the matrix are one flat array (rows are contiguous);
//           unit u owns blocks 64u .. 64u+63.  Its stores are 1 KiB of codes
//           and 64 B of scales, both contiguous.  Used when every block has
//           the same factors.
//   COLUMN  unit u owns column block j = u % nb over 64 consecutive rows
//           (lane = row), so per-block factors K^(j) (T = diag(K^(1..d/32)),
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
// One wave per workgroup; a wave unit is 64 blocks (4 KiB of bf16 input).
// The unit's 256 16-byte chunks are read with four fully coalesced,
// nontemporal 1 KiB loads (instruction k, lane l -> chunk 64k + l), parked in
// LDS and read back so that lane l holds the 4 chunks of block l.  LDS slot of
// chunk m of block b: 4b + (m ^ ((b >> 2) & 3)); the XOR keeps both the
// chunk-order writes and the block-order reads free of bank conflicts.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_nt(const uint4* p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ int lds_slot(int b, int m) { return 4 * b + (m ^ ((b >> 2) & 3)); }

// make this wave's LDS writes visible to its own later reads (same wave,
// different lanes)
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// per-block body: transform, encode, store.  codes16 / scale / y32 point at
// this lane's block in the outputs.
template <class Op>
__device__ __forceinline__ void process_block(const Op& op, const uint4 (&raw)[4], const Params& p,
                                              uint8_t* codes16, uint8_t* scale, float* y32, int64_t col) {
    float x[32], y[32];
#pragma unroll
    for (int m = 0; m < 4; ++m) unpack8(raw[m], x + 8 * m);
    op.apply(x, y, col);
    uint32_t w[4];
    const uint32_t s = encode32(y, w);
    if (p.codes) {
        *reinterpret_cast<uint4*>(codes16) = make_uint4(w[0], w[1], w[2], w[3]);
        *scale = (uint8_t)s;
    }
    if (p.y) {
        float4* dst = reinterpret_cast<float4*>(y32);
#pragma unroll
        for (int m = 0; m < 8; ++m)
            dst[m] = make_float4(y[4 * m], y[4 * m + 1], y[4 * m + 2], y[4 * m + 3]);
    }
}

// FLAT: unit u = blocks 64u .. 64u+63 of the flat block array.
// COLUMN: unit u = column block j = u % nb of rows 64*(u / nb) .. +63.
// Addresses: a wave-uniform unit base plus a 32-bit lane offset (a unit spans
// 64 rows at most, so lane offsets stay below 2^31 for any d < 2^24).
template <Mapping MAP, class Op>
__global__ __launch_bounds__(64) void quant_kernel(const Params p) {
    __shared__ uint4 lds[256];
    const int lane = threadIdx.x;
    for (int64_t u = blockIdx.x; u < p.units; u += gridDim.x) {
        int64_t j = 0, row0 = 0, first;  // first: flat index of the unit's block 0
        int nvalid;                       // blocks of the unit inside the matrix
        uint32_t bstride;                 // flat-block distance between the unit's blocks
        if (MAP == Mapping::Flat) {
            first = u * 64;
            nvalid = (int)min<int64_t>(64, p.nblocks - first);
            bstride = 1;
        } else {
            j = u % p.nb;
            row0 = (u / p.nb) * 64;
            first = row0 * p.nb + j;
            nvalid = (int)min<int64_t>(64, p.M - row0);
            bstride = (uint32_t)p.nb;
        }
        const uint4* src = reinterpret_cast<const uint4*>(p.X) + first * 4;
        uint4 v[4];
        if (nvalid == 64) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t ci = 64 * k + lane;
                v[k] = load_nt(src + ((ci >> 2) * bstride * 4 + (ci & 3)));
            }
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t ci = 64 * k + lane;
                v[k] = make_uint4(0u, 0u, 0u, 0u);
                if ((int)(ci >> 2) < nvalid) v[k] = load_nt(src + ((ci >> 2) * bstride * 4 + (ci & 3)));
            }
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int ci = 64 * k + lane;
            lds[lds_slot(ci >> 2, ci & 3)] = v[k];
        }
        wave_lds_sync();
        uint4 raw[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) raw[m] = lds[lds_slot(lane, m)];
        wave_lds_sync();  // the next unit's writes come after these reads
        if (lane < nvalid) {
            Op op;
            op.setup(p, j);
            const uint32_t lo = (uint32_t)lane * bstride;  // this lane's block, relative to `first`
            const int64_t col = (MAP == Mapping::Flat) ? (first + lane) % p.nb : j;
            process_block(op, raw, p, p.codes + first * 16 + (uint64_t)lo * 16, p.scales + first + lo,
                          p.y + first * 32 + (uint64_t)lo * 32, col);
        }
    }
}

// ------------------------------------------------------------------ matrix-core path
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// Codes of the 8 values a[o .. o+7] at scale sc as one dword (value o + 2i in
// the low nibble of byte i).  `old` only seeds the register: every byte is
// overwritten.
__device__ __forceinline__ uint32_t codes8(const f32x16& a, int o, float sc, uint32_t old) {
    uint32_t c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a[o], a[o + 1], sc, 0);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, a[o + 2], a[o + 3], sc, 1);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, a[o + 4], a[o + 5], sc, 2);
    return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, a[o + 6], a[o + 7], sc, 3);
}

// Two fp32 values as a bf16 pair (round to nearest even), the first in the low half.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16_pair(float a, float b) {
    const bf16x2 v = {(__bf16)a, (__bf16)b};
    return __builtin_bit_cast(uint32_t, v);
}

// The value `v` of lane l ^ 32 (the other half of the wave).
__device__ __forceinline__ uint32_t other_half(uint32_t v) {
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return (threadIdx.x & 32) ? r[0] : r[1];
}
__device__ __forceinline__ float other_half(float v) { return __uint_as_float(other_half(__float_as_uint(v))); }

// max(v, v of lane l ^ 32) for v >= 0 as fp32 bit patterns: after the swap one
// of the pair holds this lane's value and the other its partner's, in either
// half, so their max needs no lane select.
__device__ __forceinline__ uint32_t max_with_other_half(uint32_t v) {
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return max((uint32_t)r[0], (uint32_t)r[1]);
}

// The value of lane l ^ 1 (a DPP quad permutation, no LDS round trip).
__device__ __forceinline__ uint32_t lane_xor1(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
}

// Unsigned max over each 32-lane half of the wave (for values >= 0 this is the
// max of their fp32 bit patterns): DPP steps within rows of 16 lanes (lane ^ 1,
// lane ^ 2, mirror in 8, mirror in 16), then rows 2k and 2k + 1 swapped.
__device__ __forceinline__ uint32_t half_wave_max(uint32_t v) {
    v = max(v, lane_xor1(v));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return max((uint32_t)r[0], (uint32_t)r[1]);
}

// This lane's slice of K = A (x) B as the A operand of v_mfma_f32_32x32x16_bf16:
// lane l holds K[perm_row(m)][k] for m = l % 32 and k = 16 s + 8 (l / 32) + c
// (c = 0..7) in k-step s = 0, 1; K[n][k] = fp32(A[n / b][k / b] * B[n % b][k % b])
// (numpy.kron index order), split as hi + mid + lo with each term the bf16
// nearest to what the previous terms leave.
struct KSlices {
    bf16x8 hi[2], mid[2], lo[2];
};

// Output row m of the 32x32 product is block element perm_row(m).  The
// product's lane layout puts rows 8q + 4h + r (q, r = 0..3) in acc[4q + r] of
// lane 32h + block, so with this order lane 32h + block holds elements
// 16h .. 16h + 15 in acc[0..15]: its 8 code bytes are contiguous and need no
// exchange with the other half of the wave.
__device__ __forceinline__ constexpr int perm_row(int m) { return 16 * ((m >> 2) & 1) + 4 * (m >> 3) + (m & 3); }

// The factor entries behind this lane's slice: kv(s, c) = fa[s][c] * fb[s][c].
template <int NA, int NB>
struct KFactors {
    float fa[2][8], fb[2][8];
};

template <int NA, int NB>
__device__ __forceinline__ void load_k_factors(const float* A, const float* B, int lane, KFactors<NA, NB>& kf) {
    const int n = perm_row(lane & 31), h = lane >> 5;
    const int ia = n / NB, ib = n % NB;
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const int k = 16 * s + 8 * h + c;
            kf.fa[s][c] = A[ia * NA + k / NB];
            kf.fb[s][c] = B[ib * NB + k % NB];
        }
}

// Split the slice into bf16 terms; returns ||K||_inf.
template <int NA, int NB>
__device__ __forceinline__ float build_k(const KFactors<NA, NB>& kf, KSlices& ks) {
    float rowsum = 0.0f;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const float kv = kf.fa[s][c] * kf.fb[s][c];
            rowsum += fabsf(kv);
            const __bf16 t1 = (__bf16)kv;
            const float r1 = kv - (float)t1;  // exact
            const __bf16 t2 = (__bf16)r1;
            const float r2 = r1 - (float)t2;  // exact
            ks.hi[s][c] = t1;
            ks.mid[s][c] = t2;
            ks.lo[s][c] = (__bf16)r2;
        }
    }
    // row n is split over lanes n and n + 32; then the max over the 32 rows
    // (sums are >= 0, so their fp32 bit patterns order like the values)
    uint32_t r = __float_as_uint(rowsum + other_half(rowsum));
#pragma unroll
    for (int off = 16; off >= 1; off >>= 1) r = max(r, (uint32_t)__shfl_xor((int)r, off));
    return __uint_as_float(r);
}

// max |x| of the 16 bf16 values in two chunks, as fp32
__device__ __forceinline__ float max_abs_bf16(const uint4 (&r)[2]) {
    u16x2 m = {0, 0};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const uint32_t w[4] = {r[s].x, r[s].y, r[s].z, r[s].w};
#pragma unroll
        for (int i = 0; i < 4; ++i)
            m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, w[i] & 0x7FFF7FFFu));
    }
    const uint32_t top = m[0] > m[1] ? m[0] : m[1];
    return __uint_as_float(top << 16);
}

// SmoothQuant, column-stationary: the grid stride G (in 64-block units) is a
// multiple of nb / gcd(nb, 64), so 64 G is a multiple of nb and lane l of a
// workgroup keeps the same column block (64 u + l) mod nb in every unit it
// handles.  Its 32 multipliers are loaded once; the next unit's input loads
// are issued before the current unit is encoded.
__global__ __launch_bounds__(64) void smooth_stationary_kernel(const Params p) {
    __shared__ uint4 lds[256];
    const int lane = threadIdx.x;
    const int64_t u0 = blockIdx.x, ustep = gridDim.x;
    if (u0 >= p.units) return;
    const int64_t col = (u0 * 64 + lane) % p.nb;
    float mul[32];
    {
        const float4* mv = reinterpret_cast<const float4*>(p.mult + col * 32);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const float4 f = mv[k];
            mul[4 * k] = f.x;
            mul[4 * k + 1] = f.y;
            mul[4 * k + 2] = f.z;
            mul[4 * k + 3] = f.w;
        }
    }
    uint4 v[4];
    auto issue = [&](int64_t u) {
        const int64_t first = u * 64;
        const int nvalid = (int)min<int64_t>(64, p.nblocks - first);
        const uint4* src = reinterpret_cast<const uint4*>(p.X) + first * 4;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int ci = 64 * c + lane;
            v[c] = make_uint4(0u, 0u, 0u, 0u);
            if ((ci >> 2) < nvalid) v[c] = load_nt(src + ci);
        }
    };
    issue(u0);
    for (int64_t u = u0; u < p.units; u += ustep) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int ci = 64 * c + lane;
            lds[lds_slot(ci >> 2, ci & 3)] = v[c];
        }
        if (u + ustep < p.units) issue(u + ustep);
        wave_lds_sync();
        uint4 raw[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) raw[m] = lds[lds_slot(lane, m)];
        wave_lds_sync();
        const int64_t blk = u * 64 + lane;
        if (blk < p.nblocks) {
            float x[32], y[32];
#pragma unroll
            for (int m = 0; m < 4; ++m) unpack8(raw[m], x + 8 * m);
#pragma unroll
            for (int k = 0; k < 32; ++k) y[k] = x[k] * mul[k];
            uint32_t w[4];
            const uint32_t sb = encode32(y, w);
            if (p.codes) {
                *reinterpret_cast<uint4*>(p.codes + blk * 16) = make_uint4(w[0], w[1], w[2], w[3]);
                p.scales[blk] = (uint8_t)sb;
            }
            if (p.y) {
                float4* dst = reinterpret_cast<float4*>(p.y + blk * 32);
#pragma unroll
                for (int m = 0; m < 8; ++m)
                    dst[m] = make_float4(y[4 * m], y[4 * m + 1], y[4 * m + 2], y[4 * m + 3]);
            }
        }
    }
}

// Exact fixed-order evaluation of up to two blocks by 32 cooperating lanes
// each: half-wave h takes block blk[h] (skipped if negative); lane n
// (n = lane % 32) evaluates output y[n] = Y[o][i], n = o*b + i, with the FMA
// chains of KronOp:
//   Z[p][i] = B[i][0]*x[p*b] then fma(B[i][q], x[p*b+q], .), q = 1..b-1,
//   Y[o][i] = A[o][0]*Z[0][i] then fma(A[o][p], Z[p][i], .), p = 1..a-1.
// Called with all 64 lanes active; the blocks lie in this wave's LDS unit
// (GX: the inputs are read from X at the output blocks, unit_lds unused).
template <int NA, int NB, bool GX = false>
__device__ __forceinline__ void exact_blocks_coop(const uint4* unit_lds, int blk0, int blk1, const float* Af,
                                                  const float* Bf, const Params& p, int64_t out0, int64_t out1) {
    const int h = (threadIdx.x >> 5) & 1;  // half of this wave (workgroups may hold several waves)
    const int n = threadIdx.x & 31;
    const int o = n / NB, i = n % NB;
    const int blk = h ? blk1 : blk0;
    const int64_t out_blk = h ? out1 : out0;
    float x[32];
    if (GX) {
        const uint4* const xs = reinterpret_cast<const uint4*>(p.X) + (blk < 0 ? out0 : out_blk) * 4;
#pragma unroll
        for (int m = 0; m < 4; ++m) unpack8(xs[m], x + 8 * m);
    } else {
#pragma unroll
        for (int m = 0; m < 4; ++m) unpack8(unit_lds[lds_slot(blk < 0 ? 0 : blk, m)], x + 8 * m);
    }
    float acc = 0.0f;
#pragma unroll
    for (int pr = 0; pr < NA; ++pr) {
        float z = Bf[i * NB] * x[pr * NB];
#pragma unroll
        for (int q = 1; q < NB; ++q) z = __builtin_fmaf(Bf[i * NB + q], x[pr * NB + q], z);
        acc = (pr == 0) ? Af[o * NA] * z : __builtin_fmaf(Af[o * NA + pr], z, acc);
    }
    const uint32_t sb = e8m0_byte(__uint_as_float(half_wave_max(__float_as_uint(fabsf(acc)))));
    const float next = __uint_as_float(lane_xor1(__float_as_uint(acc)));  // y[n + 1] for even n
    const uint32_t c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, acc, next, __uint_as_float(sb << 23), 0);
    if (blk >= 0) {
        if (p.codes) {
            if ((n & 1) == 0) p.codes[out_blk * 16 + (n >> 1)] = (uint8_t)(c & 0xFFu);
            if (n == 0) p.scales[out_blk] = (uint8_t)sb;
        }
        if (p.y) p.y[out_blk * 32 + n] = acc;
        if (p.y16) p.y16[out_blk * 32 + n] = (uint16_t)(bf16_pair(acc, 0.0f) & 0xFFFFu);
    }
}

// all blocks flagged in `edges` (bit b = block b of the unit), two at a time
// (GX: their inputs read from X instead of the unit in LDS)
template <int NA, int NB, bool GX = false>
__device__ __forceinline__ void exact_flagged(uint64_t edges, const uint4* unit_lds, int64_t first, uint32_t bstride,
                                              const float* Af, const float* Bf, const Params& p) {
    while (edges) {
        const int b0 = __builtin_ctzll(edges);
        edges &= edges - 1;
        int b1 = -1;
        if (edges) {
            b1 = __builtin_ctzll(edges);
            edges &= edges - 1;
        }
        exact_blocks_coop<NA, NB, GX>(unit_lds, b0, b1, Af, Bf, p, first + (int64_t)b0 * bstride,
                                      first + (int64_t)(b1 < 0 ? 0 : b1) * bstride);
    }
}

// K2-form factors from the LU parameters of G_1..G_5 (Sec. 3.2, Sec. 3.5):
// G = [[a, b], [c a, c b - 1/a]] and, with na = log2(NA),
//   A[o][p] = prod_{k < na}  G_k[bit(p, na-1-k)][bit(o, na-1-k)],
//   B[i][q] = prod_{k >= na} G_k[bit(q, 4-k)][bit(i, 4-k)],
// so A (x) B = (G_1 (x) ... (x) G_5)^T; every product left to right, one fp32
// rounding per multiply, g11 = fma(c, b, -(1/a)).
// The 15 parameters of a pair as wave-uniform values (scalar loads).
__device__ __forceinline__ void lu_load(const float* lu, float (&pv)[15]) {
#pragma unroll
    for (int i = 0; i < 15; ++i) pv[i] = ld_uniform(lu, i);
}

// The 2x2 factors G_k = [[g0, g1], [g2, g3]] from the parameters.
__device__ __forceinline__ void lu_g(const float (&pv)[15], float (&g)[5][4]) {
#pragma unroll
    for (int k = 0; k < 5; ++k) {
        const float pa = pv[3 * k], pb = pv[3 * k + 1], pc = pv[3 * k + 2];
        g[k][0] = pa;
        g[k][1] = pb;
        g[k][2] = pc * pa;
        g[k][3] = __builtin_fmaf(pc, pb, -(1.0f / pa));
    }
}

// Entry idx of A then B (idx < NA*NA + NB*NB), branch-free: factors outside
// the entry's group multiply as exactly 1, so the product is the left-to-right
// product of the entry's own G entries.
template <int NA, int NB>
__device__ __forceinline__ float lu_entry(const float (&g)[5][4], int idx) {
    constexpr int na = NA == 1 ? 0 : NA == 2 ? 1 : NA == 4 ? 2 : 3;
    const bool in_a = idx < NA * NA;
    const int rowi = in_a ? idx / NA : (idx - NA * NA) / NB;  // o or i
    const int coli = in_a ? idx % NA : (idx - NA * NA) % NB;  // p or q
    float v = 1.0f;
#pragma unroll
    for (int k = 0; k < 5; ++k) {
        const int sh = k < na ? na - 1 - k : 4 - k;
        const int e = 2 * ((coli >> sh) & 1) + ((rowi >> sh) & 1);  // G_k[bit of col][bit of row]
        const float ge = e == 0 ? g[k][0] : e == 1 ? g[k][1] : e == 2 ? g[k][2] : g[k][3];
        v *= ((k < na) == in_a) ? ge : 1.0f;
    }
    return v;
}

// Workgroups go to the 8 XCDs round robin (workgroup i to XCD i % 8).  This
// gives XCD x the contiguous workgroup range [x q + min(x, r), ...) of a grid
// of G = 8 q + r (a bijection of [0, G)).  Used by the COLUMN mapping, where
// neighbouring workgroups hold neighbouring 32-column blocks of the same
// rows: their 64-byte input pieces share cache lines, and so do their code
// and scale writes, which then all go through one L2.
__device__ __forceinline__ int64_t xcd_order(int64_t i, int64_t G) {
    const int64_t q = G >> 3, r = G & 7, x = i & 7;
    return x * q + (x < r ? x : r) + (i >> 3);
}

// Input loads of one 64-block unit (four nontemporal 1 KiB loads, chunk
// 64 c + lane in v[c]); FULL = all 64 blocks present.  A partial unit
// (0 <= nvalid < 64) issues the same four loads, each lane at a clamped
// in-bounds address, and zeroes the chunks of missing blocks, so every path
// has exactly four loads in flight (later waits can then count them).
template <Mapping MAP, bool FULL>
__device__ __forceinline__ void load_unit(const Params& p, int64_t first, int nvalid, uint32_t bstride, uint4 (&v)[4]) {
    const int lane = threadIdx.x & 63;
    const uint4* src = reinterpret_cast<const uint4*>(p.X) + (FULL || nvalid > 0 ? first * 4 : 0);
    const uint32_t last = FULL ? 63u : (uint32_t)max(nvalid, 1) - 1u;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const uint32_t ci = 64 * c + lane;
        const uint32_t b = FULL ? (ci >> 2) : min(ci >> 2, last);
        const uint32_t off = MAP == Mapping::Flat ? (FULL ? ci : 4 * b + (ci & 3)) : b * bstride * 4 + (ci & 3);
        const uint4 t = load_nt(src + off);
        v[c] = (FULL || (int)(ci >> 2) < nvalid) ? t : make_uint4(0u, 0u, 0u, 0u);
    }
}

// The same four loads for a unit of any size, with no branch and no select:
// lanes of missing blocks read the unit's last present block (or block 0 of
// X when the unit is empty); unit_compute zeroes them when it stages the
// chunks.  Straight-line, so that a later wait for an older load can count
// these four as still in flight.
template <Mapping MAP>
__device__ __forceinline__ void load_unit_clamped(const Params& p, int64_t first, int nvalid, uint32_t bstride,
                                                  uint4 (&v)[4]) {
    const int lane = threadIdx.x & 63;
    const uint4* src = reinterpret_cast<const uint4*>(p.X) + (nvalid > 0 ? first * 4 : 0);
    const uint32_t last = (uint32_t)max(nvalid, 1) - 1u;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const uint32_t ci = 64 * c + lane;
        const uint32_t b = min(ci >> 2, last);
        const uint32_t off = MAP == Mapping::Flat ? 4 * b + (ci & 3) : b * bstride * 4 + (ci & 3);
        v[c] = load_nt(src + off);
    }
}

// How a unit decides which blocks lie on a binade edge (see the kernels below).
struct EdgeTest {
    uint32_t edge_t;  // PACKED: mantissa window T from the pack
    float kbound;     // otherwise: 2^-17 ||K||_inf (per-block window kbound * max|x|)
};

// The compute of one unit once its chunks are in v and the K slices in ks:
// both 32-block tiles through LDS, multiplied, encoded and stored (codes and
// scales last), binade-edge blocks re-evaluated in the fixed order.  FULL =
// all 64 blocks present (no per-tile bounds tests in the straight-line
// code); WY / WY16 = the fp32 / bf16 transformed values are stored too;
// PACKED selects the edge test.  lds = this wave's 256-slot staging area;
// Af, Bf = the factors (for the fixed-order fallback).  TILE: the workgroup
// has already staged the unit in lds (v is not used); the codes and scales of
// the blocks to store go to ts.out (the 16 code bytes of block b at slot b,
// its scale at byte 1024 + b) for the workgroup's row stores, which store the
// blocks whose bit is set in *ts.mask; the binade-edge blocks go to *ts.edges
// for the caller's fixed-order pass.
struct TileSink {
    uint4* out;
    uint64_t* mask;
    uint64_t* edges;
};

template <Mapping MAP, int NA, int NB, bool ILV, bool WY, bool WY16, bool FULL, bool PACKED, bool TILE = false>
__device__ __forceinline__ void unit_compute(const Params& p, uint4* lds, int64_t first, int nvalid_rt,
                                             uint32_t bstride, const uint4 (&v)[4], const KSlices& ks, bool zero_ok,
                                             EdgeTest et, const float* Af, const float* Bf, TileSink ts = {}) {
    const int lane = threadIdx.x & 63;
    const int h = lane >> 5, jl = lane & 31;
    const int nvalid = FULL ? 64 : nvalid_rt;
    // chunk 64c + lane of the unit (block (64c + lane) / 4, chunk (64c + lane) % 4
    // of that block) goes to LDS slot 64c + wslot (lds_slot is additive in c here)
    const int wslot = lds_slot(lane >> 2, lane & 3);
    // output bases of the unit (wave-uniform) and this lane's block offsets
    uint8_t* const codes_u = p.codes + first * 16;
    uint8_t* const scales_u = p.scales + first;
    float* const y_u = WY ? p.y + first * 32 : nullptr;
    uint16_t* const y16_u = WY16 ? p.y16 + first * 32 : nullptr;
    // every chunk goes to LDS as soon as it arrives (those of missing blocks as zeros)
    if (!TILE) {
        if (FULL || nvalid == 64) {
#pragma unroll
            for (int c = 0; c < 4; ++c) lds[wslot + 64 * c] = v[c];
        } else {
            // a partial unit (uniform branch): the chunks of missing blocks as zeros, branch-free
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t m = (64 * c + lane) / 4 < nvalid ? ~0u : 0u;
                lds[wslot + 64 * c] = make_uint4(v[c].x & m, v[c].y & m, v[c].z & m, v[c].w & m);
            }
        }
    }
    // lane (jl, h) reads chunks h and 2 + h of block 32 t + jl: slots 128 t + rslot
    // and 128 t + (rslot ^ 2)
    const int rslot = 4 * jl + (h ^ ((jl >> 2) & 3));
    if (!TILE) wave_lds_sync();
    uint4 raw[2][2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        raw[t][0] = lds[128 * t + rslot];
        raw[t][1] = lds[128 * t + (rslot ^ 2)];
    }
    uint64_t edges = 0;  // blocks of the unit on a binade edge (bit = block index)
    // the three terms, smallest first, of tile t: acc[n][block] += K[n][k-step] . x[block][k-step]
    auto product = [&](const uint4 (&r)[2]) {
        f32x16 acc = {};
#pragma unroll
        for (int s = 0; s < 2; ++s)
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ks.lo[s], __builtin_bit_cast(bf16x8, r[s]), acc, 0, 0, 0);
#pragma unroll
        for (int s = 0; s < 2; ++s)
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ks.mid[s], __builtin_bit_cast(bf16x8, r[s]), acc, 0, 0, 0);
#pragma unroll
        for (int s = 0; s < 2; ++s)
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ks.hi[s], __builtin_bit_cast(bf16x8, r[s]), acc, 0, 0, 0);
        return acc;
    };
    // amax, binade-edge flag, scale and codes of tile t (its y is stored at
    // once); the code and scale stores of both tiles come after both products
    struct TileOut {
        uint2 codes;
        uint32_t sb;
        bool store;
    };
    auto finish = [&](int t, const f32x16& acc, const uint4 (&r)[2]) {
        const int bt = 32 * t + jl;
        const bool valid = FULL || bt < nvalid;
        // lane holds y[16h + i] of block bt in acc[i]; values >= 0 compare as their bit patterns
        float am = 0.0f;
#pragma unroll
        for (int i = 0; i < 16; ++i) am = fmaxf(am, fabsf(acc[i]));
        const uint32_t amb = max_with_other_half(__float_as_uint(am));
        bool near;
        if (PACKED) {
            near = valid && (((amb + et.edge_t) & 0x7FFFFFu) <= 2u * et.edge_t || amb < (4u << 23));
        } else {
            // window kbound * max|x| around both powers of two that bracket amax
            const float bnd = et.kbound * __uint_as_float(max_with_other_half(__float_as_uint(max_abs_bf16(r))));
            const uint32_t e = amb >> 23;
            const float a = __uint_as_float(amb);
            near = valid && (e <= 3u || a - __uint_as_float(e << 23) <= bnd || __uint_as_float((e + 1u) << 23) - a <= bnd);
        }
        if (amb == 0u && zero_ok) {
            // all outputs +-0: exact when the inputs are all +0 (bit patterns 0)
            const uint32_t any = r[0].x | r[0].y | r[0].z | r[0].w | r[1].x | r[1].y | r[1].z | r[1].w;
            if ((any | other_half(any)) == 0u) near = false;
        }
        TileOut o;
        o.sb = max(amb >> 23, 2u) - 2u;
        const float sc = __uint_as_float(o.sb << 23);
        o.codes = make_uint2(codes8(acc, 0, sc, amb), codes8(acc, 8, sc, amb));
        o.store = valid && !near;
        if (WY && o.store) {
            float* yb = y_u + ((uint32_t)bt * bstride * 32u + 16u * h);
#pragma unroll
            for (int q = 0; q < 4; ++q)
                *reinterpret_cast<float4*>(yb + 4 * q) =
                    make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
        }
        if (WY16 && o.store) {
            uint4* yb = reinterpret_cast<uint4*>(y16_u + ((uint32_t)bt * bstride * 32u + 16u * h));
#pragma unroll
            for (int q = 0; q < 2; ++q)
                yb[q] = make_uint4(bf16_pair(acc[8 * q], acc[8 * q + 1]), bf16_pair(acc[8 * q + 2], acc[8 * q + 3]),
                                   bf16_pair(acc[8 * q + 4], acc[8 * q + 5]), bf16_pair(acc[8 * q + 6], acc[8 * q + 7]));
        }
        edges |= (__builtin_amdgcn_ballot_w64(near) & 0xFFFFFFFFull) << (32 * t);
        return o;
    };
    auto store = [&](int t, const TileOut& o) {
        const uint32_t ob = (uint32_t)(32 * t + jl) * bstride;  // this lane's block, relative to `first`
        if (o.store) {
            *reinterpret_cast<uint2*>(codes_u + (ob * 16u + 8u * h)) = o.codes;
            if (h == 0) scales_u[ob] = (uint8_t)o.sb;
        }
    };
    if (ILV && nvalid > 32) {
        // both tiles' products first (two accumulators): the second chain runs
        // on the matrix cores while the first tile's epilogue is on the VALU
        const f32x16 acc0 = product(raw[0]);
        const f32x16 acc1 = product(raw[1]);
        const TileOut o0 = finish(0, acc0, raw[0]);
        const TileOut o1 = finish(1, acc1, raw[1]);
        store(0, o0);
        store(1, o1);
    } else {
        // straight-line for full and partial units alike: a partial unit's
        // missing blocks hold zeros and are neither stored nor flagged
        // TILE: each tile's codes and scales go to ts.out as soon as they
        // exist (all blocks; the mask decides which are stored), so that the
        // first tile's accumulators are dead before the second product
        uint8_t* const ob = reinterpret_cast<uint8_t*>(ts.out);
        auto tile_write = [&](int t, const TileOut& o) {
            const int b = 32 * t + jl;
            *reinterpret_cast<uint2*>(ob + 16 * b + 8 * h) = o.codes;
            if (h == 0) ob[1024 + b] = (uint8_t)o.sb;
        };
        const TileOut o0 = finish(0, product(raw[0]), raw[0]);
        if (TILE) tile_write(0, o0);
        __builtin_amdgcn_sched_barrier(0);
        const TileOut o1 = finish(1, product(raw[1]), raw[1]);
        if (TILE) tile_write(1, o1);
        __builtin_amdgcn_sched_barrier(0);
        if (TILE) {
            const uint64_t m = (__builtin_amdgcn_ballot_w64(o0.store) & 0xFFFFFFFFull) |
                               (__builtin_amdgcn_ballot_w64(o1.store) << 32);
            if (lane == 0) {
                *ts.mask = m;
                *ts.edges = edges;
            }
            return;
        }
        store(0, o0);
        store(1, o1);
    }
    // blocks whose amax is on a binade edge: the fixed evaluation order decides
    exact_flagged<NA, NB>(edges, lds, first, bstride, Af, Bf, p);
}

// K slices and edge data of factor pair f from the pack (kq_pack_factors),
// issued after the unit's input loads.
__device__ __forceinline__ void packed_k(const Params& p, int64_t f, KSlices& ks, bool& zero_ok, EdgeTest& et) {
    const int lane = threadIdx.x & 63;
    // K slice i (i = 2 term + k-step) of this lane at byte 1024 i + 16 lane of the
    // pack: one uniform base 2 KiB in, so every offset fits the load's immediate
    const uint8_t* const pk0 = p.kpack + f * kPackBytes;
    const uint8_t* const pkm = pk0 + 2048;
    const uint32_t lo16 = 16u * (uint32_t)lane;
    auto kslice = [&](int i) {
        return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(pkm + lo16 + (1024 * i - 2048)));
    };
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        ks.hi[s] = kslice(0 * 2 + s);
        ks.mid[s] = kslice(1 * 2 + s);
        ks.lo[s] = kslice(2 * 2 + s);
    }
    const float* hdr = reinterpret_cast<const float*>(pk0 + 6 * 64 * 16);
    // nonzero when no row of A and no row of B has every sign bit set: then an
    // all-(+0) input block gives +0 for every output in the fixed order
    zero_ok = __float_as_uint(ld_uniform(hdr, 2)) != 0u;
    et.edge_t = __float_as_uint(ld_uniform(hdr, 3));
    et.kbound = 0.0f;
}

template <Mapping MAP, int NA, int NB, bool ILV, bool WY, bool FULL>
__device__ __forceinline__ void packed_unit(const Params& p, uint4* lds, int64_t jcol, int64_t first, int nvalid,
                                            uint32_t bstride) {
    uint4 v[4];
    load_unit<MAP, FULL>(p, first, nvalid, bstride, v);
    // the input loads leave first; the K slices (L2-resident) follow them
    __builtin_amdgcn_sched_barrier(0);
    const int64_t f = (p.nfac == 1) ? 0 : jcol;
    KSlices ks;
    bool zero_ok;
    EdgeTest et;
    packed_k(p, f, ks, zero_ok, et);
    unit_compute<MAP, NA, NB, ILV, WY, false, FULL, true>(p, lds, first, nvalid, bstride, v, ks, zero_ok, et,
                                                          p.A + f * (NA * NA), p.B + f * (NB * NB));
}

// Matrix-core KroQuant with K read from the pack, one 64-block unit per wave
// (no loop): few live registers, so every wave of a large grid is resident
// at once and all input loads are in flight from the start.  FLAT: unit =
// blockIdx.x;  COLUMN: with u = blockIdx.x in the XCD-contiguous order,
// column block j = u % nb, rows 64 * (u / nb).
// Per wave: the four input loads are issued first, then the K slices; all
// four chunks go through LDS; both 32-block tiles are multiplied and encoded
// back to back and their code and scale stores issued last.
//
// Binade-edge test.  With e the error of this path and of the fixed order
// (|e| <= 116 u sum_k |K_nk||x_k| <= 116 u ||K||_inf max|x|, u = 2^-24) and
// max|x| <= ||K^-1||_inf max|Kx| <= ||K^-1||_inf (amax + |e|), the two amax
// differ by at most 116 u cond (1 - 104 u cond)^-1 amax <= 2^-17 cond amax =
// rho amax whenever cond = cond_inf(K) <= 2^13.  amax = (1 + f) 2^E with
// f = mantissa / 2^23, so amax - 2^E <= rho amax implies f <= 2 rho and
// 2^(E+1) - amax <= rho amax implies 1 - f <= 2 rho: a block is re-evaluated in
// the fixed order when its amax mantissa lies within T = ceil(2^24 rho) of 0 or
// of 2^23 (T from the pack; T = 2^22 flags every block, used above cond 2^13),
// or when amax < 2^-123, so its E8M0 scale equals the fixed-order one.
template <Mapping MAP, int NA, int NB, bool ILV, bool WY>
__global__ __launch_bounds__(64) void kron_mfma_unit_kernel(const Params p) {
    __shared__ uint4 lds[256];
    const int64_t u = blockIdx.x;
    int64_t jcol = 0, first;
    int nvalid;
    uint32_t bstride;
    if (MAP == Mapping::Flat) {
        first = u * 64;
        nvalid = (int)min<int64_t>(64, p.nblocks - first);
        bstride = 1;
    } else {
        const int64_t g = xcd_order(u, gridDim.x);
        jcol = g % p.nb;
        const int64_t row0 = (g / p.nb) * 64;
        first = row0 * p.nb + jcol;
        nvalid = (int)min<int64_t>(64, p.M - row0);
        bstride = (uint32_t)p.nb;
    }
    if (nvalid == 64)
        packed_unit<MAP, NA, NB, ILV, WY, true>(p, lds, jcol, first, 64, bstride);
    else
        packed_unit<MAP, NA, NB, ILV, WY, false>(p, lds, jcol, first, nvalid, bstride);
}

// Matrix-core KroQuant with K built on chip from the factors (kq_quantize)
// or from the 15 LU parameters of G_1..G_5 (kq_quantize_lu): four waves per
// workgroup, one 64-block unit each, all four sharing one factor pair.  Every
// wave issues its input loads first; while they are in flight the workgroup
// stages A and B in LDS (or decodes them, LU), builds the split K once (wave w
// builds k-step w / 2, entries 4 (w % 2) .. 4 (w % 2) + 3 of every lane's
// slice), and wave 0 computes ||A||_inf ||B||_inf and the all-(+0) flag; LDS
// fences and bare barriers separate the phases so that no wait covers the
// input loads.  Then each wave runs the unit as in the packed kernel, with
// the binade-edge window 2^-17 ||K||_inf max|x| per block (||K||_inf =
// ||A||_inf ||B||_inf, computed in fp32 and widened by 2^-16 relative).
// FLAT: workgroup g = units 4 g .. 4 g + 3.  COLUMN: workgroup g (in the
// XCD-contiguous order) = column block j = g % nb, row units 4 (g / nb) .. + 3.
// Trailing waves with no rows take part in the build and return.
template <Mapping MAP, int NA, int NB, bool LU, bool WY, bool WY16>
__global__ __launch_bounds__(256) void kron_build_unit_kernel(const Params p) {
    constexpr int NF = NA * NA + NB * NB;
    __shared__ uint4 lds_x[4][256];   // per-wave input staging
    __shared__ uint4 lds_k[3][2][64];  // split K: [term hi, mid, lo][k-step][lane]
    __shared__ float fac[NF];          // A then B
    __shared__ float hdr[2];           // ||K||_inf bound, all-(+0) flag
    // the wave index as a uniform value, so that branches on the unit are scalar
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    int64_t jcol = 0, first;
    int nvalid;
    uint32_t bstride;
    if (MAP == Mapping::Flat) {
        first = ((int64_t)blockIdx.x * 4 + w) * 64;
        nvalid = (int)max<int64_t>(0, min<int64_t>(64, p.nblocks - first));
        bstride = 1;
    } else {
        const int64_t gi = xcd_order(blockIdx.x, gridDim.x);
        jcol = gi % p.nb;
        const int64_t row0 = ((gi / p.nb) * 4 + w) * 64;
        first = row0 * p.nb + jcol;
        nvalid = (int)max<int64_t>(0, min<int64_t>(64, p.M - row0));
        bstride = (uint32_t)p.nb;
    }
    const int64_t f = (p.nfac == 1) ? 0 : jcol;
    // the factor entries (NF <= 1040 < 256 * 5) are loaded before the input:
    // loads retire in order, so waiting for them does not wait for the input
    constexpr int FPT = (NF + 255) / 256;
    float fv[LU ? 1 : FPT];
    if (!LU) {
#pragma unroll
        for (int q = 0; q < FPT; ++q) {
            // unconditional (clamped index), so no branch hides the load from the wait counting
            const int i = min(threadIdx.x + 256 * q, (unsigned)NF - 1);
            const float* src = i < NA * NA ? p.A + f * (NA * NA) + i : p.B + f * (NB * NB) + (i - NA * NA);
            fv[q] = __builtin_nontemporal_load(src);
        }
    }
    // LU: the parameter pointer is read with the other kernel arguments, before
    // the input loads (an empty asm that takes it in scalar registers), so
    // that fetching the parameters after the input loads is one scalar round
    // trip, not two: where scalar loads are slow that saves the call 4-5%
    const float* const lu_ptr = LU ? p.lu + f * 15 : nullptr;
    if (LU) asm volatile("" ::"s"(lu_ptr), "s"(p.X), "s"(p.nblocks));
    uint4 v[4];
    load_unit_clamped<MAP>(p, first, nvalid, bstride, v);
    __builtin_amdgcn_sched_barrier(0);
    // phase 1: factors into LDS (LU: every thread decodes at most one entry)
    if (LU) {
        float g[5][4];
        float pv[15];
        lu_load(lu_ptr, pv);
        lu_g(pv, g);
#pragma unroll
        for (int q = 0; q < FPT; ++q) {
            const int i = threadIdx.x + 256 * q;
            if (i < NF) fac[i] = lu_entry<NA, NB>(g, i);
        }
    } else {
#pragma unroll
        for (int q = 0; q < FPT; ++q) {
            const int i = threadIdx.x + 256 * q;
            if (i < NF) fac[i] = fv[q];
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    // phase 2: this wave's share of the split K; wave 0 also the norms and flag
    {
        const float* Af = fac;
        const float* Bf = fac + NA * NA;
        const int n = perm_row(lane & 31), hh = lane >> 5;
        const int s = w >> 1, c0 = 4 * (w & 1);
        bf16x2 hi[2], mid[2], lo[2];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int k = 16 * s + 8 * hh + c0 + c;
            const float kv = Af[(n / NB) * NA + k / NB] * Bf[(n % NB) * NB + k % NB];
            const __bf16 t1 = (__bf16)kv;
            const float r1 = kv - (float)t1;  // exact
            const __bf16 t2 = (__bf16)r1;
            const float r2 = r1 - (float)t2;  // exact
            hi[c >> 1][c & 1] = t1;
            mid[c >> 1][c & 1] = t2;
            lo[c >> 1][c & 1] = (__bf16)r2;
        }
        auto put = [&](int term, const bf16x2 (&q)[2]) {
            uint2* dst = reinterpret_cast<uint2*>(&lds_k[term][s][lane]) + (w & 1);
            *dst = make_uint2(__builtin_bit_cast(uint32_t, q[0]), __builtin_bit_cast(uint32_t, q[1]));
        };
        put(0, hi);
        put(1, mid);
        put(2, lo);
        if (w == 0) {
            // lane i < NA: row i of A; NA <= lane < NA + NB: row lane - NA of B
            const bool in_a = lane < NA, in_b = lane >= NA && lane < NA + NB;
            const int len = in_a ? NA : NB;
            const float* row = in_a ? Af + lane * NA : Bf + (lane - NA) * NB;
            float rs = 0.0f;
            bool allneg = in_a || in_b;
            if (in_a || in_b) {
                for (int j = 0; j < len; ++j) {
                    rs += fabsf(row[j]);
                    allneg = allneg && (__float_as_uint(row[j]) >> 31);
                }
            }
            float ra = in_a ? rs : 0.0f, rb = in_b ? rs : 0.0f;
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                ra = fmaxf(ra, __shfl_xor(ra, off));
                rb = fmaxf(rb, __shfl_xor(rb, off));
            }
            const bool zero_ok = __builtin_amdgcn_ballot_w64(allneg) == 0;
            if (lane == 0) {
                hdr[0] = ra * rb * 0x1.0001p-17f;
                hdr[1] = zero_ok ? 1.0f : 0.0f;
            }
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    if (nvalid == 0) return;
    // phase 3: this lane's K slices, then the unit (one straight-line body for
    // full and partial units: fewer live registers than two specialised copies)
    KSlices ks;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        ks.hi[s] = __builtin_bit_cast(bf16x8, lds_k[0][s][lane]);
        ks.mid[s] = __builtin_bit_cast(bf16x8, lds_k[1][s][lane]);
        ks.lo[s] = __builtin_bit_cast(bf16x8, lds_k[2][s][lane]);
    }
    EdgeTest et;
    et.edge_t = 0u;
    et.kbound = hdr[0];
    const bool zero_ok = hdr[1] != 0.0f;
    unit_compute<MAP, NA, NB, false, WY, WY16, false, false>(p, lds_x[w], first, nvalid, bstride, v, ks, zero_ok, et,
                                                             fac, fac + NA * NA);
}

// Per-block factors (a pair per 32-column block, COLUMN mapping): eight waves
// per workgroup on a strip of 8 column blocks, 64 rows at a time, so that
// each row of a step is 512 contiguous bytes of X, 128 of codes and 8 of
// scales (one wave per 64-byte piece of 64 rows would touch a different cache
// line per row in every load and store).  Wave w owns column block 8 j + w of
// the strip and keeps its K in registers for all the strip's steps, built by
// each lane from its rows of A and B, which the wave stages in LDS (loaded,
// or decoded from the 15 parameters of G_1..G_5 when LU), with the window
// 2^-17 ||K||_inf max|x|, or, PW (kq_quantize_packed), with the pair's
// conditioning window T from its pack, as the flat packed kernel (with a pair
// per block, building K from the 320 bytes of A and B is cheaper than reading
// its 6 KiB pack, which would add 19-37% to a strip's input bytes; the 16-byte
// window header is all the packed call reads of it).  A step: wave w loads rows
// 8 w .. 8 w + 7 (two rows per 1 KiB load) and writes each 16-byte chunk to
// the LDS tile of the wave that owns its column block, then issues the next
// step's loads; after a barrier each wave runs the unit body on its column
// block and parks its codes and scales in LDS; after a second barrier the
// workgroup stores them along rows.  The binade-edge blocks of all steps are
// re-evaluated after the last step, their inputs read again from X (no lane
// keeps that code's registers live through the steps).  Grid: ceil(nrb / rg)
// ceil(nb / 8) workgroups (nrb = ceil(M / 64) row blocks, rg per strip) in
// the XCD-contiguous order, strips of the same rows next to each other.
// Columns and rows beyond the matrix are read clamped, staged as zeros and
// not stored.
//
// The wave tiles are 260 slots apart: the 64 extra bytes put the same chunk
// of the same row in different banks of the eight tiles, so the staging
// writes (a row's 32 chunks go to eight tiles) are free of bank conflicts.
constexpr int kTileCols = 8;
constexpr int kTileSlots = 260;
constexpr int kCodeSlots = 68;  // 64 blocks x 16 code bytes, then 64 scale bytes
constexpr int kTileMaxSteps = 8;

template <int NA, int NB, bool LU, bool WY, bool WY16, bool PW = false>
__global__ __launch_bounds__(64 * kTileCols) void kron_tile_kernel(const Params p, int rg) {
    constexpr int NF = NA * NA + NB * NB;
    constexpr int FPL = (NF + 63) / 64;  // factor entries per lane
    __shared__ uint4 lds_x[kTileCols * kTileSlots];
    __shared__ uint4 lds_c[kTileCols * kCodeSlots];
    __shared__ uint64_t stmask[kTileCols];
    __shared__ uint64_t sedges[kTileCols][kTileMaxSteps];
    __shared__ float fac[kTileCols * NF];  // each wave's A then B
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int64_t ntc = (p.nb + kTileCols - 1) / kTileCols;
    const int64_t nrb = (p.M + 63) / 64;
    const int64_t g = xcd_order(blockIdx.x, gridDim.x);
    const int64_t jt = g % ntc, rb0 = (g / ntc) * rg;
    const int nsteps = (int)min<int64_t>(rg, nrb - rb0);
    const int ncols = (int)min<int64_t>(kTileCols, p.nb - kTileCols * jt);
    const bool active = w < ncols;
    const int64_t jc = kTileCols * jt + (active ? w : 0);  // this wave's column block
    const int64_t f = (p.nfac == 1) ? 0 : jc;
    // K from the factors: this wave's A and B are staged in its LDS area,
    // loaded first (coalesced; loads retire in order, so waiting for them does
    // not wait for the input) or, LU, decoded there from the 15 parameters
    float fv[LU ? 1 : FPL];
    if (!LU) {
#pragma unroll
        for (int q = 0; q < FPL; ++q) {
            // unconditional (clamped index), so no branch hides the load from the wait counting
            const int i = min(lane + 64 * q, NF - 1);
            const float* src = i < NA * NA ? p.A + f * (NA * NA) + i : p.B + f * (NB * NB) + (i - NA * NA);
            fv[q] = __builtin_nontemporal_load(src);
        }
    }
    // load c of a step: row 8 w + 2 c + lane / 32, 16-byte chunk lane % 32 of
    // its 512 bytes; a wave-uniform base per step and 32-bit lane offsets
    // (64 rows of X span less than 4 GiB: d < 2^25, checked by the launcher)
    const int q = lane & 31;
    const int qb = min(q >> 2, ncols - 1);
    const uint32_t rowbytes = (uint32_t)(p.nb * 64);
    const uint32_t qoff = (uint32_t)(qb * 64 + (q & 3) * 16);
    const uint8_t* const xstrip = reinterpret_cast<const uint8_t*>(p.X) + kTileCols * jt * 64;
    uint4 v[4];
    auto issue = [&](int64_t row0) {
        const int nrows = (int)min<int64_t>(64, p.M - row0);
        const uint8_t* const xs = xstrip + row0 * p.nb * 64;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const uint32_t r = (uint32_t)min(8 * w + 2 * c + (lane >> 5), nrows - 1);
            v[c] = load_nt(reinterpret_cast<const uint4*>(xs + (r * rowbytes + qoff)));
        }
    };
    issue(rb0 * 64);
    __builtin_amdgcn_sched_barrier(0);
    KSlices ks;
    bool zero_ok;
    EdgeTest et;
    const float* Af = p.A + f * (NA * NA);
    const float* Bf = p.B + f * (NB * NB);
    {
        float* const facw = fac + w * NF;
        if (LU) {
            float gm[5][4];
            float pv[15];
            lu_load(p.lu + f * 15, pv);
            lu_g(pv, gm);
#pragma unroll
            for (int q2 = 0; q2 < FPL; ++q2) {
                const int i = lane + 64 * q2;
                if (i < NF) facw[i] = lu_entry<NA, NB>(gm, i);
            }
        } else {
#pragma unroll
            for (int q2 = 0; q2 < FPL; ++q2) {
                const int i = lane + 64 * q2;
                if (i < NF) facw[i] = fv[q2];
            }
        }
        wave_lds_sync();
        Af = facw;
        Bf = facw + NA * NA;
        KFactors<NA, NB> kf;
        load_k_factors<NA, NB>(Af, Bf, lane, kf);
        et.edge_t = 0u;
        et.kbound = build_k<NA, NB>(kf, ks) * 0x1.0001p-17f;
        // no row of A and no row of B with every sign bit set: then an
        // all-(+0) input block gives +0 for every output in the fixed order
        bool neg_row = false;
        if (lane < NA) {
            bool all = true;
#pragma unroll
            for (int j = 0; j < NA; ++j) all = all && (__float_as_uint(Af[lane * NA + j]) >> 31);
            neg_row = all;
        }
        if (lane < NB) {
            bool all = true;
#pragma unroll
            for (int j = 0; j < NB; ++j) all = all && (__float_as_uint(Bf[lane * NB + j]) >> 31);
            neg_row = neg_row || all;
        }
        zero_ok = __builtin_amdgcn_ballot_w64(neg_row) == 0;
        if (PW) {
            // the pair's conditioning window from its pack (kq_pack_factors)
            const float* hdr = reinterpret_cast<const float*>(p.kpack + f * kPackBytes + 6 * 64 * 16);
            zero_ok = __float_as_uint(ld_uniform(hdr, 2)) != 0u;
            et.edge_t = __float_as_uint(ld_uniform(hdr, 3));
        }
    }
    for (int it = 0; it < nsteps; ++it) {
        const int64_t row0 = (rb0 + it) * 64;
        const int nrows = (int)min<int64_t>(64, p.M - row0);
        // stage: chunk (q & 3) of column block q / 4 goes to that wave's tile
        if (nrows == 64 && ncols == kTileCols) {
            // a full step (the common case, uniform): every chunk as loaded
#pragma unroll
            for (int c = 0; c < 4; ++c)
                lds_x[kTileSlots * (q >> 2) + lds_slot(8 * w + 2 * c + (lane >> 5), q & 3)] = v[c];
        } else {
            // rows past M and column blocks past nb as zeros, branch-free
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int r = 8 * w + 2 * c + (lane >> 5);
                const uint32_t m = (r < nrows && (q >> 2) < ncols) ? ~0u : 0u;
                lds_x[kTileSlots * (q >> 2) + lds_slot(r, q & 3)] =
                    make_uint4(v[c].x & m, v[c].y & m, v[c].z & m, v[c].w & m);
            }
        }
        if (it + 1 < nsteps) issue(row0 + 64);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
        if (active)
            unit_compute<Mapping::Column, NA, NB, false, WY, WY16, false, PW, true>(
                p, lds_x + kTileSlots * w, row0 * p.nb + jc, nrows, (uint32_t)p.nb, v, ks, zero_ok, et, Af, Bf,
                TileSink{lds_c + kCodeSlots * w, &stmask[w], &sedges[w][it]});
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
        // row stores: thread t takes row t / 8, column block t % 8 of the step
        const int r = threadIdx.x >> 3, j = threadIdx.x & 7;
        const uint32_t mword = reinterpret_cast<const uint32_t*>(stmask)[2 * j + (r >> 5)];
        if (p.codes && r < nrows && j < ncols && ((mword >> (r & 31)) & 1u)) {
            const uint4* const ct = lds_c + kCodeSlots * j;
            const int64_t blk0 = row0 * p.nb + kTileCols * jt;  // wave-uniform
            const uint32_t ob = (uint32_t)r * (uint32_t)p.nb + (uint32_t)j;
            *reinterpret_cast<uint4*>(p.codes + blk0 * 16 + ob * 16u) = ct[r];
            (p.scales + blk0)[ob] = reinterpret_cast<const uint8_t*>(ct)[1024 + r];
        }
    }
    // blocks on a binade edge: the fixed evaluation order decides (this
    // wave's own records, so no barrier is needed)
    if (active) {
        for (int it = 0; it < nsteps; ++it) {
            // readfirstlane returns int: widen each half through uint32_t
            const uint64_t se = sedges[w][it];
            const uint64_t e = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)se) |
                               ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(se >> 32)) << 32);
            if (e) exact_flagged<NA, NB, true>(e, nullptr, (rb0 + it) * 64 * p.nb + jc, (uint32_t)p.nb, Af, Bf, p);
        }
    }
}

// Materialise and split K = A (x) B for every factor pair, in the lane layout
// of the matrix-core A operand (offline step; the K1 variant of Sec. 3.5
// keeps the dense 32x32 blocks in HBM).  Layout per pair (kPackBytes):
// uint4 [3 terms: hi, mid, lo][2 k-steps][64 lanes], then fp32 ||K||_inf,
// the relative binade-edge window rho, the all-(+0)-input flag and the
// mantissa window T derived from rho (see kron_mfma_unit_kernel).
// true when no row of F has every entry's sign bit set
__device__ bool no_negative_row(const float* F, int n) {
    for (int i = 0; i < n; ++i) {
        bool all = true;
        for (int j = 0; j < n; ++j) all = all && (__float_as_uint(F[i * n + j]) >> 31);
        if (all) return false;
    }
    return true;
}

__device__ double norm_inf_f64(const float* F, int n) {
    double best = 0.0;
    for (int i = 0; i < n; ++i) {
        double r = 0.0;
        for (int j = 0; j < n; ++j) r += fabs((double)F[i * n + j]);
        best = fmax(best, r);
    }
    return best;
}

// ||F^-1||_inf by fp64 Gauss-Jordan with partial pivoting in `work`
// (n x 2n doubles); +inf if a pivot vanishes.
__device__ double inverse_norm_inf_f64(const float* F, int n, double* work) {
    const int w = 2 * n;
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < w; ++j) work[i * w + j] = j < n ? (double)F[i * n + j] : (j - n == i ? 1.0 : 0.0);
    for (int c = 0; c < n; ++c) {
        int piv = c;
        for (int r = c + 1; r < n; ++r)
            if (fabs(work[r * w + c]) > fabs(work[piv * w + c])) piv = r;
        const double pv = work[piv * w + c];
        if (pv == 0.0) return __builtin_inf();
        if (piv != c)
            for (int j = 0; j < w; ++j) {
                const double t = work[c * w + j];
                work[c * w + j] = work[piv * w + j];
                work[piv * w + j] = t;
            }
        for (int j = 0; j < w; ++j) work[c * w + j] /= pv;
        for (int r = 0; r < n; ++r) {
            if (r == c) continue;
            const double fct = work[r * w + c];
            if (fct != 0.0)
                for (int j = 0; j < w; ++j) work[r * w + j] -= fct * work[c * w + j];
        }
    }
    double best = 0.0;
    for (int i = 0; i < n; ++i) {
        double r = 0.0;
        for (int j = n; j < w; ++j) r += fabs(work[i * w + j]);
        best = fmax(best, r);
    }
    return best;
}

template <int NA, int NB>
__global__ __launch_bounds__(64) void pack_kernel(const float* __restrict__ A, const float* __restrict__ B,
                                                  int64_t nfac, uint8_t* __restrict__ kpack) {
    __shared__ double pack_lds[32 * 64];  // Gauss-Jordan workspace of lane 0
    const int lane = threadIdx.x;
    for (int64_t f = blockIdx.x; f < nfac; f += gridDim.x) {
        KFactors<NA, NB> kf;
        load_k_factors<NA, NB>(A + f * (NA * NA), B + f * (NB * NB), lane, kf);
        KSlices ks;
        const float kinf = build_k<NA, NB>(kf, ks);
        // relative binade-edge window rho = 2^-17 cond_inf(K), cond_inf(K) =
        // ||A||_inf ||B||_inf ||A^-1||_inf ||B^-1||_inf (Kronecker norms multiply)
        float rho = __builtin_inff();
        uint32_t edge_t = 1u << 22;  // every block re-evaluated
        if (lane == 0) {
            double* work = reinterpret_cast<double*>(pack_lds);
            const double na = norm_inf_f64(A + f * (NA * NA), NA), nb_ = norm_inf_f64(B + f * (NB * NB), NB);
            const double nai = inverse_norm_inf_f64(A + f * (NA * NA), NA, work);
            const double nbi = inverse_norm_inf_f64(B + f * (NB * NB), NB, work);
            const double cond = 1.01 * na * nb_ * nai * nbi;
            if (cond <= 8192.0) {
                rho = (float)(cond * 0x1p-17);
                // T = ceil(2^24 rho) = ceil(2^7 cond) <= 2^20
                edge_t = (uint32_t)ceil(cond * 128.0);
            }
        }
        rho = __shfl(rho, 0);
        uint32_t zero_ok = 0u;
        if (lane == 0) zero_ok = (no_negative_row(A + f * (NA * NA), NA) && no_negative_row(B + f * (NB * NB), NB)) ? 1u : 0u;
        uint4* pk = reinterpret_cast<uint4*>(kpack + f * kPackBytes);
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            pk[(0 * 2 + s) * 64 + lane] = __builtin_bit_cast(uint4, ks.hi[s]);
            pk[(1 * 2 + s) * 64 + lane] = __builtin_bit_cast(uint4, ks.mid[s]);
            pk[(2 * 2 + s) * 64 + lane] = __builtin_bit_cast(uint4, ks.lo[s]);
        }
        if (lane == 0)
            *reinterpret_cast<uint4*>(kpack + f * kPackBytes + 6 * 64 * 16) =
                make_uint4(__float_as_uint(kinf), __float_as_uint(rho), zero_ok, edge_t);
    }
}

// The quantizers' memory traffic with no arithmetic: one wave per 64-block
// unit reads its 4 KiB with the same four nontemporal 1 KiB loads and writes
// 16 bytes and one byte per block (the XOR of the block's four 16-byte
// chunks and the low byte of that XOR's first two words), so the time of this
// kernel is what the launch shape and the bytes alone cost.
__global__ __launch_bounds__(64) void stream_floor_kernel(const Params p) {
    const int lane = threadIdx.x;
    const int64_t first = (int64_t)blockIdx.x * 64;
    const int nvalid = (int)min<int64_t>(64, p.nblocks - first);
    const uint4* src = reinterpret_cast<const uint4*>(p.X) + first * 4;
    uint4 v[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int ci = 64 * c + lane;
        v[c] = make_uint4(0u, 0u, 0u, 0u);
        if ((ci >> 2) < nvalid) v[c] = load_nt(src + ci);
    }
    // lane l holds chunk l % 4 of block 16 c + l / 4 of load c; fold the four
    // chunks of each block into the lane that owns it after the fold: the XOR
    // over lanes 4 k .. 4 k + 3 (DPP quad reductions) lands in lane 4 k
    uint4 r[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        uint32_t w[4] = {v[c].x, v[c].y, v[c].z, v[c].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            w[i] ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w[i], 0xB1, 0xF, 0xF, false);  // lane ^ 1
            w[i] ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w[i], 0x4E, 0xF, 0xF, false);  // lane ^ 2
        }
        r[c] = make_uint4(w[0], w[1], w[2], w[3]);
    }
    if ((lane & 3) == 0) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int b = 16 * c + (lane >> 2);
            if (b < nvalid) {
                *reinterpret_cast<uint4*>(p.codes + (first + b) * 16) = r[c];
                p.scales[first + b] = (uint8_t)(r[c].x ^ r[c].y);
            }
        }
    }
}

// Launch-shape probe of the same traffic, a measurement aid that is not tied
// to the quantizers' launch shape: W waves per workgroup, U units per wave
// with all U x 4 loads issued before any store; with `stride` the grid walks
// the units in a grid-stride loop, else each wave takes U units once.  Same
// outputs as stream_floor_kernel.
template <int U, int W>
__global__ __launch_bounds__(64 * W) void stream_probe_kernel(const Params p, int stride) {
    const int lane = threadIdx.x & 63;
    const int64_t nunits = (p.nblocks + 63) / 64;
    const int64_t wstep = (int64_t)gridDim.x * W;
    for (int64_t wv = (int64_t)blockIdx.x * W + (threadIdx.x >> 6); wv * U < nunits; wv += wstep) {
        uint4 v[U][4];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t first = (wv * U + k) * 64;
            const int64_t nvalid = min<int64_t>(64, max<int64_t>(0, p.nblocks - first));
            const uint4* src = reinterpret_cast<const uint4*>(p.X) + first * 4;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int ci = 64 * c + lane;
                v[k][c] = make_uint4(0u, 0u, 0u, 0u);
                if ((ci >> 2) < nvalid) v[k][c] = load_nt(src + ci);
            }
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t first = (wv * U + k) * 64;
            const int64_t nvalid = min<int64_t>(64, max<int64_t>(0, p.nblocks - first));
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                uint32_t w[4] = {v[k][c].x, v[k][c].y, v[k][c].z, v[k][c].w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    w[i] ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w[i], 0xB1, 0xF, 0xF, false);  // lane ^ 1
                    w[i] ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w[i], 0x4E, 0xF, 0xF, false);  // lane ^ 2
                }
                const int b = 16 * c + (lane >> 2);
                if ((lane & 3) == 0 && b < nvalid) {
                    *reinterpret_cast<uint4*>(p.codes + (first + b) * 16) = make_uint4(w[0], w[1], w[2], w[3]);
                    p.scales[first + b] = (uint8_t)(w[0] ^ w[1]);
                }
            }
        }
        if (!stride) break;
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

// ------------------------------------------------------------------ full-row FWHT comparator
// y = H_d x / sqrt(d) over the whole row (d = 2^LOG2D, 32 <= d <= 16384): the
// FWHT baseline of Sec. 4.4 (Table 2), then MXFP4 of every 32-element block.
// Same butterflies in the same order as the fixed-order definition -- stride
// h = 1, 2, ..., d/2, then one multiply by the fp32 nearest to 1/sqrt(d) -- so
// the outputs are bit-identical to it.  A thread owns 32 elements of its row
// at a time.  Pass q applies the strides 2^(5q) .. 2^(5q+k-1) (k <= 5 index
// bits) in registers; between passes the row goes through LDS (fp32, one pad
// float per 32) from one element assignment to the next:
//   element of slot j in pass (lo, k) =
//     deposit(v, other bits) | (j mod 2^k) << lo,   v = tl | (j >> k) << (LOG2D - 5),
// "other bits" being the index bits outside [lo, lo + k) in increasing order,
// tl the thread's index within its row.  Pass 0 is the thread's own block.
// Measurement aid: one lane stores the device's constant-rate real-time
// counter (100 MHz), so that a stream of launches can be timed between two
// of these from inside a captured graph.
__global__ __launch_bounds__(64) void timestamp_kernel(uint64_t* dst) {
    if (threadIdx.x == 0) dst[0] = __builtin_amdgcn_s_memrealtime();
}

hipError_t launch_timestamp(uint64_t* dst, hipStream_t st) {
    hipLaunchKernelGGL(timestamp_kernel, dim3(1), dim3(64), 0, st, dst);
    return hipGetLastError();
}

template <int LOG2D>
__device__ __forceinline__ int fwht_index(int lo, int k, int j, int tl) {
    const int v = tl | ((j >> k) << (LOG2D - 5));
    const int low = v & ((1 << lo) - 1);
    return low | ((j & ((1 << k) - 1)) << lo) | ((v >> lo) << (lo + k));
}

template <int LOG2D>
__global__ __launch_bounds__(LOG2D == 14 ? 512 : 256) void fwht_kernel(const Params p) {
    constexpr int D = 1 << LOG2D;
    constexpr int TPR = D / 32;                   // threads per row
    constexpr int T = TPR < 256 ? 256 : TPR;      // threads per workgroup
    constexpr int R = T / TPR;                    // rows per workgroup
    constexpr int NPASS = (LOG2D + 4) / 5;
    constexpr int RS = D + D / 32;                // padded row stride in LDS
    __shared__ float buf[NPASS > 1 ? R * RS : 1];
    const int t = threadIdx.x;
    const int r = t / TPR, tl = t % TPR;
    const int64_t row = (int64_t)blockIdx.x * R + r;
    const bool active = row < p.M;
    float u[32];
    {
        const uint4* src = reinterpret_cast<const uint4*>(p.X + (active ? row : 0) * D) + tl * 4;
#pragma unroll
        for (int m = 0; m < 4; ++m) unpack8(active ? src[m] : make_uint4(0u, 0u, 0u, 0u), u + 8 * m);
    }
    float* rb = buf + r * RS;
    auto pad = [](int i) { return i + (i >> 5); };
#pragma unroll
    for (int q = 0; q < NPASS; ++q) {
        const int lo = 5 * q, k = (LOG2D - lo) < 5 ? (LOG2D - lo) : 5;
        if (q > 0) {
            const int plo = 5 * (q - 1);
            __syncthreads();  // earlier reads of buf are done
#pragma unroll
            for (int j = 0; j < 32; ++j) rb[pad(fwht_index<LOG2D>(plo, 5, j, tl))] = u[j];
            __syncthreads();
#pragma unroll
            for (int j = 0; j < 32; ++j) u[j] = rb[pad(fwht_index<LOG2D>(lo, k, j, tl))];
        }
#pragma unroll
        for (int b = 0; b < 5; ++b) {
            if (b >= k) break;
            const int h = 1 << b;
#pragma unroll
            for (int j = 0; j < 32; ++j) {
                if (j & h) continue;
                const float s0 = u[j] + u[j + h];
                const float s1 = u[j] - u[j + h];
                u[j] = s0;
                u[j + h] = s1;
            }
        }
    }
    if (NPASS > 1) {  // back to the thread's own block
        const int llo = 5 * (NPASS - 1), lk = LOG2D - llo;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 32; ++j) rb[pad(fwht_index<LOG2D>(llo, lk, j, tl))] = u[j];
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 32; ++j) u[j] = rb[pad(fwht_index<LOG2D>(0, 5, j, tl))];
    }
    // fp32 nearest to 1/sqrt(d): 2^(-n/2) for even n, fp32(1/sqrt2) * 2^(-(n-1)/2) for odd n
    const float inv_sqrt_d = (LOG2D & 1) ? __uint_as_float(0x3F3504F3u - ((uint32_t)(LOG2D - 1) / 2u << 23))
                                         : __uint_as_float((uint32_t)(127 - LOG2D / 2) << 23);
    float y[32];
#pragma unroll
    for (int j = 0; j < 32; ++j) y[j] = u[j] * inv_sqrt_d;
    if (!active) return;
    uint32_t w[4];
    const uint32_t sbyte = encode32(y, w);
    const int64_t blk = row * TPR + tl;
    if (p.codes) {
        *reinterpret_cast<uint4*>(p.codes + blk * 16) = make_uint4(w[0], w[1], w[2], w[3]);
        p.scales[blk] = (uint8_t)sbyte;
    }
    if (p.y) {
        float4* dst = reinterpret_cast<float4*>(p.y + blk * 32);
#pragma unroll
        for (int m = 0; m < 8; ++m) dst[m] = make_float4(y[4 * m], y[4 * m + 1], y[4 * m + 2], y[4 * m + 3]);
    }
}

// ------------------------------------------------------------------ launchers
template <Mapping MAP, class Op>
static hipError_t launch_map(Params p, hipStream_t st) {
    if (MAP == Mapping::Flat)
        p.units = (p.nblocks + 63) / 64;
    else
        p.units = ((p.M + 63) / 64) * p.nb;
    int64_t g = p.units < kMaxGridStride ? p.units : kMaxGridStride;
    if (g < 1) g = 1;
    hipLaunchKernelGGL((quant_kernel<MAP, Op>), dim3((unsigned)g), dim3(64), 0, st, p);
    return hipGetLastError();
}

template <class Op>
static hipError_t launch_op(const Params& p, Mapping map, hipStream_t st) {
    if (map == Mapping::Flat) return launch_map<Mapping::Flat, Op>(p, st);
    return launch_map<Mapping::Column, Op>(p, st);
}

template <Mapping MAP, int NA, int NB>
static hipError_t launch_unit(const Params& p, int64_t units, bool ilv, hipStream_t st) {
    const dim3 g((unsigned)units), b(64);
    if (ilv) {
        if (p.y) hipLaunchKernelGGL((kron_mfma_unit_kernel<MAP, NA, NB, true, true>), g, b, 0, st, p);
        else hipLaunchKernelGGL((kron_mfma_unit_kernel<MAP, NA, NB, true, false>), g, b, 0, st, p);
    } else {
        if (p.y) hipLaunchKernelGGL((kron_mfma_unit_kernel<MAP, NA, NB, false, true>), g, b, 0, st, p);
        else hipLaunchKernelGGL((kron_mfma_unit_kernel<MAP, NA, NB, false, false>), g, b, 0, st, p);
    }
    return hipGetLastError();
}

// Per-block factors: the 8-column tile kernel (K built per wave).
template <int NA, int NB, bool LU>
static hipError_t launch_tile(const Params& p, int rg, hipStream_t st) {
    const int64_t nrb = (p.M + 63) / 64, ntc = (p.nb + kTileCols - 1) / kTileCols;
    const dim3 g((unsigned)(((nrb + rg - 1) / rg) * ntc)), b(64 * kTileCols);
    const bool wy = p.y != nullptr, wy16 = LU && p.y16 != nullptr;
#define KQ_TILE(WY, WY16) hipLaunchKernelGGL((kron_tile_kernel<NA, NB, LU, WY, WY16>), g, b, 0, st, p, rg)
    if (!LU && p.kpack) {
        if (wy) hipLaunchKernelGGL((kron_tile_kernel<NA, NB, false, true, false, true>), g, b, 0, st, p, rg);
        else hipLaunchKernelGGL((kron_tile_kernel<NA, NB, false, false, false, true>), g, b, 0, st, p, rg);
        return hipGetLastError();
    }
    if (wy16) { if (wy) KQ_TILE(true, LU); else KQ_TILE(false, LU); }
    else { if (wy) KQ_TILE(true, false); else KQ_TILE(false, false); }
#undef KQ_TILE
    return hipGetLastError();
}

// Row blocks per strip of the tile kernel (1 .. kTileMaxSteps): as many as
// keep at least ~1728 workgroups (about three rounds of the 512 that fit at
// once: more steps amortise each wave's K build).
static int tile_rows(const Params& p) {
    const int64_t tiles = ((p.M + 63) / 64) * ((p.nb + kTileCols - 1) / kTileCols);
    const int64_t rg = tiles / 1728;
    return rg < 1 ? 1 : rg > kTileMaxSteps ? kTileMaxSteps : (int)rg;
}

// The on-chip-K unit kernel: four units per workgroup (one factor pair each).
template <int NA, int NB, bool LU>
static hipError_t launch_build(const Params& p, Mapping map, hipStream_t st) {
    const int64_t g = (map == Mapping::Flat) ? ((p.nblocks + 63) / 64 + 3) / 4 : (((p.M + 63) / 64 + 3) / 4) * p.nb;
    const dim3 grid((unsigned)g), b(256);
    const bool wy = p.y != nullptr, wy16 = LU && p.y16 != nullptr;
#define KQ_BUILD(MAP, WY, WY16) hipLaunchKernelGGL((kron_build_unit_kernel<MAP, NA, NB, LU, WY, WY16>), grid, b, 0, st, p)
    if (map == Mapping::Flat) {
        if (wy16) { if (wy) KQ_BUILD(Mapping::Flat, true, LU); else KQ_BUILD(Mapping::Flat, false, LU); }
        else { if (wy) KQ_BUILD(Mapping::Flat, true, false); else KQ_BUILD(Mapping::Flat, false, false); }
    } else {
        if (wy16) { if (wy) KQ_BUILD(Mapping::Column, true, LU); else KQ_BUILD(Mapping::Column, false, LU); }
        else { if (wy) KQ_BUILD(Mapping::Column, true, false); else KQ_BUILD(Mapping::Column, false, false); }
    }
#undef KQ_BUILD
    return hipGetLastError();
}

// Per-block factors (COLUMN mapping) run on the 8-column tile kernel, which
// builds each pair's K from A and B even when a pack is given; shared
// factors on one 64-block unit per wave, K from the pack (the two tiles'
// products interleaved on grids of at most kInterleaveMaxUnits units, where
// fewer waves per SIMD hide less latency) or built per 4-wave workgroup.
// The API layer has checked that every grid fits one launch.
template <int NA, int NB>
static hipError_t launch_mfma(const Params& p, Mapping map, hipStream_t st) {
    if (map == Mapping::Column) return launch_tile<NA, NB, false>(p, tile_rows(p), st);  // K built, window from the pack
    const int64_t units = (p.nblocks + 63) / 64;
    if (p.kpack) return launch_unit<Mapping::Flat, NA, NB>(p, units, units <= kInterleaveMaxUnits, st);
    return launch_build<NA, NB, false>(p, map, st);
}

template <int NA, int NB>
static hipError_t launch_lu(const Params& p, Mapping map, hipStream_t st) {
    if (map == Mapping::Column) return launch_tile<NA, NB, true>(p, tile_rows(p), st);
    return launch_build<NA, NB, true>(p, map, st);
}

hipError_t launch_pack(int a, const float* A, const float* B, int64_t nfac, uint8_t* kpack, hipStream_t st) {
    const unsigned g = (unsigned)(nfac < 65536 ? nfac : 65536);
    switch (a) {
        case 4: hipLaunchKernelGGL((pack_kernel<4, 8>), dim3(g), dim3(64), 0, st, A, B, nfac, kpack); break;
        case 2: hipLaunchKernelGGL((pack_kernel<2, 16>), dim3(g), dim3(64), 0, st, A, B, nfac, kpack); break;
        case 8: hipLaunchKernelGGL((pack_kernel<8, 4>), dim3(g), dim3(64), 0, st, A, B, nfac, kpack); break;
        case 1: hipLaunchKernelGGL((pack_kernel<1, 32>), dim3(g), dim3(64), 0, st, A, B, nfac, kpack); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch(Kind kind, int a, const Params& p, Mapping map, hipStream_t st) {
    switch (kind) {
        case Kind::Plain: return launch_op<PlainOp>(p, map, st);
        case Kind::Smooth: {
            // column-stationary: a grid stride that is a multiple of nb / gcd(nb, 64)
            Params q = p;
            q.units = (p.nblocks + 63) / 64;
            int64_t a = p.nb, b = 64;  // gcd(nb, 64)
            while (b) { const int64_t t = a % b; a = b; b = t; }
            const int64_t period = p.nb / a;  // stride multiple that keeps columns fixed
            int64_t g = (kSmoothWaves + period - 1) / period * period;
            if (g > q.units) g = q.units;  // one unit per workgroup: no stride needed
            hipLaunchKernelGGL(smooth_stationary_kernel, dim3((unsigned)g), dim3(64), 0, st, q);
            return hipGetLastError();
        }
        case Kind::Hadamard: return launch_op<HadamardOp>(p, map, st);
        case Kind::KronMfma:
            switch (a) {
                case 4: return launch_mfma<4, 8>(p, map, st);
                case 2: return launch_mfma<2, 16>(p, map, st);
                case 8: return launch_mfma<8, 4>(p, map, st);
                case 1: return launch_mfma<1, 32>(p, map, st);
                default: return hipErrorInvalidValue;
            }
        case Kind::KronLU:
            switch (a) {
                case 4: return launch_lu<4, 8>(p, map, st);
                case 2: return launch_lu<2, 16>(p, map, st);
                case 8: return launch_lu<8, 4>(p, map, st);
                case 1: return launch_lu<1, 32>(p, map, st);
                default: return hipErrorInvalidValue;
            }
        case Kind::Kron:
            switch (a) {
                case 4: return launch_op<KronOp<4, 8>>(p, map, st);
                case 2: return launch_op<KronOp<2, 16>>(p, map, st);
                case 8: return launch_op<KronOp<8, 4>>(p, map, st);
                case 1: return launch_op<KronOp<1, 32>>(p, map, st);
                default: return hipErrorInvalidValue;
            }
    }
    return hipErrorInvalidValue;
}

template <int LOG2D>
static hipError_t launch_fwht_n(const Params& p, hipStream_t st) {
    constexpr int TPR = (1 << LOG2D) / 32;
    constexpr int T = TPR < 256 ? 256 : TPR;
    constexpr int R = T / TPR;
    const int64_t g = (p.M + R - 1) / R;
    hipLaunchKernelGGL((fwht_kernel<LOG2D>), dim3((unsigned)g), dim3(T), 0, st, p);
    return hipGetLastError();
}

hipError_t launch_fwht(const Params& p, hipStream_t st) {
    switch (p.d) {
        case 32: return launch_fwht_n<5>(p, st);
        case 64: return launch_fwht_n<6>(p, st);
        case 128: return launch_fwht_n<7>(p, st);
        case 256: return launch_fwht_n<8>(p, st);
        case 512: return launch_fwht_n<9>(p, st);
        case 1024: return launch_fwht_n<10>(p, st);
        case 2048: return launch_fwht_n<11>(p, st);
        case 4096: return launch_fwht_n<12>(p, st);
        case 8192: return launch_fwht_n<13>(p, st);
        case 16384: return launch_fwht_n<14>(p, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_stream_floor(const Params& p, hipStream_t st) {
    const int64_t units = (p.nblocks + 63) / 64;
    hipLaunchKernelGGL(stream_floor_kernel, dim3((unsigned)units), dim3(64), 0, st, p);
    return hipGetLastError();
}

template <int U>
static hipError_t launch_probe_u(const Params& p, int waves, int64_t groups, hipStream_t st) {
    const int64_t units = (p.nblocks + 63) / 64;
    const int64_t g = groups > 0 ? groups : (units + (int64_t)U * waves - 1) / ((int64_t)U * waves);
    const int stride = groups > 0 ? 1 : 0;
    const dim3 grid((unsigned)g), b(64 * waves);
    switch (waves) {
        case 1: hipLaunchKernelGGL((stream_probe_kernel<U, 1>), grid, b, 0, st, p, stride); break;
        case 2: hipLaunchKernelGGL((stream_probe_kernel<U, 2>), grid, b, 0, st, p, stride); break;
        case 4: hipLaunchKernelGGL((stream_probe_kernel<U, 4>), grid, b, 0, st, p, stride); break;
        case 8: hipLaunchKernelGGL((stream_probe_kernel<U, 8>), grid, b, 0, st, p, stride); break;
        case 16: hipLaunchKernelGGL((stream_probe_kernel<U, 16>), grid, b, 0, st, p, stride); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_stream_probe(const Params& p, int waves, int units, int64_t groups, hipStream_t st) {
    switch (units) {
        case 1: return launch_probe_u<1>(p, waves, groups, st);
        case 2: return launch_probe_u<2>(p, waves, groups, st);
        case 4: return launch_probe_u<4>(p, waves, groups, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_e2m1(const float* v, int64_t npairs, uint32_t s, uint8_t* codes, hipStream_t st) {
    int64_t g = (npairs + kThreads - 1) / kThreads;
    if (g > 65536) g = 65536;
    if (g < 1) g = 1;
    hipLaunchKernelGGL(e2m1_kernel, dim3((unsigned)g), dim3(kThreads), 0, st, v, npairs, s, codes);
    return hipGetLastError();
}

}  // namespace kq
