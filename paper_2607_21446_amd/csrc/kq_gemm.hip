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

// Four consecutive C values of row m from column n: fp32 (with the bias or
// the accumulate mode), or rounded to bf16 (nearest even) when C16 is set.
__device__ __forceinline__ void store_c4(const GemmParams& g, int64_t m, int64_t n, float4 v) {
    if (g.C16) {
        uint16_t* crow = g.C16 + m * g.ldc_out;
        const float f[4] = {v.x, v.y, v.z, v.w};
        if (g.vec_ok && n + 3 < g.N) {
            typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
            const bf16x4 b = {(__bf16)v.x, (__bf16)v.y, (__bf16)v.z, (__bf16)v.w};
            *reinterpret_cast<uint2*>(crow + n) = __builtin_bit_cast(uint2, b);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (n + e < g.N) crow[n + e] = __builtin_bit_cast(uint16_t, (__bf16)f[e]);
        }
        return;
    }
    float* crow = g.C + m * g.ldc_out;
    const float* brow = g.bias ? g.bias + m * g.ldc_out : g.accumulate ? crow : nullptr;
    if (g.vec_ok && n + 3 < g.N) {
        if (brow) {
            const float4 o = *reinterpret_cast<const float4*>(brow + n);
            v = make_float4(o.x + v.x, o.y + v.y, o.z + v.z, o.w + v.w);
        }
        *reinterpret_cast<float4*>(crow + n) = v;
    } else {
        if (n + 0 < g.N) crow[n + 0] = brow ? brow[n + 0] + v.x : v.x;
        if (n + 1 < g.N) crow[n + 1] = brow ? brow[n + 1] + v.y : v.y;
        if (n + 2 < g.N) crow[n + 2] = brow ? brow[n + 2] + v.z : v.z;
        if (n + 3 < g.N) crow[n + 3] = brow ? brow[n + 3] + v.w : v.w;
    }
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
                    if (g.C16) {
                        g.C16[row * g.ldc_out + col] = __builtin_bit_cast(uint16_t, (__bf16)acc[i][j][4 * q + e]);
                        continue;
                    }
                    float* dst = g.C + row * g.ldc_out + col;
                    const float base = g.bias ? g.bias[row * g.ldc_out + col] : g.accumulate ? *dst : 0.0f;
                    *dst = (g.bias || g.accumulate) ? base + acc[i][j][4 * q + e] : acc[i][j][4 * q + e];
                }
        }
}

// K advances 128 (four 32-blocks) per pipeline stage in the LDS-pipelined kernels below.
constexpr int kGemmTileK = 128;

// Pipelined variant (K a multiple of 128, 4-byte-aligned scales): workgroup
// tile 128 (N) x 128 (M), waves 2 x 2 of 64 x 64, K 128 per stage.  Codes and
// scales go from global memory straight into LDS (global_load_lds: lane l's
// 16 or 4 bytes land at the wave-uniform LDS address + 16 l or 4 l) with
// kGemmStages stages in flight, so no register staging and no ds_write.
// Per stage the workgroup issues 20 such loads, 5 per wave:
//   W and X codes of rows 32 w .. 32 w + 31 (two loads each, 16 rows x 64 B), and
//   one scale group: wave 0 W rows 0-63, 1 W rows 64-127, 2 X rows 0-63, 3 X rows 64-127;
// rows past N or M load row N-1 or M-1 (their products land in C rows or
// columns that are never stored).  Before a stage is used each wave waits
// until only its later stages' loads are outstanding, then one barrier.
constexpr int kGemmStages = 3;
constexpr int kPipeLoadsPerWave = 5;

struct PipeBuf {
    uint4 wc[4 * 128];   // 128 rows x 4 blocks of 16 B, slot pipe_slot(row, block)
    uint4 xc[4 * 128];
    uint32_t ws[128];    // scales of the stage's 4 blocks, one dword per row
    uint32_t xs[128];
};

__device__ __forceinline__ void lds_load16(const uint8_t* src, void* lds_base) {
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                     (__attribute__((address_space(3))) void*)lds_base, 16, 0, 0);
}
__device__ __forceinline__ void lds_load4(const uint8_t* src, void* lds_base) {
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                     (__attribute__((address_space(3))) void*)lds_base, 4, 0, 0);
}

// LDS slot of block b of tile row q: 4 q + (b ^ ((q >> 2) & 3)).  A DMA
// instruction fills 64 consecutive slots (16 rows), so lane l reads row
// 16 i + l / 4, block (l % 4) ^ (((l / 4) >> 2) & 3): each instruction reads
// 16 contiguous 64-byte row segments, and a fragment read (32 rows, one
// block) spreads over all LDS banks.
__device__ __forceinline__ int pipe_slot(int q, int b) { return 4 * q + (b ^ ((q >> 2) & 3)); }

__device__ __forceinline__ void pipe_issue(const GemmParams& g, PipeBuf& b, int wave, int lane, int64_t nb0,
                                           int64_t mb0, int64_t row_bytes, int64_t nkb, int64_t st) {
    const int q = lane >> 2;                                  // row within the instruction's 16
    const int blk = (lane & 3) ^ ((q >> 2) & 3);
    const int64_t kbyte = (4 * st + blk) * 16;
#pragma unroll
    for (int gr = 0; gr < 2; ++gr) {
        const int row = 16 * (2 * wave + gr) + q;             // this wave fills rows 32 w .. 32 w + 31
        const int64_t n = min(nb0 + row, g.N - 1);
        const int64_t m = min(mb0 + row, g.M - 1);
        lds_load16(g.b_codes + n * row_bytes + kbyte, &b.wc[64 * (2 * wave + gr)]);
        lds_load16(g.a_codes + m * row_bytes + kbyte, &b.xc[64 * (2 * wave + gr)]);
    }
    const int gr = wave & 1;
    if (wave < 2) {
        const int64_t n = min(nb0 + 64 * gr + lane, g.N - 1);
        lds_load4(g.b_scales + n * nkb + 4 * st, &b.ws[64 * gr]);
    } else {
        const int64_t m = min(mb0 + 64 * gr + lane, g.M - 1);
        lds_load4(g.a_scales + m * nkb + 4 * st, &b.xs[64 * gr]);
    }
}

template <int STEP>
__device__ __forceinline__ void pipe_step(const PipeBuf& b, int h, int wn, int wm, int r, const uint32_t (&scw)[2],
                                          const uint32_t (&scx)[2], f32x16g (&acc)[2][2]) {
    uint4 fw[2], fx[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) fw[i] = b.wc[pipe_slot(wn * 64 + 32 * i + r, 2 * STEP + h)];
#pragma unroll
    for (int j = 0; j < 2; ++j) fx[j] = b.xc[pipe_slot(wm * 64 + 32 * j + r, 2 * STEP + h)];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                operand(Frag{fw[i], 0u}), operand(Frag{fx[j], 0u}), acc[i][j], 4, 4, STEP, (int)scw[i], STEP, (int)scx[j]);
}

// The three stage buffers are distinct LDS objects, and the main loop is
// unrolled by three so that every access names its buffer at compile time:
// the waits the compiler adds before LDS reads then cover only loads into
// that buffer, and the barrier between stages is a bare s_barrier after an
// explicit vmcnt wait (a fenced barrier would drain the loads in flight for
// the later stages).
__shared__ PipeBuf g_pipe0, g_pipe1, g_pipe2;

template <int B>
__device__ __forceinline__ PipeBuf& pipe_buf() {
    if constexpr (B == 0) return g_pipe0;
    else if constexpr (B == 1) return g_pipe1;
    else return g_pipe2;
}

struct PipeCtx {
    int wave, lane, r, h, wn, wm;
    int64_t nb0, mb0, nkb, row_bytes, nst;
    uint32_t psel;
};

// stage st lives in buffer CUR = st % 3; stage st + 2 is issued into NXT = (st + 2) % 3
template <int CUR, int NXT>
__device__ __forceinline__ void pipe_iter(const GemmParams& g, const PipeCtx& c, int64_t st, f32x16g (&acc)[2][2]) {
    if (st + 1 < c.nst)
        __builtin_amdgcn_s_waitcnt((kPipeLoadsPerWave & 15) | (7 << 4) | (15 << 8));  // vmcnt(5)
    else
        __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
    __builtin_amdgcn_s_barrier();
    if (st + 2 < c.nst) pipe_issue(g, pipe_buf<NXT>(), c.wave, c.lane, c.nb0, c.mb0, c.row_bytes, c.nkb, st + 2);
    const PipeBuf& b = pipe_buf<CUR>();
    uint32_t scw[2], scx[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) scw[i] = __builtin_amdgcn_perm(0u, b.ws[c.wn * 64 + 32 * i + c.r], c.psel);
#pragma unroll
    for (int j = 0; j < 2; ++j) scx[j] = __builtin_amdgcn_perm(0u, b.xs[c.wm * 64 + 32 * j + c.r], c.psel);
    pipe_step<0>(b, c.h, c.wn, c.wm, c.r, scw, scx, acc);
    pipe_step<1>(b, c.h, c.wn, c.wm, c.r, scw, scx, acc);
}

__global__ __launch_bounds__(256) void mxfp4_gemm_pipe_kernel(const GemmParams g) {
    PipeCtx c;
    const int t = threadIdx.x;
    c.wave = t >> 6;
    c.lane = t & 63;
    c.r = c.lane & 31;
    c.h = c.lane >> 5;
    c.wn = c.wave >> 1;
    c.wm = c.wave & 1;
    c.nb0 = (int64_t)blockIdx.x * 128;
    c.mb0 = (int64_t)blockIdx.y * 128;
    c.nkb = g.K / 32;
    c.row_bytes = g.K / 2;
    c.nst = g.K / 128;
    c.psel = c.h ? 0x0c0c0301u : 0x0c0c0200u;
    f32x16g acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16g{};
    pipe_issue(g, g_pipe0, c.wave, c.lane, c.nb0, c.mb0, c.row_bytes, c.nkb, 0);
    if (c.nst > 1) pipe_issue(g, g_pipe1, c.wave, c.lane, c.nb0, c.mb0, c.row_bytes, c.nkb, 1);
    for (int64_t st = 0; st < c.nst; st += 3) {
        pipe_iter<0, 2>(g, c, st, acc);
        if (st + 1 < c.nst) pipe_iter<1, 0>(g, c, st + 1, acc);
        if (st + 2 < c.nst) pipe_iter<2, 1>(g, c, st + 2, acc);
    }
    const int r = c.r, h = c.h, wn = c.wn, wm = c.wm;
    const int64_t nb0 = c.nb0, mb0 = c.mb0;
    // acc[i][j][4q + e] = C[mb0 + wm 64 + 32 j + r][nb0 + wn 64 + 32 i + 8 q + 4 h + e]
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int64_t m = mb0 + wm * 64 + 32 * j + r;
        if (m >= g.M) continue;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                store_c4(g, m, nb0 + wn * 64 + 32 * i + 8 * q + 4 * h,
                         make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]));
    }
}

// Large-tile pipelined variant (same conditions as the one above): 512
// threads own a 256 (N) x 256 (M) tile, 8 waves as 2 (N) x 4 (M) of 128 x 64
// (4 x 2 instruction tiles, 128 accumulator registers), K 128 per stage in
// three LDS stage buffers of 34 KB.  Twice the matrix-core work per operand
// byte of the 128 x 128 tile and per barrier; each wave still issues 5 loads
// per stage: W and X codes of rows 32 w .. 32 w + 31 (two 16-row loads each)
// and one 64-row scale group (waves 0-3: W, waves 4-7: X).
struct BigBuf {
    uint4 wc[4 * 256];
    uint4 xc[4 * 256];
    uint32_t ws[256];
    uint32_t xs[256];
};

__shared__ BigBuf g_big0, g_big1, g_big2;

constexpr int64_t kBigTileMin = 96;  // 256 x 256 tiles needed before that kernel is chosen

template <int B>
__device__ __forceinline__ BigBuf& big_buf() {
    if constexpr (B == 0) return g_big0;
    else if constexpr (B == 1) return g_big1;
    else return g_big2;
}

__device__ __forceinline__ void big_issue(const GemmParams& g, BigBuf& b, int wave, int lane, int64_t nb0, int64_t mb0,
                                          int64_t row_bytes, int64_t nkb, int64_t st) {
    const int q = lane >> 2;
    const int blk = (lane & 3) ^ ((q >> 2) & 3);
    const int64_t kbyte = (4 * st + blk) * 16;
#pragma unroll
    for (int gr = 0; gr < 2; ++gr) {
        const int grp = 2 * wave + gr;
        const int row = 16 * grp + q;
        const int64_t n = min(nb0 + row, g.N - 1);
        const int64_t m = min(mb0 + row, g.M - 1);
        lds_load16(g.b_codes + n * row_bytes + kbyte, &b.wc[64 * grp]);
        lds_load16(g.a_codes + m * row_bytes + kbyte, &b.xc[64 * grp]);
    }
    if (wave < 4) {
        const int64_t n = min(nb0 + 64 * wave + lane, g.N - 1);
        lds_load4(g.b_scales + n * nkb + 4 * st, &b.ws[64 * wave]);
    } else {
        const int64_t m = min(mb0 + 64 * (wave - 4) + lane, g.M - 1);
        lds_load4(g.a_scales + m * nkb + 4 * st, &b.xs[64 * (wave - 4)]);
    }
}

// A wave's fragments of one stage: both 64-wide K steps of its 4 W and 2 X tiles and their scales.
struct BigFrags {
    uint4 fw[2][4], fx[2][2];
    uint32_t scw[4], scx[2];
};

__device__ __forceinline__ void big_frags(const BigBuf& b, const PipeCtx& c, BigFrags& f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) f.scw[i] = __builtin_amdgcn_perm(0u, b.ws[c.wn * 128 + 32 * i + c.r], c.psel);
#pragma unroll
    for (int j = 0; j < 2; ++j) f.scx[j] = __builtin_amdgcn_perm(0u, b.xs[c.wm * 64 + 32 * j + c.r], c.psel);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
        for (int i = 0; i < 4; ++i) f.fw[s][i] = b.wc[pipe_slot(c.wn * 128 + 32 * i + c.r, 2 * s + c.h)];
#pragma unroll
        for (int j = 0; j < 2; ++j) f.fx[s][j] = b.xc[pipe_slot(c.wm * 64 + 32 * j + c.r, 2 * s + c.h)];
    }
}

template <int STEP>
__device__ __forceinline__ void big_step(const BigFrags& f, f32x16g (&acc)[4][2]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(operand(Frag{f.fw[STEP][i], 0u}),
                                                                         operand(Frag{f.fx[STEP][j], 0u}), acc[i][j], 4,
                                                                         4, STEP, (int)f.scw[i], STEP, (int)f.scx[j]);
}

// All LDS reads of stage st come before stage st + 2 is issued, so the
// vmcnt(0) the compiler still places before LDS reads in one of the three
// unrolled iterations waits only for stage st + 1, already in flight.
template <int CUR, int NXT>
__device__ __forceinline__ void big_iter(const GemmParams& g, const PipeCtx& c, int64_t st, f32x16g (&acc)[4][2]) {
    if (st + 1 < c.nst)
        __builtin_amdgcn_s_waitcnt((kPipeLoadsPerWave & 15) | (7 << 4) | (15 << 8));  // vmcnt(5)
    else
        __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
    __builtin_amdgcn_s_barrier();
    BigFrags f;
    big_frags(big_buf<CUR>(), c, f);
    if (st + 2 < c.nst) big_issue(g, big_buf<NXT>(), c.wave, c.lane, c.nb0, c.mb0, c.row_bytes, c.nkb, st + 2);
    big_step<0>(f, acc);
    big_step<1>(f, acc);
}

__device__ __forceinline__ void big_store(const GemmParams& g, const PipeCtx& c, const f32x16g (&acc)[4][2]) {
    const int r = c.r, h = c.h, wn = c.wn, wm = c.wm;
    // acc[i][j][4q + e] = C[mb0 + wm 64 + 32 j + r][nb0 + wn 128 + 32 i + 8 q + 4 h + e]
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int64_t m = c.mb0 + wm * 64 + 32 * j + r;
        if (m >= g.M) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                store_c4(g, m, c.nb0 + wn * 128 + 32 * i + 8 * q + 4 * h,
                         make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]));
    }
}

// Tile of workgroup (blockIdx.x, blockIdx.y) of a gx x gy grid.  Workgroups
// are dealt to the 8 XCDs round-robin by linear id, so XCD k runs ids
// k, k + 8, ...; those get consecutive logical ids (a bijection for any
// count), and logical ids walk the tiles in groups of 4 M rows (N fastest
// within a group, M fastest within a column), so each XCD's L2 sees a compact
// block of about 4 x (T / 32) tiles instead of every M row.
__device__ __forceinline__ void xcd_tile(int64_t gx, int64_t gy, int64_t& tn, int64_t& tm) {
    const int64_t T = gx * gy;
    const int64_t i = (int64_t)blockIdx.y * gx + blockIdx.x;
    const int64_t k = i % 8, j = i / 8;
    const int64_t L = k * (T / 8) + (k < T % 8 ? k : T % 8) + j;
    constexpr int64_t GM = 4;
    const int64_t gsize = GM * gx;
    const int64_t first_m = (L / gsize) * GM;
    const int64_t gm = gy - first_m < GM ? gy - first_m : GM;
    tm = first_m + (L % gsize) % gm;
    tn = (L % gsize) / gm;
}

__global__ __launch_bounds__(512) void mxfp4_gemm_big_kernel(const GemmParams g) {
    PipeCtx c;
    const int t = threadIdx.x;
    c.wave = __builtin_amdgcn_readfirstlane(t >> 6);  // wave-uniform: LDS bases and row offsets stay scalar
    c.lane = t & 63;
    c.r = c.lane & 31;
    c.h = c.lane >> 5;
    c.wn = c.wave >> 2;
    c.wm = c.wave & 3;
    int64_t tn, tm;
    xcd_tile(gridDim.x, gridDim.y, tn, tm);
    c.nb0 = tn * 256;
    c.mb0 = tm * 256;
    c.nkb = g.K / 32;
    c.row_bytes = g.K / 2;
    c.nst = g.K / 128;
    c.psel = c.h ? 0x0c0c0301u : 0x0c0c0200u;
    f32x16g acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16g{};
    big_issue(g, g_big0, c.wave, c.lane, c.nb0, c.mb0, c.row_bytes, c.nkb, 0);
    if (c.nst > 1) big_issue(g, g_big1, c.wave, c.lane, c.nb0, c.mb0, c.row_bytes, c.nkb, 1);
    for (int64_t st = 0; st < c.nst; st += 3) {
        big_iter<0, 2>(g, c, st, acc);
        if (st + 1 < c.nst) big_iter<1, 0>(g, c, st + 1, acc);
        if (st + 2 < c.nst) big_iter<2, 1>(g, c, st + 2, acc);
    }
    big_store(g, c, acc);
}

hipError_t launch_mxfp4_gemm(const GemmParams& g, hipStream_t st) {
    // the 256 x 256 tile once there are enough of them to spread over the chip, else 128 x 128
    const int64_t big_tiles = ((g.N + 255) / 256) * ((g.M + 255) / 256);
    if (g.K % kGemmTileK == 0 && g.scales_aligned && big_tiles >= kBigTileMin) {
        const dim3 grid((unsigned)((g.N + 255) / 256), (unsigned)((g.M + 255) / 256));
        hipLaunchKernelGGL(mxfp4_gemm_big_kernel, grid, dim3(512), 0, st, g);
    } else if (g.K % kGemmTileK == 0 && g.scales_aligned) {
        const dim3 grid((unsigned)((g.N + 127) / 128), (unsigned)((g.M + 127) / 128));
        hipLaunchKernelGGL(mxfp4_gemm_pipe_kernel, grid, dim3(256), 0, st, g);
    } else {
        const dim3 grid((unsigned)((g.N + 127) / 128), (unsigned)((g.M + 127) / 128));
        hipLaunchKernelGGL(mxfp4_gemm_kernel, grid, dim3(256), 0, st, g);
    }
    return hipGetLastError();
}

}  // namespace kq
