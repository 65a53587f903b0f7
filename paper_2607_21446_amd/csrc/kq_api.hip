// C ABI of libkroquant.so: argument validation, dispatch to the kernels and
// the host-side helpers of the offline weight path.  See include/kroquant.h
// for the contract of every entry point.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdint>
#include <cstdlib>
#include <mutex>
#include <string>
#include <vector>

#include "kq_calib.h"
#include "kq_kernels.h"
#include "kroquant.h"

namespace {

thread_local std::string g_detail;

kq_status fail(kq_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_detail = buf;
    return st;
}

kq_status ok() {
    g_detail.clear();
    return KQ_SUCCESS;
}

kq_status from_hip(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(KQ_ERROR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, uintptr_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

bool supported_split(int a, int b) {
    return (a == 4 && b == 8) || (a == 2 && b == 16) || (a == 8 && b == 4) || (a == 1 && b == 32);
}

// Shape and output checks common to every quantize entry point.
kq_status check_common(const void* X, int64_t M, int64_t d, const void* codes, const void* scales,
                       const void* y, bool codes_required) {
    if (M < 0) return fail(KQ_ERROR_INVALID_VALUE, "M = %lld must be >= 0", (long long)M);
    if (d <= 0 || d % 32 != 0)
        return fail(KQ_ERROR_INVALID_VALUE, "d = %lld must be a positive multiple of 32", (long long)d);
    if (M > 0 && d > INT64_MAX / 4 / M)
        return fail(KQ_ERROR_INVALID_VALUE, "M * d = %lld * %lld is too large", (long long)M, (long long)d);
    if (!X) return fail(KQ_ERROR_NULL_POINTER, "X is NULL");
    if (codes_required && (!codes || !scales))
        return fail(KQ_ERROR_NULL_POINTER, "codes and scales must not be NULL");
    if (!codes_required && ((codes == nullptr) != (scales == nullptr)))
        return fail(KQ_ERROR_NULL_POINTER, "codes and scales must be both NULL or both set");
    if (!aligned(X, 16)) return fail(KQ_ERROR_MISALIGNED, "X must be 16-byte aligned");
    if (codes && !aligned(codes, 16)) return fail(KQ_ERROR_MISALIGNED, "codes must be 16-byte aligned");
    if (y && !aligned(y, 16)) return fail(KQ_ERROR_MISALIGNED, "y_out must be 16-byte aligned");
    return ok();
}

kq::Params make_params(const uint16_t* X, int64_t M, int64_t d, uint8_t* codes, uint8_t* scales, float* y) {
    kq::Params p{};
    p.X = X;
    p.M = M;
    p.d = d;
    p.nb = d / 32;
    p.nblocks = M * (d / 32);
    p.nfac = 1;
    p.codes = codes;
    p.scales = scales;
    p.y = y;
    return p;
}

// fp64 Gauss-Jordan inverse with partial pivoting of an n x n fp32 matrix.
// Returns false if a pivot is below 1e-12 times the infinity norm of its row
// or if the infinity-norm condition number exceeds 1e6.
bool invert(const float* A, int n, double* inv, std::string& why) {
    std::vector<double> m(n * 2 * n, 0.0);
    double norm_a = 0.0;
    for (int i = 0; i < n; ++i) {
        double row = 0.0;
        for (int j = 0; j < n; ++j) {
            m[i * 2 * n + j] = A[i * n + j];
            row += std::fabs((double)A[i * n + j]);
        }
        norm_a = std::max(norm_a, row);
        m[i * 2 * n + n + i] = 1.0;
    }
    for (int c = 0; c < n; ++c) {
        int piv = c;
        for (int r = c + 1; r < n; ++r)
            if (std::fabs(m[r * 2 * n + c]) > std::fabs(m[piv * 2 * n + c])) piv = r;
        double rownorm = 0.0;
        for (int j = 0; j < n; ++j) rownorm = std::max(rownorm, std::fabs(m[piv * 2 * n + j]));
        const double pv = m[piv * 2 * n + c];
        if (!(std::fabs(pv) > 1e-12 * rownorm)) {
            why = "zero or tiny pivot";
            return false;
        }
        if (piv != c)
            for (int j = 0; j < 2 * n; ++j) std::swap(m[c * 2 * n + j], m[piv * 2 * n + j]);
        for (int j = 0; j < 2 * n; ++j) m[c * 2 * n + j] /= pv;
        for (int r = 0; r < n; ++r) {
            if (r == c) continue;
            const double f = m[r * 2 * n + c];
            if (f == 0.0) continue;
            for (int j = 0; j < 2 * n; ++j) m[r * 2 * n + j] -= f * m[c * 2 * n + j];
        }
    }
    double norm_i = 0.0;
    for (int i = 0; i < n; ++i) {
        double row = 0.0;
        for (int j = 0; j < n; ++j) {
            inv[i * n + j] = m[i * 2 * n + n + j];
            row += std::fabs(inv[i * n + j]);
        }
        norm_i = std::max(norm_i, row);
    }
    if (!(norm_a * norm_i <= 1e6)) {
        why = "condition number above 1e6";
        return false;
    }
    return true;
}

kq_status inverse_transpose(const float* F, int n, int64_t nfac, float* out, const char* name) {
    std::vector<double> inv(n * n);
    std::string why;
    for (int64_t f = 0; f < nfac; ++f) {
        if (!invert(F + f * n * n, n, inv.data(), why))
            return fail(KQ_ERROR_SINGULAR, "%s[%lld]: %s", name, (long long)f, why.c_str());
        for (int i = 0; i < n; ++i)
            for (int j = 0; j < n; ++j) out[f * n * n + i * n + j] = (float)inv[j * n + i];
    }
    return ok();
}

kq_status check_factors(int a, int b, int64_t nfac, int64_t d) {
    if (!supported_split(a, b))
        return fail(KQ_ERROR_UNSUPPORTED, "(a, b) = (%d, %d) is not one of (4,8), (2,16), (8,4), (1,32)", a, b);
    if (nfac != 1 && nfac != d / 32)
        return fail(KQ_ERROR_UNSUPPORTED, "nfac = %lld must be 1 or d/32 = %lld", (long long)nfac,
                    (long long)(d / 32));
    // per-block factors run the column-mapped kernels, whose offsets within
    // a 64-row unit are 32-bit
    if (nfac > 1 && d >= (int64_t(1) << 25))
        return fail(KQ_ERROR_UNSUPPORTED, "per-block factors (nfac = d/32) need d < 2^25, got d = %lld",
                    (long long)d);
    return ok();
}

// The matrix-core kernels launch one workgroup per 64-block unit (shared
// factors) or per 64-row x 8-column-block tile (per-block factors); both
// counts must fit one launch (2^31 - 1 workgroups, i.e. more than 2^42
// elements of X).
kq_status check_grid(int64_t M, int64_t d, int64_t nfac) {
    const int64_t nb = d / 32;
    const int64_t groups = nfac == 1 ? (M / 64) * nb + ((M % 64) * nb + 63) / 64
                                     : ((M + 63) / 64) * ((nb + 7) / 8);
    if (groups > kq::kMaxUnitGrid)
        return fail(KQ_ERROR_UNSUPPORTED, "M = %lld, d = %lld needs %lld workgroups, more than one launch holds",
                    (long long)M, (long long)d, (long long)groups);
    return ok();
}

}  // namespace

extern "C" {

static kq_status quantize_kron(kq::Kind kind, const char* name, const uint16_t* X, int64_t M, int64_t d,
                               const float* A, const float* B, int a, int b, int64_t nfac, const void* kpack,
                               uint8_t* codes, uint8_t* scales, float* y_out, void* stream) {
    kq_status st = check_common(X, M, d, codes, scales, y_out, true);
    if (st != KQ_SUCCESS) return st;
    if ((st = check_factors(a, b, nfac, d)) != KQ_SUCCESS) return st;
    if (!A || !B) return fail(KQ_ERROR_NULL_POINTER, "A and B must not be NULL");
    if (!aligned(A, 4) || !aligned(B, 4)) return fail(KQ_ERROR_MISALIGNED, "A and B must be 4-byte aligned");
    if (kpack && !aligned(kpack, 16)) return fail(KQ_ERROR_MISALIGNED, "kpack must be 16-byte aligned");
    if (M == 0) return ok();
    if (kind != kq::Kind::Kron && (st = check_grid(M, d, nfac)) != KQ_SUCCESS) return st;
    kq::Params p = make_params(X, M, d, codes, scales, y_out);
    p.A = A;
    p.B = B;
    p.nfac = nfac;
    p.kpack = static_cast<const uint8_t*>(kpack);
    const kq::Mapping map = (nfac == 1) ? kq::Mapping::Flat : kq::Mapping::Column;
    return from_hip(kq::launch(kind, a, p, map, (hipStream_t)stream), name);
}

kq_status kq_quantize(const uint16_t* X, int64_t M, int64_t d, const float* A, const float* B, int a,
                      int b, int64_t nfac, uint8_t* codes, uint8_t* scales, float* y_out, void* stream) {
    return quantize_kron(kq::Kind::KronMfma, "kq_quantize", X, M, d, A, B, a, b, nfac, nullptr, codes, scales,
                         y_out, stream);
}

kq_status kq_quantize_packed(const uint16_t* X, int64_t M, int64_t d, const float* A, const float* B, int a,
                             int b, int64_t nfac, const void* kpack, uint8_t* codes, uint8_t* scales, float* y_out,
                             void* stream) {
    if (!kpack) return fail(KQ_ERROR_NULL_POINTER, "kpack must not be NULL");
    return quantize_kron(kq::Kind::KronMfma, "kq_quantize_packed", X, M, d, A, B, a, b, nfac, kpack, codes,
                         scales, y_out, stream);
}

kq_status kq_quantize_lu(const uint16_t* X, int64_t M, int64_t d, const float* lu, int a, int64_t nfac,
                         uint8_t* codes, uint8_t* scales, float* y_out, uint16_t* y16_out, void* stream) {
    kq_status st = check_common(X, M, d, codes, scales, y_out, true);
    if (st != KQ_SUCCESS) return st;
    if (a != 1 && a != 2 && a != 4 && a != 8)
        return fail(KQ_ERROR_UNSUPPORTED, "a = %d must be 1, 2, 4 or 8 (the number of G factors in A is log2 a)", a);
    if ((st = check_factors(a, 32 / a, nfac, d)) != KQ_SUCCESS) return st;
    if (!lu) return fail(KQ_ERROR_NULL_POINTER, "lu must not be NULL");
    if (!aligned(lu, 4)) return fail(KQ_ERROR_MISALIGNED, "lu must be 4-byte aligned");
    if (y16_out && !aligned(y16_out, 16)) return fail(KQ_ERROR_MISALIGNED, "y16_out must be 16-byte aligned");
    if (M == 0) return ok();
    if ((st = check_grid(M, d, nfac)) != KQ_SUCCESS) return st;
    kq::Params p = make_params(X, M, d, codes, scales, y_out);
    p.nfac = nfac;
    p.lu = lu;
    p.y16 = y16_out;
    const kq::Mapping map = (nfac == 1) ? kq::Mapping::Flat : kq::Mapping::Column;
    return from_hip(kq::launch(kq::Kind::KronLU, a, p, map, (hipStream_t)stream), "kq_quantize_lu");
}

kq_status kq_pack_factors(const float* A, const float* B, int a, int b, int64_t nfac, void* kpack, void* stream) {
    if (!supported_split(a, b))
        return fail(KQ_ERROR_UNSUPPORTED, "(a, b) = (%d, %d) is not one of (4,8), (2,16), (8,4), (1,32)", a, b);
    if (nfac < 1) return fail(KQ_ERROR_INVALID_VALUE, "nfac = %lld must be >= 1", (long long)nfac);
    if (!A || !B || !kpack) return fail(KQ_ERROR_NULL_POINTER, "A, B and kpack must not be NULL");
    if (!aligned(A, 4) || !aligned(B, 4)) return fail(KQ_ERROR_MISALIGNED, "A and B must be 4-byte aligned");
    if (!aligned(kpack, 16)) return fail(KQ_ERROR_MISALIGNED, "kpack must be 16-byte aligned");
    return from_hip(kq::launch_pack(a, A, B, nfac, static_cast<uint8_t*>(kpack), (hipStream_t)stream),
                    "kq_pack_factors");
}

kq_status kq_quantize_exact(const uint16_t* X, int64_t M, int64_t d, const float* A, const float* B, int a,
                            int b, int64_t nfac, uint8_t* codes, uint8_t* scales, float* y_out, void* stream) {
    return quantize_kron(kq::Kind::Kron, "kq_quantize_exact", X, M, d, A, B, a, b, nfac, nullptr, codes, scales,
                         y_out, stream);
}

kq_status kq_smoothquant_quantize(const uint16_t* X, int64_t M, int64_t d, const float* mult, uint8_t* codes,
                                  uint8_t* scales, float* y_out, void* stream) {
    kq_status st = check_common(X, M, d, codes, scales, y_out, true);
    if (st != KQ_SUCCESS) return st;
    if (!mult) return fail(KQ_ERROR_NULL_POINTER, "mult must not be NULL");
    if (!aligned(mult, 16)) return fail(KQ_ERROR_MISALIGNED, "mult must be 16-byte aligned");
    if (M == 0) return ok();
    kq::Params p = make_params(X, M, d, codes, scales, y_out);
    p.mult = mult;
    return from_hip(kq::launch(kq::Kind::Smooth, 0, p, kq::Mapping::Flat, (hipStream_t)stream),
                    "kq_smoothquant_quantize");
}

kq_status kq_hadamard32_quantize(const uint16_t* X, int64_t M, int64_t d, uint8_t* codes, uint8_t* scales,
                                 float* y_out, void* stream) {
    kq_status st = check_common(X, M, d, codes, scales, y_out, true);
    if (st != KQ_SUCCESS) return st;
    if (M == 0) return ok();
    kq::Params p = make_params(X, M, d, codes, scales, y_out);
    return from_hip(kq::launch(kq::Kind::Hadamard, 0, p, kq::Mapping::Flat, (hipStream_t)stream),
                    "kq_hadamard32_quantize");
}

kq_status kq_fwht_quantize(const uint16_t* X, int64_t M, int64_t d, uint8_t* codes, uint8_t* scales,
                           float* y_out, void* stream) {
    kq_status st = check_common(X, M, d, codes, scales, y_out, true);
    if (st != KQ_SUCCESS) return st;
    if (d > 16384 || (d & (d - 1)) != 0)
        return fail(KQ_ERROR_UNSUPPORTED, "d = %lld must be a power of two from 32 to 16384", (long long)d);
    if (M == 0) return ok();
    kq::Params p = make_params(X, M, d, codes, scales, y_out);
    return from_hip(kq::launch_fwht(p, (hipStream_t)stream), "kq_fwht_quantize");
}

kq_status kq_stream_floor(const uint16_t* X, int64_t M, int64_t d, uint8_t* out16, uint8_t* out1, void* stream) {
    kq_status st = check_common(X, M, d, out16, out1, nullptr, true);
    if (st != KQ_SUCCESS) return st;
    if (M == 0) return ok();
    kq::Params p = make_params(X, M, d, out16, out1, nullptr);
    if (p.nblocks / 64 >= (int64_t)1 << 31)
        return fail(KQ_ERROR_INVALID_VALUE, "M * d = %lld * %lld is too large for one launch", (long long)M, (long long)d);
    return from_hip(kq::launch_stream_floor(p, (hipStream_t)stream), "kq_stream_floor");
}

kq_status kq_stream_probe(const uint16_t* X, int64_t M, int64_t d, uint8_t* out16, uint8_t* out1,
                          int waves_per_group, int units_per_wave, int64_t groups, void* stream) {
    kq_status st = check_common(X, M, d, out16, out1, nullptr, true);
    if (st != KQ_SUCCESS) return st;
    const int w = waves_per_group, u = units_per_wave;
    if (w != 1 && w != 2 && w != 4 && w != 8 && w != 16)
        return fail(KQ_ERROR_INVALID_VALUE, "waves_per_group = %d must be 1, 2, 4, 8 or 16", w);
    if (u != 1 && u != 2 && u != 4) return fail(KQ_ERROR_INVALID_VALUE, "units_per_wave = %d must be 1, 2 or 4", u);
    if (groups < 0 || groups > kq::kMaxUnitGrid)
        return fail(KQ_ERROR_INVALID_VALUE, "groups = %lld must be in [0, 2^31 - 1]", (long long)groups);
    if (M == 0) return ok();
    kq::Params p = make_params(X, M, d, out16, out1, nullptr);
    if (groups == 0 && ((p.nblocks + 63) / 64 + (int64_t)w * u - 1) / ((int64_t)w * u) > kq::kMaxUnitGrid)
        return fail(KQ_ERROR_INVALID_VALUE, "M * d = %lld * %lld is too large for one pass", (long long)M, (long long)d);
    return from_hip(kq::launch_stream_probe(p, w, u, groups, (hipStream_t)stream), "kq_stream_probe");
}

kq_status kq_timestamp(uint64_t* dst, void* stream) {
    if (!dst) return fail(KQ_ERROR_NULL_POINTER, "dst is null");
    if (!aligned(dst, 8)) return fail(KQ_ERROR_MISALIGNED, "dst must be 8-byte aligned");
    return from_hip(kq::launch_timestamp(dst, (hipStream_t)stream), "kq_timestamp");
}

static kq::GemmParams gemm_params(const uint8_t* a_codes, const uint8_t* a_scales, int64_t M, const uint8_t* b_codes,
                                  const uint8_t* b_scales, int64_t N, int64_t K, float* C, int64_t ldc, int accumulate,
                                  const float* bias) {
    kq::GemmParams g{};
    g.a_codes = a_codes;
    g.a_scales = a_scales;
    g.M = M;
    g.b_codes = b_codes;
    g.b_scales = b_scales;
    g.N = N;
    g.K = K;
    g.C = C;
    g.ldc_out = ldc;
    g.accumulate = accumulate;
    g.bias = bias;
    g.vec_ok = aligned(C, 16) && ldc % 4 == 0 && (!bias || aligned(bias, 16));
    g.scales_aligned = aligned(a_scales, 4) && aligned(b_scales, 4);
    return g;
}

static kq_status check_gemm(const uint8_t* a_codes, const uint8_t* a_scales, int64_t M, const uint8_t* b_codes,
                            const uint8_t* b_scales, int64_t N, int64_t K, const void* C, int64_t ldc, int accumulate,
                            size_t c_align) {
    if (M < 0 || N < 0) return fail(KQ_ERROR_INVALID_VALUE, "M = %lld and N = %lld must be >= 0", (long long)M, (long long)N);
    if (K <= 0 || K % 32 != 0) return fail(KQ_ERROR_INVALID_VALUE, "K = %lld must be a positive multiple of 32", (long long)K);
    if (ldc < N) return fail(KQ_ERROR_INVALID_VALUE, "ldc = %lld must be >= N = %lld", (long long)ldc, (long long)N);
    if (accumulate != 0 && accumulate != 1) return fail(KQ_ERROR_INVALID_VALUE, "accumulate must be 0 or 1");
    if ((M + 127) / 128 > 65535 || (N + 127) / 128 > 2147483647)
        return fail(KQ_ERROR_INVALID_VALUE, "M = %lld is too large (at most 65535 * 128 rows)", (long long)M);
    if (M == 0 || N == 0) return ok();
    if (!a_codes || !a_scales || !b_codes || !b_scales || !C)
        return fail(KQ_ERROR_NULL_POINTER, "codes, scales and C must not be NULL");
    if (!aligned(a_codes, 16) || !aligned(b_codes, 16)) return fail(KQ_ERROR_MISALIGNED, "codes must be 16-byte aligned");
    if (!aligned(C, c_align)) return fail(KQ_ERROR_MISALIGNED, "C must be %zu-byte aligned", c_align);
    return ok();
}

kq_status kq_mxfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, int64_t M, const uint8_t* b_codes,
                        const uint8_t* b_scales, int64_t N, int64_t K, float* C, int64_t ldc, int accumulate,
                        void* stream) {
    const kq_status st = check_gemm(a_codes, a_scales, M, b_codes, b_scales, N, K, C, ldc, accumulate, 4);
    if (st != KQ_SUCCESS || M == 0 || N == 0) return st;
    const kq::GemmParams g = gemm_params(a_codes, a_scales, M, b_codes, b_scales, N, K, C, ldc, accumulate, nullptr);
    return from_hip(kq::launch_mxfp4_gemm(g, (hipStream_t)stream), "kq_mxfp4_gemm");
}

kq_status kq_mxfp4_gemm_bf16(const uint8_t* a_codes, const uint8_t* a_scales, int64_t M, const uint8_t* b_codes,
                             const uint8_t* b_scales, int64_t N, int64_t K, uint16_t* C, int64_t ldc, void* stream) {
    const kq_status st = check_gemm(a_codes, a_scales, M, b_codes, b_scales, N, K, C, ldc, 0, 2);
    if (st != KQ_SUCCESS || M == 0 || N == 0) return st;
    kq::GemmParams g = gemm_params(a_codes, a_scales, M, b_codes, b_scales, N, K, nullptr, ldc, 0, nullptr);
    g.C16 = C;
    g.vec_ok = aligned(C, 8) && ldc % 4 == 0;
    return from_hip(kq::launch_mxfp4_gemm(g, (hipStream_t)stream), "kq_mxfp4_gemm_bf16");
}

kq_status kq_mxfp4_quantize(const uint16_t* X, int64_t M, int64_t d, uint8_t* codes, uint8_t* scales,
                            void* stream) {
    kq_status st = check_common(X, M, d, codes, scales, nullptr, true);
    if (st != KQ_SUCCESS) return st;
    if (M == 0) return ok();
    kq::Params p = make_params(X, M, d, codes, scales, nullptr);
    return from_hip(kq::launch(kq::Kind::Plain, 0, p, kq::Mapping::Flat, (hipStream_t)stream),
                    "kq_mxfp4_quantize");
}

kq_status kq_e2m1_encode(const float* v, int64_t n, int s, uint8_t* codes, void* stream) {
    if (n < 0 || n % 2 != 0) return fail(KQ_ERROR_INVALID_VALUE, "n = %lld must be even and >= 0", (long long)n);
    if (s < 0 || s > 254) return fail(KQ_ERROR_INVALID_VALUE, "s = %d must be in [0, 254]", s);
    if (n == 0) return ok();
    if (!v || !codes) return fail(KQ_ERROR_NULL_POINTER, "v and codes must not be NULL");
    if (!aligned(v, 8)) return fail(KQ_ERROR_MISALIGNED, "v must be 8-byte aligned");
    return from_hip(kq::launch_e2m1(v, n / 2, (uint32_t)s, codes, (hipStream_t)stream), "kq_e2m1_encode");
}

kq_status kq_factors_inverse_transpose(const float* A, const float* B, int a, int b, int64_t nfac, float* A_it,
                                       float* B_it) {
    if (!supported_split(a, b))
        return fail(KQ_ERROR_UNSUPPORTED, "(a, b) = (%d, %d) is not one of (4,8), (2,16), (8,4), (1,32)", a, b);
    if (nfac < 1) return fail(KQ_ERROR_INVALID_VALUE, "nfac = %lld must be >= 1", (long long)nfac);
    if (!A || !B || !A_it || !B_it) return fail(KQ_ERROR_NULL_POINTER, "factor pointers must not be NULL");
    kq_status st = inverse_transpose(A, a, nfac, A_it, "A");
    if (st != KQ_SUCCESS) return st;
    return inverse_transpose(B, b, nfac, B_it, "B");
}

kq_status kq_weight_transform(const uint16_t* W, int64_t o, int64_t d, const float* A_host, const float* B_host,
                              int a, int b, int64_t nfac, float* W_out, uint8_t* codes, uint8_t* scales,
                              void* stream) {
    kq_status st = check_common(W, o, d, codes, scales, W_out, false);
    if (st != KQ_SUCCESS) return st;
    if ((st = check_factors(a, b, nfac, d)) != KQ_SUCCESS) return st;
    if (!W_out) return fail(KQ_ERROR_NULL_POINTER, "W_out must not be NULL");
    if (!A_host || !B_host) return fail(KQ_ERROR_NULL_POINTER, "A_host and B_host must not be NULL");
    std::vector<float> Ait(nfac * a * a), Bit(nfac * b * b);
    if ((st = inverse_transpose(A_host, a, nfac, Ait.data(), "A")) != KQ_SUCCESS) return st;
    if ((st = inverse_transpose(B_host, b, nfac, Bit.data(), "B")) != KQ_SUCCESS) return st;
    if (o == 0) return ok();
    hipStream_t s = (hipStream_t)stream;
    const size_t bytesA = Ait.size() * sizeof(float), bytesB = Bit.size() * sizeof(float);
    float* dev = nullptr;
    hipError_t e = hipMalloc(&dev, bytesA + bytesB);
    if (e != hipSuccess) return from_hip(e, "kq_weight_transform: hipMalloc");
    e = hipMemcpyAsync(dev, Ait.data(), bytesA, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(dev + Ait.size(), Bit.data(), bytesB, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) {
        kq::Params p = make_params(W, o, d, codes, scales, W_out);
        p.A = dev;
        p.B = dev + Ait.size();
        p.nfac = nfac;
        const kq::Mapping map = (nfac == 1) ? kq::Mapping::Flat : kq::Mapping::Column;
        e = kq::launch(kq::Kind::Kron, a, p, map, s);
    }
    // the host vectors and the device buffer must outlive the queued work
    const hipError_t es = hipStreamSynchronize(s);
    if (e == hipSuccess) e = es;
    const hipError_t ef = hipFree(dev);
    if (e == hipSuccess) e = ef;
    return from_hip(e, "kq_weight_transform");
}

kq_status kq_lu_to_factors(const float* abc, int a, int64_t nfac, float* A, float* B) {
    if (a != 1 && a != 2 && a != 4 && a != 8) return fail(KQ_ERROR_UNSUPPORTED, "a = %d must be 1, 2, 4 or 8", a);
    if (nfac < 1) return fail(KQ_ERROR_INVALID_VALUE, "nfac = %lld must be >= 1", (long long)nfac);
    if (!abc || !A || !B) return fail(KQ_ERROR_NULL_POINTER, "abc, A and B must not be NULL");
    const int b = 32 / a;
    const int na = (a == 1) ? 0 : (a == 2) ? 1 : (a == 4) ? 2 : 3;
    for (int64_t f = 0; f < nfac; ++f) {
        double G[5][2][2];
        for (int k = 0; k < 5; ++k) {
            const double ak = abc[f * 15 + 3 * k], bk = abc[f * 15 + 3 * k + 1], ck = abc[f * 15 + 3 * k + 2];
            if (ak == 0.0) return fail(KQ_ERROR_SINGULAR, "block %lld: a_%d = 0", (long long)f, k + 1);
            // L = [[1,0],[c,1]], U = [[a,b],[0,-1/a]]:  G = L U
            G[k][0][0] = ak;
            G[k][0][1] = bk;
            G[k][1][0] = ck * ak;
            G[k][1][1] = ck * bk - 1.0 / ak;
        }
        // Kronecker entries: (G_1 (x) .. (x) G_n)[r][c] = prod_k G_k[bit_(n-k)(r)][bit_(n-k)(c)];
        // the library factors are the transposes (A (x) B = K^T).
        for (int r = 0; r < a; ++r)
            for (int c = 0; c < a; ++c) {
                double v = 1.0;
                for (int k = 0; k < na; ++k) {
                    const int sh = na - 1 - k;
                    v *= G[k][(r >> sh) & 1][(c >> sh) & 1];
                }
                A[f * a * a + c * a + r] = (float)v;
            }
        const int nbits = 5 - na;
        for (int r = 0; r < b; ++r)
            for (int c = 0; c < b; ++c) {
                double v = 1.0;
                for (int k = 0; k < nbits; ++k) {
                    const int sh = nbits - 1 - k;
                    v *= G[na + k][(r >> sh) & 1][(c >> sh) & 1];
                }
                B[f * b * b + c * b + r] = (float)v;
            }
    }
    return ok();
}

// ------------------------------------------------ layer-wise calibration

static kq_status check_calib(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o, int a,
                             int64_t nfac) {
    if (R < 1 || o < 1) return fail(KQ_ERROR_INVALID_VALUE, "R = %lld and o = %lld must be >= 1", (long long)R,
                                    (long long)o);
    if (d <= 0 || d % 32 != 0)
        return fail(KQ_ERROR_INVALID_VALUE, "d = %lld must be a positive multiple of 32", (long long)d);
    if (R > int64_t(65535) * 128 || o > int64_t(65535) * 64 || d > int64_t(65535) * 64)
        return fail(KQ_ERROR_INVALID_VALUE, "R must be at most 65535 * 128, o and d at most 65535 * 64");
    if (R > INT64_MAX / 4 / std::max(d, o) || o > INT64_MAX / 4 / d)
        return fail(KQ_ERROR_INVALID_VALUE, "R, o, d = %lld, %lld, %lld are too large", (long long)R, (long long)o,
                    (long long)d);
    if (a != 1 && a != 2 && a != 4 && a != 8) return fail(KQ_ERROR_UNSUPPORTED, "a = %d must be 1, 2, 4 or 8", a);
    if (nfac != 1 && nfac != d / 32)
        return fail(KQ_ERROR_UNSUPPORTED, "nfac = %lld must be 1 or d / 32 = %lld", (long long)nfac,
                    (long long)(d / 32));
    if (!X || !W) return fail(KQ_ERROR_NULL_POINTER, "X and W must not be NULL");
    if (!aligned(X, 16) || !aligned(W, 16)) return fail(KQ_ERROR_MISALIGNED, "X and W must be 16-byte aligned");
    return ok();
}

kq_status kq_calib_workspace_size(int64_t R, int64_t o, int64_t d, int a, int64_t nfac, size_t* bytes) {
    if (!bytes) return fail(KQ_ERROR_NULL_POINTER, "bytes is NULL");
    static const uint16_t dummy[8] __attribute__((aligned(16))) = {0};
    const kq_status st = check_calib(dummy, R, d, dummy, o, a, nfac);
    if (st != KQ_SUCCESS) return st;
    *bytes = kq::calib_plan(R, o, d, a, nfac).total;
    return ok();
}

kq_status kq_calib_reference(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o, float* Yneg,
                             void* stream) {
    const kq_status st = check_calib(X, R, d, W, o, 4, 1);
    if (st != KQ_SUCCESS) return st;
    if (!Yneg) return fail(KQ_ERROR_NULL_POINTER, "Yneg is NULL");
    if (!aligned(Yneg, 4)) return fail(KQ_ERROR_MISALIGNED, "Yneg must be 4-byte aligned");
    return from_hip(kq::launch_calib_reference(X, R, d, W, o, Yneg, (hipStream_t)stream), "kq_calib_reference");
}

// Forward products of one step into the workspace, then the backward pass.
static kq_status calib_step_impl(const kq::CalibPlan& pl, const uint16_t* X, const uint16_t* W, const float* Yneg,
                                 float* lu, const float* lambdas, float* grad, double* losses, float* adam_m,
                                 float* adam_v, int adam_t, float lr, unsigned char* ws, hipStream_t s) {
    const int a = pl.a, b = 32 / a;
    float* fa = reinterpret_cast<float*>(ws + pl.fa);
    float* fb = reinterpret_cast<float*>(ws + pl.fb);
    hipError_t e = kq::launch_calib_inverse_factors(lu, a, pl.nfac, fa, fb, s);
    if (e != hipSuccess) return from_hip(e, "kq_calib_step (inverse factors)");
    kq_status st = kq_quantize_lu(X, pl.R, pl.d, lu, a, pl.nfac, ws + pl.cA, ws + pl.sA,
                                  reinterpret_cast<float*>(ws + pl.yA), nullptr, s);
    if (st != KQ_SUCCESS) return st;
    st = kq_quantize(W, pl.o, pl.d, fa, fb, a, b, pl.nfac, ws + pl.cW, ws + pl.sW,
                     reinterpret_cast<float*>(ws + pl.yW), s);
    if (st != KQ_SUCCESS) return st;
    // residual Q(X T) Q(W T^-T)^T - X W^T on the W4A4 GEMM with Yneg as its bias
    float* res = reinterpret_cast<float*>(ws + pl.res);
    const kq::GemmParams g =
        gemm_params(ws + pl.cA, ws + pl.sA, pl.R, ws + pl.cW, ws + pl.sW, pl.o, pl.d, res, pl.o, 0, Yneg);
    e = kq::launch_mxfp4_gemm(g, s);
    if (e != hipSuccess) return from_hip(e, "kq_calib_step (residual)");
    kq::CalibStepArgs args{X, W, lu, lambdas, grad, losses, lu, adam_m, adam_v, adam_t, lr, ws};
    return from_hip(kq::launch_calib_backward(pl, args, s), "kq_calib_step (backward)");
}

static kq_status check_workspace(const kq::CalibPlan& pl, const void* ws, size_t ws_bytes) {
    if (!ws) return fail(KQ_ERROR_NULL_POINTER, "workspace is NULL");
    if (!aligned(ws, 256)) return fail(KQ_ERROR_MISALIGNED, "workspace must be 256-byte aligned");
    if (ws_bytes < pl.total)
        return fail(KQ_ERROR_INVALID_VALUE, "workspace_bytes = %zu, need %zu", ws_bytes, pl.total);
    return ok();
}

// Argument checks of one calibration step (everything but the workspace).
static kq_status check_step(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o, const float* Yneg,
                            const float* lu, int a, int64_t nfac, const float* lambdas, const float* grad,
                            const double* losses, const float* adam_m, const float* adam_v, int adam_t) {
    kq_status st = check_calib(X, R, d, W, o, a, nfac);
    if (st != KQ_SUCCESS) return st;
    if (!Yneg || !lu || !lambdas || !grad || !losses)
        return fail(KQ_ERROR_NULL_POINTER, "Yneg, lu, lambdas, grad and losses must not be NULL");
    if (!aligned(Yneg, 16) || !aligned(lu, 4) || !aligned(lambdas, 4) || !aligned(grad, 4) || !aligned(losses, 8))
        return fail(KQ_ERROR_MISALIGNED, "Yneg must be 16-byte, losses 8-byte and lu, lambdas, grad 4-byte aligned");
    if (adam_t < 0) return fail(KQ_ERROR_INVALID_VALUE, "adam_t = %d must be >= 0", adam_t);
    if (adam_t > 0 && (!adam_m || !adam_v))
        return fail(KQ_ERROR_NULL_POINTER, "adam_m and adam_v must not be NULL when adam_t > 0");
    if (adam_t > 0 && (!aligned(adam_m, 4) || !aligned(adam_v, 4)))
        return fail(KQ_ERROR_MISALIGNED, "adam_m and adam_v must be 4-byte aligned");
    return ok();
}

kq_status kq_calib_step(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o, const float* Yneg,
                        float* lu, int a, int64_t nfac, const float* lambdas, float* grad, double* losses,
                        float* adam_m, float* adam_v, int adam_t, float lr, void* workspace,
                        size_t workspace_bytes, void* stream) {
    kq_status st = check_step(X, R, d, W, o, Yneg, lu, a, nfac, lambdas, grad, losses, adam_m, adam_v, adam_t);
    if (st != KQ_SUCCESS) return st;
    const kq::CalibPlan pl = kq::calib_plan(R, o, d, a, nfac);
    st = check_workspace(pl, workspace, workspace_bytes);
    if (st != KQ_SUCCESS) return st;
    return calib_step_impl(pl, X, W, Yneg, lu, lambdas, grad, losses, adam_m, adam_v, adam_t, lr,
                           static_cast<unsigned char*>(workspace), (hipStream_t)stream);
}

}  // extern "C"

// Device-resident scratch of kq_calib_step_noalloc: one copy per GPU, held
// until the process ends.  Host code never passes `calib_scratch` itself (on
// the host that name is a stand-in, not a device address): the device address
// of each GPU's copy comes from hipGetSymbolAddress, taken once per device
// with that device current, and only that address reaches the kernels.
static __device__ __align__(256) unsigned char calib_scratch[KQ_CALIB_NOALLOC_MAX_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of the current device's calib_scratch (looked up on the
// first call on that device).
kq_status scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return from_hip(e, "kq_calib_step_noalloc: hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(KQ_ERROR_UNSUPPORTED, "kq_calib_step_noalloc: device %d is beyond the %d devices supported", dev,
                    kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(calib_scratch));
        if (e != hipSuccess) return from_hip(e, "kq_calib_step_noalloc: hipGetSymbolAddress");
        if (!ptr || !aligned(ptr, 256))
            return fail(KQ_ERROR_HIP, "kq_calib_step_noalloc: unusable scratch address %p", ptr);
        g_scratch[dev] = ptr;
    }
    *out = g_scratch[dev];
    return ok();
}

}  // namespace

extern "C" {

kq_status kq_calib_step_noalloc(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o,
                                const float* Yneg, float* lu, int a, int64_t nfac, const float* lambdas, float* grad,
                                double* losses, float* adam_m, float* adam_v, int adam_t, float lr, void* stream) {
    kq_status st = check_step(X, R, d, W, o, Yneg, lu, a, nfac, lambdas, grad, losses, adam_m, adam_v, adam_t);
    if (st != KQ_SUCCESS) return st;
    const kq::CalibPlan pl = kq::calib_plan(R, o, d, a, nfac);
    if (pl.total > (size_t)KQ_CALIB_NOALLOC_MAX_BYTES)
        return fail(KQ_ERROR_INVALID_VALUE,
                    "kq_calib_step_noalloc: these sizes need %zu bytes of scratch, more than the %zu it holds "
                    "(use kq_calib_step with a workspace)", pl.total, (size_t)KQ_CALIB_NOALLOC_MAX_BYTES);
    void* ws = nullptr;
    if ((st = scratch_address(&ws)) != KQ_SUCCESS) return st;
    // every buffer of the plan is written before it is read within the step,
    // so the previous call's contents need no clearing
    return calib_step_impl(pl, X, W, Yneg, lu, lambdas, grad, losses, adam_m, adam_v, adam_t, lr,
                           static_cast<unsigned char*>(ws), (hipStream_t)stream);
}

kq_status kq_calibrate(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o, const float* Yneg,
                       float* lu, int a, int64_t nfac, int steps, float lr, double* losses, void* workspace,
                       size_t workspace_bytes, void* stream) {
    kq_status st = check_calib(X, R, d, W, o, a, nfac);
    if (st != KQ_SUCCESS) return st;
    if (steps < 0) return fail(KQ_ERROR_INVALID_VALUE, "steps = %d must be >= 0", steps);
    if (!Yneg || !lu || !losses) return fail(KQ_ERROR_NULL_POINTER, "Yneg, lu and losses must not be NULL");
    if (!aligned(Yneg, 16) || !aligned(lu, 4) || !aligned(losses, 8))
        return fail(KQ_ERROR_MISALIGNED, "Yneg must be 16-byte, losses 8-byte and lu 4-byte aligned");
    const kq::CalibPlan pl = kq::calib_plan(R, o, d, a, nfac);
    st = check_workspace(pl, workspace, workspace_bytes);
    if (st != KQ_SUCCESS) return st;
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    const hipStream_t s = (hipStream_t)stream;
    float* lam = reinterpret_cast<float*>(ws + pl.lam);
    float* am = reinterpret_cast<float*>(ws + pl.am);
    float* av = reinterpret_cast<float*>(ws + pl.av);
    float* grad = reinterpret_cast<float*>(ws + pl.grad);
    hipError_t e = kq::launch_calib_init(am, av, pl.nfac * 15, lam, s);
    if (e != hipSuccess) return from_hip(e, "kq_calibrate (init)");
    // losses at the initial transform, with lambda = 0, set the automatic weights
    st = calib_step_impl(pl, X, W, Yneg, lu, lam, grad, losses, am, av, 0, lr, ws, s);
    if (st != KQ_SUCCESS) return st;
    e = kq::launch_calib_set_lambdas(losses, lam, s);
    if (e != hipSuccess) return from_hip(e, "kq_calibrate (lambdas)");
    for (int t = 1; t <= steps; ++t) {
        st = calib_step_impl(pl, X, W, Yneg, lu, lam, grad, losses + 4 * int64_t(t), am, av, t, lr, ws, s);
        if (st != KQ_SUCCESS) return st;
    }
    // losses of the final transform
    return calib_step_impl(pl, X, W, Yneg, lu, lam, grad, losses + 4 * (int64_t(steps) + 1), am, av, 0, lr, ws, s);
}

const char* kq_status_string(kq_status s) {
    switch (s) {
        case KQ_SUCCESS: return "KQ_SUCCESS";
        case KQ_ERROR_INVALID_VALUE: return "KQ_ERROR_INVALID_VALUE";
        case KQ_ERROR_NULL_POINTER: return "KQ_ERROR_NULL_POINTER";
        case KQ_ERROR_MISALIGNED: return "KQ_ERROR_MISALIGNED";
        case KQ_ERROR_UNSUPPORTED: return "KQ_ERROR_UNSUPPORTED";
        case KQ_ERROR_SINGULAR: return "KQ_ERROR_SINGULAR";
        case KQ_ERROR_HIP: return "KQ_ERROR_HIP";
    }
    return "KQ_ERROR_UNKNOWN";
}

const char* kq_last_error_detail(void) { return g_detail.c_str(); }

int kq_version(void) { return 100; }

}  // extern "C"
