// A client of libkroquant's C ABI with no Python and no torch: device buffers
// from the HIP runtime, the packed (K1 of Sec. 3.5), on-the-fly and fixed-order
// quantizers on one stream, results checked against the C oracle
// (oracle/kq_oracle.c, test infrastructure) on the same input.
//
// Input: X [300, 1152] bf16 (36 blocks per row, 10,800 blocks: a partial last
// 64-block unit), values from a fixed 64-bit LCG, two channels scaled by 40 as
// outliers; one shared factor pair A = I + 0.1 U, B = I + 0.1 U (4x4, 8x8).
// Checks (the method's tolerance): the fixed-order path equals the oracle bit
// for bit, codes, scales and y; the matrix-core paths have identical scales,
// codes that differ only by one magnitude step at a rounding tie of the
// oracle's y (at most 1e-4 of them), and y within 1e-5 of the oracle's,
// relative to max(|y|, block amax / 32).  Also checks that a bad size is
// refused with a status and a detail string.  Prints one line and exits 0 when
// every check holds, 1 otherwise.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "kroquant.h"

extern "C" int kqo_quantize(const uint16_t* X, int64_t M, int64_t d, const float* A, const float* B, int a, int b,
                            int64_t nfac, uint8_t* codes, uint8_t* scales, float* yout);

namespace {

constexpr int64_t kM = 300, kD = 1152;
constexpr int kA = 4, kB = 8;

struct Lcg {
    uint64_t s;
    double next() {  // uniform in [0, 1)
        s = s * 6364136223846793005ull + 1442695040888963407ull;
        return (double)(s >> 11) * (1.0 / 9007199254740992.0);
    }
};

uint16_t to_bf16(float f) {  // round to nearest even (finite inputs)
    uint32_t u;
    std::memcpy(&u, &f, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

#define HIP_OK(call)                                                               \
    do {                                                                           \
        hipError_t e_ = (call);                                                    \
        if (e_ != hipSuccess) {                                                    \
            std::printf("c_abi FAIL: %s -> %s\n", #call, hipGetErrorString(e_));  \
            return 1;                                                              \
        }                                                                          \
    } while (0)

#define KQ_OK(call)                                                                                    \
    do {                                                                                               \
        kq_status s_ = (call);                                                                         \
        if (s_ != KQ_SUCCESS) {                                                                        \
            std::printf("c_abi FAIL: %s -> %s (%s)\n", #call, kq_status_string(s_), kq_last_error_detail()); \
            return 1;                                                                                  \
        }                                                                                              \
    } while (0)

struct Result {
    std::vector<uint8_t> codes, scales;
    std::vector<float> y;
};

// MXFP4 rounding decision points of |y| / 2^(s-127)
const double kDecision[] = {0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0};

// 0 when `got` meets the tolerance against `ref`; prints the first failure otherwise
int compare(const char* name, const Result& got, const Result& ref, bool exact, long* flips_out) {
    long flips = 0;
    if (got.scales != ref.scales) {
        std::printf("c_abi FAIL: %s scales differ from the oracle\n", name);
        return 1;
    }
    if (exact) {
        if (got.codes != ref.codes || std::memcmp(got.y.data(), ref.y.data(), got.y.size() * 4) != 0) {
            std::printf("c_abi FAIL: %s is not bit-identical to the oracle\n", name);
            return 1;
        }
        *flips_out = 0;
        return 0;
    }
    const int64_t nb = kD / 32;
    for (int64_t i = 0; i < kM * kD; ++i) {
        const int gc = (got.codes[i / 2] >> (4 * (i & 1))) & 15, rc = (ref.codes[i / 2] >> (4 * (i & 1))) & 15;
        const int64_t blk = (i / kD) * nb + (i % kD) / 32;
        // y against the oracle's, relative to max(|y|, block amax / 32, 2^-126)
        float amax = 0.0f;
        for (int k = 0; k < 32; ++k) amax = std::fmax(amax, std::fabs(ref.y[blk * 32 + k]));
        const double den = std::fmax(std::fmax(std::fabs((double)ref.y[i]), amax / 32.0), std::ldexp(1.0, -126));
        if (std::fabs((double)got.y[i] - (double)ref.y[i]) > 1e-5 * den) {
            std::printf("c_abi FAIL: %s y[%lld] = %.9g, oracle %.9g\n", name, (long long)i, got.y[i], ref.y[i]);
            return 1;
        }
        if (gc == rc) continue;
        ++flips;
        const int dmag = std::abs((gc & 7) - (rc & 7));
        const bool sign_only_zero = (gc & 7) == 0 && (rc & 7) == 0;
        if (!(dmag == 1 || sign_only_zero)) {
            std::printf("c_abi FAIL: %s code %lld is %d, oracle %d (not adjacent)\n", name, (long long)i, gc, rc);
            return 1;
        }
        const double v = std::fabs((double)ref.y[i]) * std::ldexp(1.0, 127 - (int)ref.scales[blk]);
        double dist = 1e30;
        for (double t : kDecision) dist = std::fmin(dist, std::fabs(v - t));
        if (dist > 8e-5) {
            std::printf("c_abi FAIL: %s code %lld flipped %.6g from a rounding tie\n", name, (long long)i, dist);
            return 1;
        }
    }
    if ((double)flips > 1e-4 * (double)(kM * kD)) {
        std::printf("c_abi FAIL: %s %ld code flips\n", name, flips);
        return 1;
    }
    *flips_out = flips;
    return 0;
}

}  // namespace

int main() {
    const int64_t n = kM * kD, nblk = n / 32;
    Lcg rng{12345};
    std::vector<uint16_t> X(n);
    for (int64_t r = 0; r < kM; ++r)
        for (int64_t c = 0; c < kD; ++c) {
            float v = (float)(4.0 * rng.next() - 2.0);
            if (c == 7 || c == 700) v *= 40.0f;  // outlier channels
            X[r * kD + c] = to_bf16(v);
        }
    std::vector<float> A(kA * kA), B(kB * kB);
    for (int i = 0; i < kA * kA; ++i) A[i] = (i % (kA + 1) == 0 ? 1.0f : 0.0f) + (float)(0.1 * (rng.next() - 0.5));
    for (int i = 0; i < kB * kB; ++i) B[i] = (i % (kB + 1) == 0 ? 1.0f : 0.0f) + (float)(0.1 * (rng.next() - 0.5));

    Result ref{std::vector<uint8_t>(n / 2), std::vector<uint8_t>(nblk), std::vector<float>(n)};
    if (kqo_quantize(X.data(), kM, kD, A.data(), B.data(), kA, kB, 1, ref.codes.data(), ref.scales.data(),
                     ref.y.data()) != 0) {
        std::printf("c_abi FAIL: the oracle refused the input\n");
        return 1;
    }

    uint16_t* dX;
    float *dA, *dB, *dY;
    uint8_t *dC, *dS, *dK;
    hipStream_t st;
    HIP_OK(hipStreamCreate(&st));
    HIP_OK(hipMalloc(&dX, n * 2));
    HIP_OK(hipMalloc(&dA, A.size() * 4));
    HIP_OK(hipMalloc(&dB, B.size() * 4));
    HIP_OK(hipMalloc(&dY, n * 4));
    HIP_OK(hipMalloc(&dC, n / 2));
    HIP_OK(hipMalloc(&dS, nblk));
    HIP_OK(hipMalloc(&dK, KQ_PACK_BYTES_PER_FACTOR));
    HIP_OK(hipMemcpy(dX, X.data(), n * 2, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dA, A.data(), A.size() * 4, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dB, B.data(), B.size() * 4, hipMemcpyHostToDevice));

    KQ_OK(kq_pack_factors(dA, dB, kA, kB, 1, dK, st));
    const char* names[] = {"kq_quantize_packed", "kq_quantize", "kq_quantize_exact"};
    long flips[3] = {0, 0, 0};
    for (int path = 0; path < 3; ++path) {
        HIP_OK(hipMemsetAsync(dC, 0xEE, n / 2, st));
        HIP_OK(hipMemsetAsync(dS, 0xEE, nblk, st));
        if (path == 0) KQ_OK(kq_quantize_packed(dX, kM, kD, dA, dB, kA, kB, 1, dK, dC, dS, dY, st));
        if (path == 1) KQ_OK(kq_quantize(dX, kM, kD, dA, dB, kA, kB, 1, dC, dS, dY, st));
        if (path == 2) KQ_OK(kq_quantize_exact(dX, kM, kD, dA, dB, kA, kB, 1, dC, dS, dY, st));
        HIP_OK(hipStreamSynchronize(st));
        Result got{std::vector<uint8_t>(n / 2), std::vector<uint8_t>(nblk), std::vector<float>(n)};
        HIP_OK(hipMemcpy(got.codes.data(), dC, n / 2, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(got.scales.data(), dS, nblk, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(got.y.data(), dY, n * 4, hipMemcpyDeviceToHost));
        if (compare(names[path], got, ref, path == 2, &flips[path])) return 1;
    }

    // a row length that is not a multiple of 32 is refused before any launch
    const kq_status bad = kq_quantize(dX, kM, kD - 1, dA, dB, kA, kB, 1, dC, dS, nullptr, st);
    if (bad != KQ_ERROR_INVALID_VALUE || kq_last_error_detail() == nullptr || kq_last_error_detail()[0] == '\0') {
        std::printf("c_abi FAIL: d = %lld gave status %d\n", (long long)(kD - 1), (int)bad);
        return 1;
    }

    HIP_OK(hipFree(dX));
    HIP_OK(hipFree(dA));
    HIP_OK(hipFree(dB));
    HIP_OK(hipFree(dY));
    HIP_OK(hipFree(dC));
    HIP_OK(hipFree(dS));
    HIP_OK(hipFree(dK));
    HIP_OK(hipStreamDestroy(st));
    std::printf("c_abi ok: X [%lld, %lld], packed %ld and on-the-fly %ld code flips at ties, fixed order bit-exact, "
                "bad size refused (%s)\n",
                (long long)kM, (long long)kD, flips[0], flips[1], kq_status_string(bad));
    return 0;
}
