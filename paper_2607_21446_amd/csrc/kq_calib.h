// Internal interface of the layer-wise calibration kernels (kq_calib.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kq {

// Work split and workspace layout of one calibration problem: R activation
// rows, o output features, d input features, nfac factor sets of split a.
struct CalibPlan {
    int64_t R = 0, o = 0, d = 0, nb = 0, nfac = 0;
    int a = 4;
    int64_t ntn = 0;                      // 256-column tiles of the d axis (backward GEMMs)
    int64_t act_mt = 0, act_chunks = 0;   // activation-side backward: row tiles, workgroup rows
    int64_t w_mt = 0, w_ks = 0, w_kchunk = 0, w_chunks = 0;  // weight side: row tiles, K splits
    int64_t nsum = 0;                     // partial sums of the residual's squares (one per 64 x 64 tile)
    int64_t Rp = 0, op = 0;               // R and o rounded up to the 32-deep K stage
    // byte offsets into the workspace (each 256-byte aligned)
    size_t yA = 0, cA = 0, sA = 0, yW = 0, cW = 0, sW = 0, res = 0, fa = 0, fb = 0;
    size_t rnh = 0, rnl = 0, rth = 0, rtl = 0, aht = 0, wht = 0;  // K-contiguous bf16 operands of the backward products
    size_t gpa = 0, gpw = 0, sqa = 0, sqw = 0, sr = 0, ga = 0, gw = 0;
    size_t grad = 0, am = 0, av = 0, lam = 0;
    size_t total = 0;
};

CalibPlan calib_plan(int64_t R, int64_t o, int64_t d, int a, int64_t nfac);

// Yneg[r][n] = -sum_c X[r][c] W[n][c] (bf16 matrix cores, exact products, fp32 accumulation).
hipError_t launch_calib_reference(const uint16_t* X, int64_t R, int64_t d, const uint16_t* W, int64_t o,
                                  float* Yneg, hipStream_t st);

// Factors of the inverse block T^-1 = G_1^-1 (x) ... (x) G_5^-1 for the weight side.
hipError_t launch_calib_inverse_factors(const float* lu, int a, int64_t nfac, float* Ainv, float* Binv,
                                        hipStream_t st);

struct CalibStepArgs {
    const uint16_t* X;      // [R, d] bf16
    const uint16_t* W;      // [o, d] bf16
    const float* lu;        // [nfac, 5, 3]
    const float* lambdas;   // device [2]: lambda_A, lambda_W
    float* grad;            // [nfac, 5, 3]
    double* losses;         // device [4]: L_out, L_A, L_W, L
    float* lu_out;          // parameters updated in place when adam_t > 0 (== lu)
    float* adam_m;          // [nfac * 15]
    float* adam_v;          // [nfac * 15]
    int adam_t;             // 1-based Adam step; 0 = no update
    float lr;
    unsigned char* ws;      // workspace laid out by the plan
};

// Backward and update part of a step; the forward products (quantized operands,
// their fp32 values and the residual) must already be in the workspace.
hipError_t launch_calib_backward(const CalibPlan& pl, const CalibStepArgs& s, hipStream_t st);

// Small helpers of the calibration loop.
hipError_t launch_calib_init(float* adam_m, float* adam_v, int64_t n, float* lambdas, hipStream_t st);
hipError_t launch_calib_set_lambdas(const double* losses, float* lambdas, hipStream_t st);

}  // namespace kq
