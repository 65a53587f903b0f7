"""KroQuant CPU oracle -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously-correct reference for the online activation quantizer of
"KroQuant: Kronecker-Structured Block Transforms for Efficient Post-Training
Quantization of Diffusion Transformers".  Only ``tests/``, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import it.  It
shares no code with the HIP library and never imports it.

Two layers:

* ``kq_oracle.c`` (built here with gcc into ``libkqoracle.so``): the scalar
  per-block definition in the canonical fp32 order -- the Kronecker transform
  of Sec. 3.2 and the OCP MX v1.0 MXFP4 encode of Sec. 3.1 -- plus the
  SmoothQuant, Hadamard-32 and plain-MXFP4 comparators of Sec. 4.4.
* numpy helpers below: fp64 forms used to pin the C code (dense
  ``numpy.kron`` transform, Sylvester Hadamard), the offline weight side of
  Sec. 3.4 (W~ = W T^-T with an fp64 LAPACK inverse), the LU factor
  construction of Sec. 3.2 and the dequantizer Q_b of Sec. 3.1.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from functools import lru_cache

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kq_oracle.c")
_LIB = os.path.join(_HERE, "libkqoracle.so")

# E2M1 magnitudes indexed by the low three code bits (OCP MX v1.0 FP4 E2M1).
E2M1_MAGNITUDES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc.  ``-ffp-contract=off`` so that only the
    explicit ``fmaf`` calls fuse; OpenMP over rows."""
    if force or not os.path.exists(_LIB):
        cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-shared",
               "-fPIC", "-std=c11", "-Wall", "-Wextra", _SRC, "-o", _LIB + ".tmp", "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


@lru_cache(maxsize=1)
def _lib():
    if not os.path.exists(_LIB):
        build(force=False)
    lib = ctypes.CDLL(_LIB)
    P, I64, I = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    lib.kqo_quantize.argtypes = [P, I64, I64, P, P, I, I, I64, P, P, P]
    lib.kqo_quantize_f32.argtypes = [P, I64, I64, P, P, I, I, I64, P, P, P]
    lib.kqo_smoothquant.argtypes = [P, I64, I64, P, P, P, P]
    lib.kqo_hadamard32.argtypes = [P, I64, I64, P, P, P]
    lib.kqo_mxfp4.argtypes = [P, I64, I64, P, P]
    lib.kqo_e2m1_codes.argtypes = [P, I64, I, P]
    lib.kqo_e8m0_scales.argtypes = [P, I64, P]
    lib.kqo_lu_factors.argtypes = [P, I, I64, P, P]
    lib.kqo_lu_inverse_factors.argtypes = [P, I, I64, P, P]
    lib.kqo_fwht.argtypes = [P, I64, I64, P, P, P]
    lib.kqo_f32_to_bf16.argtypes = [P, I64, P]
    lib.kqo_num_threads.argtypes = []
    lib.kqo_set_num_threads.argtypes = [I]
    for name in ("kqo_quantize", "kqo_quantize_f32", "kqo_smoothquant", "kqo_hadamard32",
                 "kqo_mxfp4", "kqo_e2m1_codes", "kqo_e8m0_scales", "kqo_num_threads", "kqo_lu_factors",
                 "kqo_lu_inverse_factors", "kqo_f32_to_bf16", "kqo_fwht"):
        getattr(lib, name).restype = ctypes.c_int
    lib.kqo_set_num_threads.restype = None
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc, name):
    if rc != 0:
        raise ValueError(f"{name}: oracle rejected the arguments (code {rc})")


def _outputs(M, d, want_y):
    codes = np.empty((M, d // 2), dtype=np.uint8)
    scales = np.empty((M, d // 32), dtype=np.uint8)
    y = np.empty((M, d), dtype=np.float32) if want_y else None
    return codes, scales, y


def _bf16_bits(X):
    X = np.ascontiguousarray(X)
    if X.dtype != np.uint16 or X.ndim != 2:
        raise TypeError("X must be a 2-D uint16 array of bf16 bit patterns")
    return X


def _factors(A, B, a, b):
    A = np.ascontiguousarray(A, dtype=np.float32).reshape(-1, a, a)
    B = np.ascontiguousarray(B, dtype=np.float32).reshape(-1, b, b)
    if A.shape[0] != B.shape[0]:
        raise ValueError("A and B must hold the same number of factor pairs")
    return A, B


# ---------------------------------------------------------------- C entry points
def quantize(X, A, B, want_y=False):
    """KroQuant quantizer (Sec. 3.2 transform + Sec. 3.1 MXFP4): returns
    (codes[M, d/2], scales[M, d/32], y[M, d] fp32 or None)."""
    X = _bf16_bits(X)
    A = np.asarray(A, dtype=np.float32)
    B = np.asarray(B, dtype=np.float32)
    a, b = A.shape[-1], B.shape[-1]
    A, B = _factors(A, B, a, b)
    M, d = X.shape
    codes, scales, y = _outputs(M, d, want_y)
    _check(_lib().kqo_quantize(_ptr(X), M, d, _ptr(A), _ptr(B), a, b, A.shape[0], _ptr(codes),
                               _ptr(scales), _ptr(y)), "quantize")
    return codes, scales, y


def quantize_f32(X32, A, B, want_y=False):
    """Same as ``quantize`` on fp32 rows (no bf16 rounding of the input)."""
    X32 = np.ascontiguousarray(X32, dtype=np.float32)
    A = np.asarray(A, dtype=np.float32)
    B = np.asarray(B, dtype=np.float32)
    a, b = A.shape[-1], B.shape[-1]
    A, B = _factors(A, B, a, b)
    M, d = X32.shape
    codes, scales, y = _outputs(M, d, want_y)
    _check(_lib().kqo_quantize_f32(_ptr(X32), M, d, _ptr(A), _ptr(B), a, b, A.shape[0],
                                   _ptr(codes), _ptr(scales), _ptr(y)), "quantize_f32")
    return codes, scales, y


def lu_factors_f32(lu, a):
    """K2 factors decoded from the paper's LU parameters in the oracle's fixed
    fp32 order (kq_oracle.c, kqo_lu_factors): lu [nfac, 5, 3] = (a_k, b_k, c_k)
    of G_1..G_5 -> A [nfac, a, a], B [nfac, b, b] fp32 with A (x) B = K^T."""
    lu = np.ascontiguousarray(lu, dtype=np.float32).reshape(-1, 5, 3)
    nfac = lu.shape[0]
    b = 32 // a
    A = np.empty((nfac, a, a), dtype=np.float32)
    B = np.empty((nfac, b, b), dtype=np.float32)
    _check(_lib().kqo_lu_factors(_ptr(lu), a, nfac, _ptr(A), _ptr(B)), "lu_factors_f32")
    return A, B


def lu_inverse_factors_f32(lu, a):
    """Weight-side factors for the same parameters: A' (x) B' = K^-1 with the
    closed-form inverse of every unit-determinant factor, G^-1 = [[-g11, g01],
    [g10, -g00]] (Sec. 3.2), fp32 products left to right (kq_oracle.c,
    kqo_lu_inverse_factors).  quantize(W, A', B') is then Q(W T^-T) (Sec. 3.4)."""
    lu = np.ascontiguousarray(lu, dtype=np.float32).reshape(-1, 5, 3)
    nfac = lu.shape[0]
    b = 32 // a
    A = np.empty((nfac, a, a), dtype=np.float32)
    B = np.empty((nfac, b, b), dtype=np.float32)
    _check(_lib().kqo_lu_inverse_factors(_ptr(lu), a, nfac, _ptr(A), _ptr(B)), "lu_inverse_factors_f32")
    return A, B


def quantize_lu(X, lu, a, want_y=False):
    """KroQuant quantizer with K2-form factors (Sec. 3.5): decode the LU
    parameters (``lu_factors_f32``), then ``quantize``.  Returns (codes,
    scales, y fp32 or None, y16 = bf16(y) or None)."""
    A, B = lu_factors_f32(lu, a)
    codes, scales, y = quantize(X, A, B, want_y=True)
    y16 = f32_to_bf16(y)
    return codes, scales, (y if want_y else None), (y16 if want_y else None)


def fwht(X, want_y=False):
    """Full-row FWHT comparator: y = H_d x / sqrt(d) (d a power of two, Sylvester
    order, butterflies h = 1 .. d/2 in fp32), then MXFP4 (Sec. 4.4, Table 2)."""
    X = _bf16_bits(X)
    M, d = X.shape
    codes, scales, y = _outputs(M, d, want_y)
    _check(_lib().kqo_fwht(_ptr(X), M, d, _ptr(codes), _ptr(scales), _ptr(y)), "fwht")
    return codes, scales, y


def f32_to_bf16(v):
    """fp32 -> bf16 bit patterns, round to nearest, ties to even."""
    v = np.ascontiguousarray(v, dtype=np.float32)
    out = np.empty(v.shape, dtype=np.uint16)
    _check(_lib().kqo_f32_to_bf16(_ptr(v), v.size, _ptr(out)), "f32_to_bf16")
    return out


def smoothquant(X, mult, want_y=False):
    """SmoothQuant comparator: y_c = x_c * mult_c then MXFP4 (Appendix D)."""
    X = _bf16_bits(X)
    mult = np.ascontiguousarray(mult, dtype=np.float32)
    M, d = X.shape
    if mult.shape != (d,):
        raise ValueError("mult must have shape [d]")
    codes, scales, y = _outputs(M, d, want_y)
    _check(_lib().kqo_smoothquant(_ptr(X), M, d, _ptr(mult), _ptr(codes), _ptr(scales), _ptr(y)),
           "smoothquant")
    return codes, scales, y


def hadamard32(X, want_y=False):
    """Hadamard-32 comparator: y = H32 x / sqrt(32) then MXFP4."""
    X = _bf16_bits(X)
    M, d = X.shape
    codes, scales, y = _outputs(M, d, want_y)
    _check(_lib().kqo_hadamard32(_ptr(X), M, d, _ptr(codes), _ptr(scales), _ptr(y)), "hadamard32")
    return codes, scales, y


def mxfp4(X):
    """Plain MXFP4 of the bf16 input (Q4)."""
    X = _bf16_bits(X)
    M, d = X.shape
    codes, scales, _ = _outputs(M, d, False)
    _check(_lib().kqo_mxfp4(_ptr(X), M, d, _ptr(codes), _ptr(scales)), "mxfp4")
    return codes, scales


def e2m1_codes(v, s=127):
    """Unpacked E2M1 code (sign in bit 3) of every fp32 value at E8M0 byte s."""
    v = np.ascontiguousarray(v, dtype=np.float32).ravel()
    out = np.empty(v.shape, dtype=np.uint8)
    _check(_lib().kqo_e2m1_codes(_ptr(v), v.size, int(s), _ptr(out)), "e2m1_codes")
    return out


def e8m0_scales(amax):
    """E8M0 byte of each block maximum."""
    amax = np.ascontiguousarray(amax, dtype=np.float32).ravel()
    out = np.empty(amax.shape, dtype=np.uint8)
    _check(_lib().kqo_e8m0_scales(_ptr(amax), amax.size, _ptr(out)), "e8m0_scales")
    return out


def num_threads():
    return int(_lib().kqo_num_threads())


def set_num_threads(n):
    _lib().kqo_set_num_threads(int(n))


# ---------------------------------------------------------------- numpy, fp64
def bf16_to_f32(X):
    """Widen bf16 bit patterns to fp32 (exact)."""
    return (np.asarray(X, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def unpack_codes(codes):
    """[.., n/2] packed bytes -> [.., n] codes; element 2i is the low nibble."""
    codes = np.asarray(codes, dtype=np.uint8)
    out = np.empty(codes.shape[:-1] + (codes.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = codes & 0xF
    out[..., 1::2] = codes >> 4
    return out


def dequantize(codes, scales):
    """Q_b of Sec. 3.1: value = (-1)^sign * E2M1[mag] * 2^(s-127), fp64."""
    c = unpack_codes(codes)
    mag = E2M1_MAGNITUDES[c & 7]
    sign = np.where(c & 8, -1.0, 1.0)
    s = np.repeat(np.asarray(scales, dtype=np.int64), 32, axis=-1)
    return sign * mag * np.exp2(s - 127.0)


def mxfp4_gemm(a_codes, a_scales, b_codes, b_scales):
    """The W4A4 product that consumes the quantizer's output (Sec. 3.1 eq. (1)):
    C[M, N] = deq(A)[M, K] . deq(B)[N, K]^T in fp64 (every product of two
    dequantized values is exact in fp64; the sum is a library matmul)."""
    return dequantize(a_codes, a_scales) @ dequantize(b_codes, b_scales).T


def layer_error(X, W, A, B):
    """E(T) of Sec. 3.1: || X W^T - Q(X T) Q(W T^-T)^T ||_F with the KroQuant
    block transform T = diag(A (x) B) on the activation (oracle quantizer) and
    the inverse transpose on the weight (Sec. 3.4), in fp64.  Also returns the
    two quantized operands and the fp64 X W^T."""
    x = bf16_to_f32(X).astype(np.float64) if np.asarray(X).dtype == np.uint16 else np.asarray(X, np.float64)
    w = bf16_to_f32(W).astype(np.float64) if np.asarray(W).dtype == np.uint16 else np.asarray(W, np.float64)
    xc, xs, _ = quantize(X, A, B)
    _, wc, ws = weight_transform(W, A, B)
    ref = x @ w.T
    return float(np.linalg.norm(ref - mxfp4_gemm(xc, xs, wc, ws))), (xc, xs), (wc, ws), ref


def kron_dense(A, B):
    """Materialised 32x32 blocks K = A (x) B, fp64, numpy.kron index order
    (row index = i_A * b + i_B): [nfac, 32, 32]."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    A = A.reshape(-1, A.shape[-1], A.shape[-1])
    B = B.reshape(-1, B.shape[-1], B.shape[-1])
    return np.stack([np.kron(A[f], B[f]) for f in range(A.shape[0])])


def transform_f64(X, A, B):
    """y = (A (x) B) x per 32-block in fp64 through the dense Kronecker
    product (Sec. 3.2).  X: [M, d] bf16 bits or any float array."""
    Xf = bf16_to_f32(X) if np.asarray(X).dtype == np.uint16 else np.asarray(X)
    Xf = Xf.astype(np.float64)
    M, d = Xf.shape
    K = kron_dense(A, B)
    blocks = Xf.reshape(M, d // 32, 32)
    if K.shape[0] == 1:
        y = blocks @ K[0].T
    else:
        y = np.einsum("fij,mfj->mfi", K, blocks)
    return y.reshape(M, d)


def hadamard32_f64(X):
    """y = H32 x / sqrt(32) per block in fp64 with the Sylvester H32."""
    from scipy.linalg import hadamard
    Xf = bf16_to_f32(X).astype(np.float64)
    M, d = Xf.shape
    H = hadamard(32).astype(np.float64) / np.sqrt(32.0)
    return (Xf.reshape(M, d // 32, 32) @ H.T).reshape(M, d)


def factors_inverse_transpose(A, B):
    """(A^-T, B^-T) in fp64 via LAPACK, rounded to fp32, so that
    (A (x) B)^-T = A^-T (x) B^-T (Sec. 3.2: the inverse of a Kronecker product
    is the Kronecker product of the inverses)."""
    A64 = np.asarray(A, dtype=np.float64)
    B64 = np.asarray(B, dtype=np.float64)
    Ai = np.swapaxes(np.linalg.inv(A64), -1, -2)
    Bi = np.swapaxes(np.linalg.inv(B64), -1, -2)
    return Ai.astype(np.float32), Bi.astype(np.float32)


def weight_transform(W, A, B, want_codes=True):
    """Offline weight side, Sec. 3.4 / eq. (1): W~ = W T^-T, i.e. per block
    w' = (A (x) B)^-T w; returns (W~ fp32, codes, scales)."""
    Ait, Bit = factors_inverse_transpose(A, B)
    codes, scales, y = quantize(W, Ait, Bit, want_y=True)
    return (y, codes, scales) if want_codes else (y, None, None)


def lu_factor(a, b, c):
    """G = L U with L = [[1, 0], [c, 1]], U = [[a, b], [0, -1/a]] (Sec. 3.2)."""
    L = np.array([[1.0, 0.0], [c, 1.0]])
    U = np.array([[a, b], [0.0, -1.0 / a]])
    return L @ U


def lu_to_factors(abc, a_dim):
    """Paper parameters (a_k, b_k, c_k), k = 1..5, per block -> library
    factors (A, B) with A (x) B = K^T, K = G1 (x) ... (x) G5.

    The paper right-multiplies row activations (A -> A T, eq. (1)), so a
    block row x^T maps to x^T K, i.e. y = K^T x; (G1 (x) .. (x) G5)^T =
    G1^T (x) .. (x) G5^T, split after log2(a_dim) factors."""
    abc = np.asarray(abc, dtype=np.float64).reshape(-1, 5, 3)
    na = int(round(np.log2(a_dim)))
    As, Bs = [], []
    for blk in abc:
        Gs = [lu_factor(*blk[k]) for k in range(5)]
        Ka = np.ones((1, 1))
        for G in Gs[:na]:
            Ka = np.kron(Ka, G)
        Kb = np.ones((1, 1))
        for G in Gs[na:]:
            Kb = np.kron(Kb, G)
        As.append(Ka.T)
        Bs.append(Kb.T)
    return np.array(As, dtype=np.float32), np.array(Bs, dtype=np.float32)


# ---------------------------------------------------------------- tolerance rule
# Decision points of the E2M1 encode on v = |y| / 2^(s - 127): the sign decision
# at 0 and the midpoints between neighbouring magnitudes (Sec. 3.1 quantizer,
# OCP MX v1.0 E2M1).
E2M1_DECISION_POINTS = np.array([0.0, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0], dtype=np.float64)


def mx_compare(codes, scales, codes_ref, scales_ref, y_ref=None, y=None, rel_tol=1e-5, max_flip_frac=1e-4,
               y_exact=None):
    """Compare an MXFP4 result with the oracle's under the tolerance of a path
    whose fp32 accumulation order differs from the oracle's:

    * E8M0 scales identical;
    * codes identical except flips to the adjacent magnitude (|dmag| = 1) or a
      sign-only flip of magnitude 0, at most ``max_flip_frac`` of all codes;
    * with ``y_ref`` (the oracle's fp32 transformed values): every flip sits at
      a rounding decision, |v_ref - t| <= rel_tol * 8 with v_ref = |y_ref| /
      2^(s - 127) and t the nearest decision point (an fp32 result within
      rel_tol of max(|y_ref|, amax_block / 32) moves v by at most that much,
      since v < 8);
    * with ``y`` as well: max |y - y_t| / max(|y_t|, amax_block(y_t) / 32) <=
      rel_tol, y_t = ``y_exact`` (the exact transform of the input, e.g.
      ``transform_f64``) when given, else ``y_ref``.  The fixed-order fp32
      values are themselves one rounding of the exact ones (up to 33 u
      sum_k |K_nk| |x_k| away, u = 2^-24), so two fp32 evaluation orders can
      differ by the sum of their errors; the exact value is the reference the
      relative error is meant against.  Below the smallest normal fp32 the
      denominator is 2^-126: subnormal fp32 values are spaced 2^-149 apart,
      so no fp32 result holds a relative error of 1e-5 there.

    Works on the packed bytes and unpacks only the differing ones, so it is
    cheap at full size.  Returns a dict with the counts and ``ok``."""
    codes, codes_ref = np.asarray(codes, np.uint8), np.asarray(codes_ref, np.uint8)
    scales, scales_ref = np.asarray(scales, np.uint8), np.asarray(scales_ref, np.uint8)
    if codes.shape != codes_ref.shape or scales.shape != scales_ref.shape:
        raise ValueError("result and reference shapes differ")
    M = codes.shape[0]
    nbytes_row = codes.shape[1]
    rep = {"codes": int(codes.size * 2), "scale_mismatches": int(np.count_nonzero(scales != scales_ref))}
    flat, flat_ref = codes.reshape(-1), codes_ref.reshape(-1)
    byte_idx = np.flatnonzero(flat != flat_ref)
    lo = (flat[byte_idx] & 0xF, flat_ref[byte_idx] & 0xF)
    hi = (flat[byte_idx] >> 4, flat_ref[byte_idx] >> 4)
    elem = np.concatenate([2 * byte_idx[lo[0] != lo[1]], 2 * byte_idx[hi[0] != hi[1]] + 1])
    got = np.concatenate([lo[0][lo[0] != lo[1]], hi[0][hi[0] != hi[1]]]).astype(np.int64)
    ref = np.concatenate([lo[1][lo[0] != lo[1]], hi[1][hi[0] != hi[1]]]).astype(np.int64)
    dmag = np.abs((got & 7) - (ref & 7))
    sign_only_zero = ((got & 7) == 0) & ((ref & 7) == 0)
    rep["flips"] = int(elem.size)
    rep["non_adjacent"] = int(np.count_nonzero(~((dmag == 1) | sign_only_zero)))
    rep["flip_frac"] = rep["flips"] / max(rep["codes"], 1)
    rep["off_tie"] = None
    if y_ref is not None and elem.size:
        y_ref_flat = np.asarray(y_ref, np.float32).reshape(-1)
        r, k = elem // (2 * nbytes_row), elem % (2 * nbytes_row)
        s = scales_ref[r, k // 32].astype(np.float64)
        v = np.abs(y_ref_flat[elem].astype(np.float64)) * np.exp2(127.0 - s)
        dist = np.min(np.abs(v[:, None] - E2M1_DECISION_POINTS[None, :]), axis=1)
        rep["off_tie"] = int(np.count_nonzero(dist > rel_tol * 8.0))
        rep["max_tie_distance"] = float(dist.max())
    elif y_ref is not None:
        rep["off_tie"] = 0
    rep["y_max_err"] = None
    y_t = y_exact if y_exact is not None else y_ref
    if y is not None and y_t is not None:
        worst = 0.0
        step = max(1, (1 << 22) // max(nbytes_row * 2, 1))
        for r0 in range(0, M, step):
            yr = np.asarray(y_t[r0:r0 + step], np.float64)
            yg = np.asarray(y[r0:r0 + step], np.float64)
            amax = np.abs(yr).reshape(yr.shape[0], -1, 32).max(-1)
            den = np.maximum(np.maximum(np.abs(yr), np.repeat(amax, 32, axis=1) / 32.0), 2.0 ** -126)
            if yr.size:
                worst = max(worst, float(np.max(np.abs(yg - yr) / den)))
        rep["y_max_err"] = worst
    rep["ok"] = bool(rep["scale_mismatches"] == 0 and rep["non_adjacent"] == 0
                     and rep["flip_frac"] <= max_flip_frac and (rep["off_tie"] in (None, 0))
                     and (rep["y_max_err"] is None or rep["y_max_err"] <= rel_tol))
    return rep
