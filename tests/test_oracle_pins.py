"""Pins of the CPU oracle to facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: hand-derived
encodes (tests/golden/), closed forms (the Kronecker identity, the inverse of
a Kronecker product, the Sylvester Hadamard), an independently derived
threshold rule checked over every fp32 value in [0, 8], the bit-level scale
rule, and invariants (sign symmetry, power-of-two equivariance, eq. (1)
invariance, thread-count independence).  CPU only.
"""
import functools

import numpy as np
import pytest

import oracle
import synth
from conftest import load_golden, parse_values

AB_SPLITS = [(4, 8), (2, 16), (8, 4), (1, 32)]


def _row(vals):
    return synth.to_bf16_bits(np.array([vals], dtype=np.float32))


# ---------------------------------------------------------------- golden blocks
@pytest.mark.parametrize("case", load_golden("mxfp4_blocks.txt"), ids=lambda c: c[0])
def test_golden_mxfp4_block(case):
    name, spec, s, hexcodes = case
    vals = parse_values(spec)
    X = _row(vals)
    # the fixture values must be bf16-exact, so the encode sees exactly them
    assert np.array_equal(oracle.bf16_to_f32(X)[0], np.array(vals, dtype=np.float32))
    codes, scales = oracle.mxfp4(X)
    assert int(scales[0, 0]) == int(s), name
    assert codes[0].tobytes().hex() == hexcodes, name


@pytest.mark.parametrize("case", load_golden("transform_blocks.txt"), ids=lambda c: c[0] + c[1])
def test_golden_transform_block(case):
    method, spec, s, hexcodes = case
    X = _row(parse_values(spec))
    if method == "hadamard32":
        codes, scales, _ = oracle.hadamard32(X)
    else:
        from scipy.linalg import hadamard
        A = (hadamard(4) / 2.0).astype(np.float32)
        B = (hadamard(8) / np.sqrt(8.0)).astype(np.float32)
        codes, scales, _ = oracle.quantize(X, A[None], B[None])
    assert int(scales[0, 0]) == int(s)
    assert codes[0].tobytes().hex() == hexcodes


# ---------------------------------------------------------------- element encode
def _threshold_magnitude(v):
    """E2M1 magnitude index from the decision thresholds: the midpoints of
    consecutive magnitudes {0,.5,1,1.5,2,3,4,6}; at a midpoint the even index
    wins, so the comparison is '>' when the upper neighbour is odd and '>='
    when it is even."""
    return ((v > 0.25).astype(np.uint8) + (v >= 0.75) + (v > 1.25) + (v >= 1.75) + (v > 2.5)
            + (v >= 3.5) + (v > 5.0)).astype(np.uint8)


def test_e2m1_exhaustive_unit_scale():
    """Every fp32 bit pattern in [0, 8] (and its negation) at scale 2^0."""
    lo, hi = 0, np.float32(8.0).view(np.uint32) + 1
    chunk = 1 << 24
    for start in range(int(lo), int(hi), chunk):
        bits = np.arange(start, min(start + chunk, int(hi)), dtype=np.uint32)
        v = bits.view(np.float32)
        got = oracle.e2m1_codes(v, 127)
        assert np.array_equal(got, _threshold_magnitude(v)), hex(start)
        gotn = oracle.e2m1_codes(-v, 127)
        assert np.array_equal(gotn, _threshold_magnitude(v) | 8), hex(start)


def test_e2m1_saturation_and_other_scales():
    rng = np.random.default_rng(7)
    big = np.float32(8.0) * (1 + rng.random(100000, dtype=np.float32) * 1e6)
    assert np.all(oracle.e2m1_codes(big, 127) == 7)
    for s in (0, 1, 2, 100, 127, 128, 200, 254):
        # values whose scaled magnitude |y| / 2^(s-127) spans [0, 8)
        v = np.minimum(rng.random(200000) * 8.0 * np.exp2(s - 127.0),
                       np.finfo(np.float32).max).astype(np.float32)
        scaled = np.abs(v.astype(np.float64)) * np.exp2(127.0 - s)
        assert np.array_equal(oracle.e2m1_codes(v, s), _threshold_magnitude(scaled)), s


# ---------------------------------------------------------------- E8M0 scale
def test_e8m0_bit_rule():
    """s = max(biased exponent field - 2, 0), from the fp32 bit pattern; this
    is floor(log2 amax) - emax(E2M1) + 127 clamped at 0 for normal amax, and 0
    for subnormal amax."""
    rng = np.random.default_rng(3)
    bits = rng.integers(0, 0x7F800000, size=2_000_000, dtype=np.uint32)
    amax = bits.view(np.float32)
    got = oracle.e8m0_scales(amax)
    expfield = ((bits >> 23) & 0xFF).astype(np.int64)
    want = np.maximum(expfield - 2, 0)
    assert np.array_equal(got.astype(np.int64), want)
    # for s > 0 the scaled maximum lands in [4, 8): largest magnitude 6 fits
    pos = got > 0
    r = amax[pos].astype(np.float64) / np.exp2(got[pos].astype(np.float64) - 127.0)
    assert r.min() >= 4.0 and r.max() < 8.0
    assert oracle.e8m0_scales(np.zeros(1))[0] == 0


# ---------------------------------------------------------------- transform
def _kron_bound(X, A, B):
    """Per-element sum_j |K_kj| |x_j|, fp64."""
    K = np.abs(oracle.kron_dense(A, B))
    Xa = np.abs(oracle.bf16_to_f32(X).astype(np.float64))
    M, d = Xa.shape
    blocks = Xa.reshape(M, d // 32, 32)
    if K.shape[0] == 1:
        return (blocks @ K[0].T).reshape(M, d)
    return np.einsum("fij,mfj->mfi", K, blocks).reshape(M, d)


@pytest.mark.parametrize("ab", AB_SPLITS)
@pytest.mark.parametrize("per_block", [False, True])
def test_kron_identity(ab, per_block):
    """(A (x) B) x via the canonical separable fp32 order equals the dense
    numpy.kron product in fp64 to within fp32 accumulation error."""
    a, b = ab
    M, d = 37, 1152
    X = synth.activations(M, d, "student_t3", seed=11, chan_frac=0.01, chan_factor=30)
    A, B = synth.factors(a, b, d // 32 if per_block else 1, seed=5)
    _, _, y = oracle.quantize(X, A, B, want_y=True)
    ref = oracle.transform_f64(X, A, B)
    bound = _kron_bound(X, A, B)
    err = np.abs(y.astype(np.float64) - ref)
    assert np.all(err <= (a + b + 2) * 2.0**-24 * bound + 1e-30)
    # a transposed factor would break the identity by far more than rounding
    At = np.swapaxes(A, -1, -2).copy()
    _, _, y_bad = oracle.quantize(X, At, B, want_y=True)
    if a > 1:
        assert np.max(np.abs(y_bad - ref) / (bound + 1e-30)) > 1e-3


def test_kronecker_bit_formula_and_lu():
    """Sec. 3.5 (K2): K[r, c] = prod_k G_k[r_(5-k), c_(5-k)] equals
    G1 (x) ... (x) G5 in numpy.kron order; LU factors have det -1; the
    Hadamard init is LU(1/sqrt2, 1/sqrt2, 1)."""
    rng = np.random.default_rng(1)
    abc = rng.normal(size=(5, 3))
    abc[:, 0] = np.where(np.abs(abc[:, 0]) < 0.2, 0.5, abc[:, 0])
    Gs = [oracle.lu_factor(*abc[k]) for k in range(5)]
    for G in Gs:
        assert abs(np.linalg.det(G) + 1.0) < 1e-12
    K = Gs[0]
    for G in Gs[1:]:
        K = np.kron(K, G)
    Kbit = np.ones((32, 32))
    for r in range(32):
        for c in range(32):
            for k in range(1, 6):
                Kbit[r, c] *= Gs[k - 1][(r >> (5 - k)) & 1, (c >> (5 - k)) & 1]
    assert np.allclose(K, Kbit, rtol=0, atol=1e-12 * np.abs(K).max())
    h = 1 / np.sqrt(2)
    H2 = np.array([[h, h], [h, -h]])
    assert np.allclose(oracle.lu_factor(h, h, 1.0), H2, atol=1e-15)
    # lu_to_factors: A (x) B = K^T for every split
    for a, b in AB_SPLITS:
        A, B = oracle.lu_to_factors(abc[None], a)
        assert A.shape == (1, a, a) and B.shape == (1, b, b)
        KT = np.kron(A[0].astype(np.float64), B[0].astype(np.float64))
        assert np.allclose(KT, K.T, rtol=0, atol=1e-6 * np.abs(K).max())


def _k_paper_f64(abc):
    """K = G1 (x) ... (x) G5 written out from the K2 entry formula of Sec. 3.5,
    G_k = [[a, b], [c a, c b - 1/a]] in fp64 (the L U product of Sec. 3.2)."""
    G = [np.array([[a, b], [c * a, c * b - 1.0 / a]]) for a, b, c in np.asarray(abc, np.float64)]
    K = np.ones((32, 32))
    for r in range(32):
        for c in range(32):
            for k in range(5):
                K[r, c] *= G[k][(r >> (4 - k)) & 1, (c >> (4 - k)) & 1]
    return K, G


@pytest.mark.parametrize("seed", [3, 4, 5])
def test_lu_factors_f32_against_paper_formula(seed):
    """kqo_lu_factors (fp32 decode of the K2 parameters) against the paper's
    entry formula in fp64: A (x) B = K^T for every split, to within the
    roundings of at most five fp32 products, for two factor pairs at once."""
    rng = np.random.default_rng(seed)
    lu = rng.normal(size=(2, 5, 3)).astype(np.float32)
    lu[..., 0] = np.where(np.abs(lu[..., 0]) < 0.3, np.float32(0.7), lu[..., 0])
    for f in range(2):
        K, G = _k_paper_f64(lu[f])
        scale = np.prod([np.abs(g).max() for g in G])
        Ks = []
        for a, b in AB_SPLITS:
            A, B = oracle.lu_factors_f32(lu, a)
            KT = np.kron(A[f].astype(np.float64), B[f].astype(np.float64))
            assert np.abs(KT - K.T).max() <= 2e-6 * scale, (a, f)
            Ks.append(KT)
        # the split only moves fp32 roundings
        for KT in Ks[1:]:
            assert np.abs(KT - Ks[0]).max() <= 2e-6 * scale
        # det K = prod_k det(G_k)^16 = (-1)^80 = 1
        assert abs(np.linalg.det(Ks[0]) - 1.0) < 1e-3


def test_lu_factors_f32_hadamard_init_and_exact_entries():
    """LU(1/sqrt2, 1/sqrt2, 1) for all five factors is the Hadamard init
    H32/sqrt(32) (Sec. 3.2); with a = 1 the A factor is the empty product 1;
    with integer parameters every product is exact."""
    from scipy.linalg import hadamard
    h = np.float32(1 / np.sqrt(2))
    lu = np.array([[[h, h, 1.0]] * 5], dtype=np.float32)
    for a, b in AB_SPLITS:
        A, B = oracle.lu_factors_f32(lu, a)
        KT = np.kron(A[0].astype(np.float64), B[0].astype(np.float64))
        assert np.abs(KT - hadamard(32) / np.sqrt(32)).max() < 1e-6
    A, B = oracle.lu_factors_f32(lu, 1)
    assert A.shape == (1, 1, 1) and A[0, 0, 0] == 1.0
    lu = np.array([[[1.0, 2.0, 1.0], [-1.0, 1.0, 2.0], [2.0, 0.0, 1.0], [1.0, -1.0, -1.0], [-2.0, 1.0, 0.0]]],
                  dtype=np.float32)   # 1/a exact, every entry a small integer or half-integer
    K, _ = _k_paper_f64(lu[0])
    for a, b in AB_SPLITS:
        A, B = oracle.lu_factors_f32(lu, a)
        assert np.array_equal(np.kron(A[0].astype(np.float64), B[0].astype(np.float64)), K.T), a


def test_f32_to_bf16_round_to_nearest_even():
    """The 16-bit output rounding against torch's fp32 -> bfloat16 conversion
    (round to nearest, ties to even), on random values and on every kind of
    exact tie."""
    import torch
    rng = np.random.default_rng(9)
    v = np.concatenate([rng.normal(size=200000) * 10.0 ** rng.integers(-30, 30, 200000),
                        rng.normal(size=1000)]).astype(np.float32)
    ties = (rng.integers(0, 1 << 31, 4000, dtype=np.uint64).astype(np.uint32) & 0x7F7F0000) | 0x8000
    ties[::2] |= 0x10000                       # odd and even bf16 neighbours below
    sign = (rng.integers(0, 2, ties.size).astype(np.uint32) << 31)
    v = np.concatenate([v, (ties | sign).view(np.float32), np.float32([0.0, -0.0, 1.0, -3.5])])
    v = v[np.isfinite(v) & (np.abs(v) < 3e38)]
    want = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.f32_to_bf16(v), want)


def test_fwht_against_dense_and_hadamard32():
    """Full-row FWHT comparator: for d = 32 bit-identical to the Hadamard-32
    comparator (same butterflies, same constant); for larger d within the
    fp32 butterfly error bound of the dense fp64 H_d x / sqrt(d) (Sylvester
    order); energy preserved (H_d / sqrt(d) orthonormal)."""
    from scipy.linalg import hadamard
    X = synth.activations(48, 32, "normal", seed=11)
    for got, want in zip(oracle.fwht(X, want_y=True), oracle.hadamard32(X, want_y=True)):
        assert np.array_equal(got, want)
    for d in (256, 2048):
        X = synth.activations(16, d, "student_t3", seed=12, chan_frac=0.02, chan_factor=30.0)
        x = oracle.bf16_to_f32(X).astype(np.float64)
        _, _, y = oracle.fwht(X, want_y=True)
        ref = x @ hadamard(d).T / np.sqrt(d)
        n = int(np.log2(d))
        bound = (n + 2) * 2.0 ** -24 * np.abs(x).sum(1, keepdims=True) / np.sqrt(d)
        assert np.all(np.abs(y - ref) <= bound)
        assert np.allclose((y.astype(np.float64) ** 2).sum(1), (x ** 2).sum(1), rtol=1e-5)
    with pytest.raises(ValueError):
        oracle.fwht(synth.activations(4, 96, "normal", seed=1))


def test_mxfp4_gemm_brute_force_and_layer_error():
    """W4A4 product: against a scalar triple loop over decoded codes (pins the
    operand orientation: C = deq(A) deq(B)^T) on a tiny case; E(T) of
    eq. (1): zero for lossless stand-ins, equal to the plain MXFP4 error for
    identity factors, and the exact-arithmetic invariance X W^T = (X T)(W T^-T)^T."""
    rng = np.random.default_rng(13)
    M, N, K = 3, 5, 64
    ac = rng.integers(0, 256, (M, K // 2), dtype=np.uint8)
    bc = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    as_ = rng.integers(120, 134, (M, K // 32), dtype=np.uint8)
    bs = rng.integers(120, 134, (N, K // 32), dtype=np.uint8)
    C = oracle.mxfp4_gemm(ac, as_, bc, bs)
    mags = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]

    def val(codes, scales, r, k):
        byte = int(codes[r, k // 2])
        c = byte & 15 if k % 2 == 0 else byte >> 4
        return (-1.0 if c & 8 else 1.0) * mags[c & 7] * 2.0 ** (int(scales[r, k // 32]) - 127)
    for m in range(M):
        for n in range(N):
            ref = sum(val(ac, as_, m, k) * val(bc, bs, n, k) for k in range(K))
            assert C[m, n] == ref
    # identity factors: E(T) is the plain MXFP4 layer error
    X = synth.activations(32, 256, "student_t3", seed=14)
    W = synth.activations(48, 256, "normal", seed=15)
    a, b = 4, 8
    Ai, Bi = np.eye(a, dtype=np.float32)[None], np.eye(b, dtype=np.float32)[None]
    e_id, _, _, ref = oracle.layer_error(X, W, Ai, Bi)
    xc, xs = oracle.mxfp4(X)
    wc, ws = oracle.mxfp4(W)
    assert np.isclose(e_id, np.linalg.norm(ref - oracle.mxfp4_gemm(xc, xs, wc, ws)), rtol=1e-12)
    # eq. (1): the unquantized transformed product equals X W^T
    A, B = synth.factors(a, b, 1, seed=16)
    Ait, Bit = oracle.factors_inverse_transpose(A, B)
    xt = oracle.transform_f64(X, A, B)
    wt = oracle.transform_f64(oracle.bf16_to_f32(W), Ait, Bit)
    assert np.allclose(xt @ wt.T, ref, rtol=0, atol=1e-5 * np.abs(ref).max())
    e_kq, _, _, _ = oracle.layer_error(X, W, A, B)
    assert 0 < e_kq < 0.5 * np.linalg.norm(ref)


def test_sylvester_hadamard_split():
    from scipy.linalg import hadamard
    assert np.array_equal(np.kron(hadamard(4), hadamard(8)), hadamard(32))
    H2 = hadamard(2)
    H = H2
    for _ in range(4):
        H = np.kron(H, H2)
    assert np.array_equal(H, hadamard(32))


def test_identity_factors_reduce_to_plain_mxfp4():
    X = synth.activations(64, 1152, "normal", seed=2)
    X[X == 0x8000] = 0  # -0.0 would become +0.0 through the products (sign of zero)
    for a, b in AB_SPLITS:
        A = np.eye(a, dtype=np.float32)[None]
        B = np.eye(b, dtype=np.float32)[None]
        c1, s1, y = oracle.quantize(X, A, B, want_y=True)
        c0, s0 = oracle.mxfp4(X)
        assert np.array_equal(y, oracle.bf16_to_f32(X))
        assert np.array_equal(s1, s0) and np.array_equal(c1, c0)


def test_hadamard32_against_dense():
    X = synth.activations(33, 2240, "laplace", seed=4, chan_frac=0.02, chan_factor=20)
    _, _, y = oracle.hadamard32(X, want_y=True)
    ref = oracle.hadamard32_f64(X)
    bound = np.abs(oracle.bf16_to_f32(X).astype(np.float64)).reshape(33, -1, 32).sum(-1)
    bound = np.repeat(bound, 32, axis=1) / np.sqrt(32.0)
    assert np.all(np.abs(y - ref) <= 7 * 2.0**-24 * bound + 1e-30)


def test_smoothquant_single_rounding():
    """y_c = fp32(x_c * m_c): the product of two fp32 values is exact in
    fp64, so one rounding to fp32 gives the expected value bit for bit."""
    X = synth.activations(40, 2240, "laplace", seed=8, chan_frac=0.02, chan_factor=20)
    m = synth.smoothquant_multipliers(X)
    _, _, y = oracle.smoothquant(X, m, want_y=True)
    ref = (oracle.bf16_to_f32(X).astype(np.float64) * m.astype(np.float64)).astype(np.float32)
    assert np.array_equal(y.view(np.uint32), ref.view(np.uint32))
    c1, s1, _ = oracle.smoothquant(X, np.ones(2240, np.float32))
    c0, s0 = oracle.mxfp4(X)
    assert np.array_equal(c1, c0) and np.array_equal(s1, s0)


# ---------------------------------------------------------------- layout and error
@pytest.mark.parametrize("method", ["kron", "kron_pb", "had", "smooth", "plain"])
def test_dequantized_error_bound(method):
    """Q_b(y) - y stays within half the local E2M1 spacing times the scale
    (at most 1 * 2^(s-127)), or equals the clip when |y| > 6 * 2^(s-127).
    A wrong row/block/nibble offset in the packing fails this."""
    M, d = 29, 2240
    X = synth.activations(M, d, "student_t3", seed=21, chan_frac=0.005, chan_factor=50)
    if method in ("kron", "kron_pb"):
        A, B = synth.factors(4, 8, d // 32 if method == "kron_pb" else 1, seed=9)
        codes, scales, y = oracle.quantize(X, A, B, want_y=True)
    elif method == "had":
        codes, scales, y = oracle.hadamard32(X, want_y=True)
    elif method == "smooth":
        codes, scales, y = oracle.smoothquant(X, synth.smoothquant_multipliers(X), want_y=True)
    else:
        codes, scales = oracle.mxfp4(X)
        y = oracle.bf16_to_f32(X)
    deq = oracle.dequantize(codes, scales)
    unit = np.exp2(np.repeat(scales.astype(np.float64), 32, axis=1) - 127.0)
    yd = y.astype(np.float64)
    clip = np.maximum(np.abs(yd) - 6.0 * unit, 0.0)
    assert np.all(np.abs(deq - yd) <= np.maximum(1.0 * unit, clip) * (1 + 1e-12))
    # and the block maximum never clips by more than 8/6
    amax = np.abs(yd).reshape(M, -1, 32).max(-1)
    assert np.all(amax < 8.0 * np.exp2(scales.astype(np.float64) - 127.0) + 1e-300)


# ---------------------------------------------------------------- invariants
def test_sign_symmetry():
    X = synth.activations(50, 1152, "normal", seed=12)
    A, B = synth.factors(4, 8, 1, seed=13)
    c, s, _ = oracle.quantize(X, A, B)
    cn, sn, _ = oracle.quantize(X ^ np.uint16(0x8000), A, B)
    assert np.array_equal(s, sn)
    u, un = oracle.unpack_codes(c), oracle.unpack_codes(cn)
    nz = (u & 7) != 0
    assert np.array_equal(u[nz] ^ 8, un[nz])
    assert np.array_equal(u & 7, un & 7)


def test_power_of_two_equivariance():
    X = synth.activations(50, 1152, "normal", seed=14)
    A, B = synth.factors(4, 8, 1, seed=15)
    c, s, _ = oracle.quantize(X, A, B)
    for k in (-5, 3):
        Xk = synth.to_bf16_bits(oracle.bf16_to_f32(X) * np.float32(2.0**k))
        ck, sk, _ = oracle.quantize(Xk, A, B)
        assert np.array_equal(ck, c)
        assert np.array_equal(sk.astype(int), s.astype(int) + k)


def test_thread_count_independence():
    X = synth.activations(96, 1152, "student_t3", seed=16)
    A, B = synth.factors(4, 8, 36, seed=17)
    n = oracle.num_threads()
    try:
        oracle.set_num_threads(1)
        c1, s1, y1 = oracle.quantize(X, A, B, want_y=True)
        oracle.set_num_threads(max(n, 4))
        c2, s2, y2 = oracle.quantize(X, A, B, want_y=True)
    finally:
        oracle.set_num_threads(n)
    assert np.array_equal(c1, c2) and np.array_equal(s1, s2)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))


# ---------------------------------------------------------------- weight side
@pytest.mark.parametrize("ab", AB_SPLITS)
def test_weight_side_invariance_and_round_trip(ab):
    """Eq. (1): (x T) . (w T^-T) = x . w, with the per-block inverse built as
    A^-1 (x) B^-1 (Sec. 3.2); and transforming by (A, B) then by (A^-1, B^-1)
    returns the input."""
    a, b = ab
    d = 1152
    X = synth.activations(16, d, "normal", seed=18)
    W = synth.activations(12, d, "normal", seed=19, chan_frac=0.0)
    A, B = synth.factors(a, b, d // 32, seed=20)
    _, _, y = oracle.quantize(X, A, B, want_y=True)
    wt, wc, ws = oracle.weight_transform(W, A, B)
    lhs = y.astype(np.float64) @ wt.astype(np.float64).T
    xf = oracle.bf16_to_f32(X).astype(np.float64)
    wf = oracle.bf16_to_f32(W).astype(np.float64)
    rhs = xf @ wf.T
    scale = np.abs(xf) @ np.abs(wf).T
    assert np.max(np.abs(lhs - rhs) / scale) < 2e-5
    # inverse transpose really is (A (x) B)^-T per block
    Ait, Bit = oracle.factors_inverse_transpose(A, B)
    Kinv = np.linalg.inv(oracle.kron_dense(A, B))
    assert np.allclose(oracle.kron_dense(Ait, Bit), np.swapaxes(Kinv, -1, -2), atol=1e-5)
    # round trip through the inverse factors
    Ai = np.linalg.inv(A.astype(np.float64)).astype(np.float32)
    Bi = np.linalg.inv(B.astype(np.float64)).astype(np.float32)
    _, _, back = oracle.quantize_f32(y, Ai, Bi, want_y=True)
    assert np.max(np.abs(back - xf)) <= 1e-5 * np.abs(xf).max()
    assert wc.shape == (12, d // 2) and ws.shape == (12, d // 32)


def test_rejects_bad_arguments():
    X = np.zeros((2, 64), np.uint16)
    A, B = synth.factors(4, 8, 1, seed=0)
    with pytest.raises(ValueError):
        oracle.quantize(X, A, np.eye(16, dtype=np.float32)[None])  # a*b != 32
    with pytest.raises(ValueError):
        oracle.quantize(np.zeros((2, 48), np.uint16), A, B)      # d % 32 != 0
    c, s, _ = oracle.quantize(np.zeros((0, 64), np.uint16), A, B)
    assert c.shape == (0, 32) and s.shape == (0, 2)


# ---------------------------------------------------------------- the tolerance rule itself
def _tie_row():
    # one block, amax 6 (s = 127, v = |y|): element 1 sits exactly on the 1.25 tie,
    # element 2 at 1.1 (no tie near), element 3 at -0.2 (rounds to -0)
    vals = np.zeros(32, np.float32)
    vals[:4] = [6.0, 1.25, 1.1, -0.2]
    eye_a, eye_b = np.eye(4, dtype=np.float32)[None], np.eye(8, dtype=np.float32)[None]
    c, s, y = oracle.quantize_f32(vals[None], eye_a, eye_b, want_y=True)
    assert int(s[0, 0]) == 127 and c[0, 0] == 0x27 and c[0, 1] == 0x82   # 6 -> 7, 1.25 -> 1.0 (2); 1.1 -> 2, -0.2 -> 8
    return c, s, y


def test_mx_compare_accepts_tie_flips_and_rejects_the_rest():
    """Planted mistakes in the oracle's own output: an adjacent flip at an exact
    tie passes; the same flip off a tie, a two-step flip, a sign flip of a
    nonzero code, a scale change and a y error beyond 1e-5 all fail."""
    c, s, y = _tie_row()
    cmp = functools.partial(oracle.mx_compare, max_flip_frac=0.5)   # one block: 1 flip = 1/32 of its codes
    assert cmp(c, s, c, s, y, y)["ok"]
    at_tie = c.copy()
    at_tie[0, 0] = 0x37                          # element 1: 1.0 -> 1.5 at the 1.25 tie
    assert cmp(at_tie, s, c, s, y)["ok"]
    off_tie = c.copy()
    off_tie[0, 1] = 0x83                         # element 2: 1.0 -> 1.5 at v = 1.1
    rep = cmp(off_tie, s, c, s, y)
    assert not rep["ok"] and rep["off_tie"] == 1 and rep["non_adjacent"] == 0
    assert cmp(off_tie, s, c, s)["ok"]        # without y only adjacency is checked
    two_step = c.copy()
    two_step[0, 0] = 0x47
    assert cmp(two_step, s, c, s, y)["non_adjacent"] == 1
    sign = c.copy()
    sign[0, 0] = 0xA7                            # element 1: +1.0 -> -1.0
    assert cmp(sign, s, c, s)["non_adjacent"] == 1
    zero_sign = c.copy()
    zero_sign[0, 1] = 0x02                       # element 3: -0 -> +0 (v = 0.2, not at the 0 decision)
    rep = cmp(zero_sign, s, c, s, y)
    assert rep["non_adjacent"] == 0 and rep["off_tie"] == 1
    s2 = s.copy()
    s2[0, 0] += 1
    assert not cmp(c, s2, c, s, y)["ok"]
    y2 = y.copy()
    y2[0, 2] *= np.float32(1 + 2e-5)
    assert not cmp(c, s, c, s, y, y2)["ok"]
    y2[0, 2] = y[0, 2] * np.float32(1 + 4e-6)
    assert cmp(c, s, c, s, y, y2)["ok"]
    # with the exact values given, y is measured against them instead of the fixed-order y
    y_exact = y.astype(np.float64)
    y_exact[0, 2] *= 1 + 1.5e-5
    assert not cmp(c, s, c, s, y, y, y_exact=y_exact)["ok"]
    y2[0, 2] = np.float32(y_exact[0, 2])
    assert cmp(c, s, c, s, y, y2, y_exact=y_exact)["ok"] and not cmp(c, s, c, s, y, y2)["ok"]
    # subnormal results: measured against 2^-126 (fp32 spacing 2^-149 there)
    tiny = np.zeros((1, 32), np.float32)
    tiny[0, 0] = np.float32(2.0 ** -140)
    tiny2 = tiny.copy()
    tiny2[0, 0] = np.float32(2.0 ** -140 + 2.0 ** -148)    # 1/256 relative, 2^-22 of 2^-126
    ct, st, _ = oracle.quantize_f32(tiny, np.eye(4, dtype=np.float32)[None], np.eye(8, dtype=np.float32)[None])
    assert cmp(ct, st, ct, st, tiny, tiny2)["ok"]
    tiny2[0, 0] = np.float32(2.0 ** -140 + 2.0 ** -133)    # 2^-7 of 2^-126: too far
    assert not cmp(ct, st, ct, st, tiny, tiny2)["ok"]
    assert not oracle.mx_compare(at_tie, s, c, s, y)["ok"]  # 1 of 32 codes is above the 1e-4 budget


def test_fwht_rejects_rows_longer_than_its_buffer():
    with pytest.raises(ValueError):
        oracle.fwht(np.zeros((2, 1 << 17), np.uint16))
