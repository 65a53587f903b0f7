"""GPU parity: the HIP path through the C ABI against the CPU oracle on the
same seeded inputs.

Two bars.  `assert_exact`: E8M0 scales, packed E2M1 codes and the fp32
transformed values bit-identical -- the fixed-order path, the comparators and
the element convert, which keep the oracle's fp32 evaluation order.
`assert_mx_close` (oracle.mx_compare): the tolerance of the matrix-core paths
and the offline weight side, whose fp32 order differs -- scales bit-exact,
codes bit-exact except adjacent-magnitude flips at rounding ties of the
oracle's y (at most 1e-4 of the codes), fp32 values within 1e-5 relative error
measured against max(|y_ref|, amax_block / 32).
"""
import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
kq = pytest.importorskip("paper_2607_21446_amd")

pytestmark = pytest.mark.gpu

AB_SPLITS = [(4, 8), (2, 16), (8, 4), (1, 32)]


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    kq.lib()
    yield


def dev_bf16(X):
    return torch.from_numpy(np.ascontiguousarray(X).view(np.int16)).view(torch.bfloat16).cuda()


def dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def assert_exact(got, want, what=""):
    cg, sg, yg = got
    cr, sr, yr = want
    assert np.array_equal(sg, sr), f"{what}: scales differ at {np.argwhere(sg != sr)[:5].tolist()}"
    assert np.array_equal(cg, cr), f"{what}: codes differ at {np.argwhere(cg != cr)[:5].tolist()}"
    if yr is not None:
        assert np.array_equal(yg.view(np.uint32), yr.view(np.uint32)), f"{what}: y differs"


def assert_mx_close(got, want, what="", y_exact=None):
    """The tolerance of a path whose fp32 order differs from the oracle's
    (oracle.mx_compare): scales identical; codes identical except adjacent
    flips (or a sign-only flip of magnitude 0) at most 1e-4 of them, each at a
    rounding decision of the oracle's y when the oracle's y is given; the
    path's y within 1e-5 of y_exact (the exact transform, oracle.transform_f64)
    when given, else of the oracle's fixed-order fp32 y."""
    cg, sg, yg = got
    cr, sr, yr = want
    rep = oracle.mx_compare(cg, sg, cr, sr, y_ref=yr, y=yg, y_exact=y_exact)
    assert rep["ok"], f"{what}: {rep}"


def gpu_quantize(X, A, B, want_y=True, exact=True):
    fn = kq.quantize_exact if exact else kq.quantize
    codes, scales, y = fn(dev_bf16(X), dev_f32(A), dev_f32(B), want_y=want_y)
    return host(codes), host(scales), (host(y) if want_y else None)


def gpu_quantize_packed(X, A, B, want_y=True):
    Ad, Bd = dev_f32(A), dev_f32(B)
    kpack = kq.pack_factors(Ad, Bd)
    codes, scales, y = kq.quantize_packed(dev_bf16(X), Ad, Bd, kpack, want_y=want_y)
    return host(codes), host(scales), (host(y) if want_y else None)


# ------------------------------------------------------------------ element encode
def test_e2m1_convert_exhaustive():
    """Every fp32 bit pattern with |v| <= 8 through the device convert at
    scale 2^0, against the oracle's nearest-magnitude rule."""
    hi = int(np.float32(8.0).view(np.uint32)) + 1
    chunk = 1 << 26
    for sign in (0, 1):
        for start in range(0, hi, chunk):
            n = min(chunk, hi - start)
            n += n % 2
            bits = torch.arange(start, start + n, dtype=torch.int64, device="cuda")
            bits = torch.clamp(bits, max=hi - 1).to(torch.int32)
            if sign:
                bits = bits | torch.tensor(-(1 << 31), dtype=torch.int32, device="cuda")
            v = bits.view(torch.float32)
            got = oracle.unpack_codes(host(kq.e2m1_encode(v, 127)))
            want = oracle.e2m1_codes(host(v), 127)
            assert np.array_equal(got, want), f"sign {sign} chunk {start:#x}"


@pytest.mark.parametrize("s", [0, 1, 2, 3, 100, 126, 128, 200, 252, 254])
def test_e2m1_convert_other_scales(s):
    rng = np.random.default_rng(s)
    mags = rng.random(1 << 20) * 8.0 * np.exp2(s - 127.0)
    v = (mags * np.where(rng.random(1 << 20) < 0.5, -1, 1))
    v = np.clip(v, -np.finfo(np.float32).max, np.finfo(np.float32).max).astype(np.float32)
    got = oracle.unpack_codes(host(kq.e2m1_encode(dev_f32(v), s)))
    assert np.array_equal(got, oracle.e2m1_codes(v, s))


# ------------------------------------------------------------------ small shapes, every variant
@pytest.mark.parametrize("ab", AB_SPLITS)
@pytest.mark.parametrize("per_block", [False, True])
@pytest.mark.parametrize("M,d", [(1, 32), (3, 64), (257, 1152), (64, 2240), (130, 3072)])
def test_kroquant_parity(ab, per_block, M, d):
    a, b = ab
    X = synth.activations(M, d, "student_t3", seed=M * 7 + d, chan_frac=0.005, chan_factor=50)
    A, B = synth.factors(a, b, d // 32 if per_block else 1, seed=d + a)
    want = oracle.quantize(X, A, B, want_y=True)
    assert_exact(gpu_quantize(X, A, B, exact=True), want, f"exact {ab} pb={per_block} {M}x{d}")
    ye = oracle.transform_f64(X, A, B)
    hot = gpu_quantize(X, A, B, exact=False)
    assert_mx_close(hot, want, f"mfma {ab} pb={per_block} {M}x{d}", ye)
    packed = gpu_quantize_packed(X, A, B)
    assert_mx_close(packed, want, f"packed {ab} pb={per_block} {M}x{d}", ye)


@pytest.mark.parametrize("M,d", [(1, 32), (3, 64), (257, 1152), (64, 2240), (130, 5600)])
def test_comparators_parity(M, d):
    X = synth.activations(M, d, "laplace", seed=M + d, chan_frac=0.02, chan_factor=20)
    Xd = dev_bf16(X)
    mult = synth.smoothquant_multipliers(X)
    c, s, y = kq.smoothquant(Xd, dev_f32(mult), want_y=True)
    assert_exact((host(c), host(s), host(y)), oracle.smoothquant(X, mult, want_y=True), "smooth")
    c, s, y = kq.hadamard32(Xd, want_y=True)
    assert_exact((host(c), host(s), host(y)), oracle.hadamard32(X, want_y=True), "hadamard")
    c, s = kq.mxfp4(Xd)
    cr, sr = oracle.mxfp4(X)
    assert_exact((host(c), host(s), None), (cr, sr, None), "mxfp4")


@pytest.mark.parametrize("M,d", [(1, 32), (3, 64), (257, 1152), (130, 5600)])
def test_stream_floor_outputs(M, d):
    """kq_stream_floor (the traffic-only timing aid) writes, per block, the XOR
    of its four 16-byte chunks and the low byte of that XOR's words 0 ^ 1;
    ragged unit counts included."""
    X = synth.activations(M, d, "normal", seed=M * d, chan_frac=0.0)
    o16, o1 = kq.stream_floor(dev_bf16(X))
    w = np.ascontiguousarray(X).view(np.uint32).reshape(M, d // 32, 4, 4)
    fold = w[:, :, 0] ^ w[:, :, 1] ^ w[:, :, 2] ^ w[:, :, 3]
    assert np.array_equal(host(o16).view(np.uint32).reshape(M, d // 32, 4), fold)
    assert np.array_equal(host(o1), ((fold[:, :, 0] ^ fold[:, :, 1]) & 0xFF).astype(np.uint8))


@pytest.mark.parametrize("M,d", [(37, 96), (300, 3072)])
def test_stream_probe_matches_stream_floor(M, d):
    """kq_stream_probe (the same traffic in other launch shapes) writes what
    kq_stream_floor writes, for one-pass and grid-stride shapes."""
    X = synth.activations(M, d, "normal", seed=M + d)
    Xd = dev_bf16(X)
    f16, f1 = (host(t) for t in kq.stream_floor(Xd))
    for waves, units, groups in ((1, 1, 0), (2, 4, 0), (16, 1, 0), (4, 2, 3), (1, 1, 5), (8, 4, 1)):
        o16, o1 = (host(t) for t in kq.stream_probe(Xd, waves, units, groups))
        assert np.array_equal(o16, f16) and np.array_equal(o1, f1), (waves, units, groups)


def test_timestamp_counts_at_100_mhz():
    """kq_timestamp: stamps around 1000 launches, on the launch stream and
    inside a captured graph, advance at the documented 100 MHz: they lie
    inside the HIP-event window around the same work and cover at least 97%
    of it (the rest is the host-side gap before the first stamp, or the
    graph's own launch)."""
    X = dev_bf16(synth.activations(4608, 3072, "normal", seed=5))
    f16, f1 = kq.stream_floor(X)
    ts = torch.zeros(4, dtype=torch.int64, device="cuda")
    st = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(st)
    kq.timestamp(ts, 0)
    for _ in range(1000):
        kq.stream_floor(X, out16=f16, out1=f1)
    kq.timestamp(ts, 1)
    b.record(st)
    torch.cuda.synchronize()
    t = host(ts)
    assert t[1] > t[0] > 0
    ratio = (t[1] - t[0]) / kq.TIMESTAMP_HZ * 1e3 / a.elapsed_time(b)
    assert 0.97 < ratio <= 1.001, ratio
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        kq.timestamp(ts, 2)
        for _ in range(1000):
            kq.stream_floor(X, out16=f16, out1=f1)
        kq.timestamp(ts, 3)
    g.replay()
    torch.cuda.synchronize()
    a.record(st)
    g.replay()
    b.record(st)
    torch.cuda.synchronize()
    t = host(ts)
    ratio = (t[3] - t[2]) / kq.TIMESTAMP_HZ * 1e3 / a.elapsed_time(b)
    assert 0.97 < ratio <= 1.001, ratio


def test_tiny_config_all_paths():
    w = synth.workload("tiny_256x1152")
    want = oracle.quantize(w.X, w.A, w.B, want_y=True)
    assert_exact(gpu_quantize(w.X, w.A, w.B), want, "tiny exact")
    assert_mx_close(gpu_quantize(w.X, w.A, w.B, exact=False), want, "tiny mfma", oracle.transform_f64(w.X, w.A, w.B))


# ------------------------------------------------------------------ edge blocks
def _edge_matrix():
    rows = []
    f = np.float32
    rows.append(np.zeros(64, f))                                            # all zero
    rows.append(np.concatenate([np.full(32, -0.0, f), np.zeros(32, f)]))     # -0.0 inputs
    sub = (np.arange(64, dtype=np.uint32) % 127 + 1).astype(np.uint32)      # bf16 subnormals
    rows.append((sub << 16).view(np.float32) * np.where(np.arange(64) % 3, 1, -1).astype(f))
    ties = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0] * 8, f)     # exact ties at s = 127
    ties[0] = 6.0
    rows.append(ties * np.where(np.arange(64) % 2, -1, 1).astype(f))
    sat = np.full(64, 7.0, f)                                               # saturation
    sat[0] = 7.5
    rows.append(sat)
    big = np.zeros(64, f)
    big[5] = np.float32((np.uint32(0x7F7F) << 16).view(np.float32))         # largest finite bf16
    big[40] = -big[5]
    rows.append(big)
    tiny = np.zeros(64, f)
    tiny[3] = (np.uint32(1) << 16).view(np.float32)                        # smallest bf16 subnormal
    rows.append(tiny)
    return synth.to_bf16_bits(np.stack(rows))


def _sweep_case(seed):
    """Shape, factors and input of one randomized case (seeded)."""
    rng = np.random.default_rng(1000 + seed)
    M = int(rng.integers(1, 700))
    d = 32 * int(rng.integers(1, 200))
    a = int(rng.choice([1, 2, 4, 8]))
    b = 32 // a
    nfac = d // 32 if rng.random() < 0.5 else 1
    dist = str(rng.choice(["normal", "student_t3", "laplace"]))
    X = synth.activations(M, d, dist, seed=2000 + seed, chan_frac=float(rng.choice([0.0, 0.01, 0.05])),
                          chan_factor=float(rng.choice([5.0, 50.0])))
    e = int(rng.integers(-60, 61))  # a power-of-two scale keeps the bf16 values exact
    x = (X.astype(np.uint32) << 16).view(np.float32) * np.float32(2.0 ** e)
    X = (x.view(np.uint32) >> 16).astype(np.uint16)
    # factor families of the method: perturbed identities (the calibrated transforms start at the identity or
    # a Hadamard and move little) at three strengths, and random orthogonal pairs (Hadamard-like, condition 1)
    kind = str(rng.choice(["identity+0.05", "identity+0.15", "identity+0.3", "orthogonal"]))

    def draw(n):
        if kind == "orthogonal":
            return np.stack([np.linalg.qr(rng.normal(size=(n, n)))[0] for _ in range(nfac)]).astype(np.float32)
        eps = float(kind.split("+")[1])
        return (np.eye(n) + eps * rng.normal(size=(nfac, n, n)) / np.sqrt(n)).astype(np.float32)

    A, B = draw(a), draw(b)
    return M, d, a, b, nfac, dist, e, kind, X, A, B


@pytest.mark.parametrize("seed", range(32))
def test_randomized_sweep(seed):
    """Seeded random cases -- rows 1..699, d = 32..6368, every split, shared or
    per-block factors (cond_inf(K) from 1
    to about 30), three input distributions with or without outlier
    channels, scaled by 2^-60..2^60; factors perturbed identities or random
    orthogonal pairs) -- through every quantizer entry point:
    the fixed-order path and the comparators bit-exact, the matrix-core paths
    (on the fly, packed, LU form) within the tolerance, and the y-less calls
    byte-identical to the calls that also write y."""
    M, d, a, b, nfac, dist, e, kind, X, A, B = _sweep_case(seed)
    what = f"seed {seed}: {M}x{d} ({a},{b}) nfac={nfac} {dist} 2^{e} {kind}"
    want = oracle.quantize(X, A, B, want_y=True)
    ye = oracle.transform_f64(X, A, B)
    assert_exact(gpu_quantize(X, A, B, exact=True), want, what + " exact")
    hot = gpu_quantize(X, A, B, exact=False)
    assert_mx_close(hot, want, what + " on the fly", ye)
    packed = gpu_quantize_packed(X, A, B)
    assert_mx_close(packed, want, what + " packed", ye)
    for got, full in ((gpu_quantize(X, A, B, want_y=False, exact=False), hot),
                      (gpu_quantize_packed(X, A, B, want_y=False), packed)):
        assert np.array_equal(got[0], full[0]) and np.array_equal(got[1], full[1]), what + " without y"
    lu = synth.lu_params(nfac, seed=4000 + seed)
    cr, sr, yr, _ = oracle.quantize_lu(X, lu, a, want_y=True)
    c, s, y, y16 = gpu_quantize_lu(X, lu, a)
    assert_mx_close((c, s, y), (cr, sr, yr), what + " lu", oracle.transform_f64(X, *oracle.lu_factors_f32(lu, a)))
    assert np.array_equal(y16, oracle.f32_to_bf16(y)), what + " y16"
    Xd = dev_bf16(X)
    mult = synth.smoothquant_multipliers(X)
    c, s, y = kq.smoothquant(Xd, dev_f32(mult), want_y=True)
    assert_exact((host(c), host(s), host(y)), oracle.smoothquant(X, mult, want_y=True), what + " smooth")
    c, s, y = kq.hadamard32(Xd, want_y=True)
    assert_exact((host(c), host(s), host(y)), oracle.hadamard32(X, want_y=True), what + " hadamard")
    c, s = kq.mxfp4(Xd)
    cr, sr = oracle.mxfp4(X)
    assert_exact((host(c), host(s), None), (cr, sr, None), what + " mxfp4")


def test_edge_blocks_plain_smooth_hadamard():
    X = _edge_matrix()
    Xd = dev_bf16(X)
    c, s = kq.mxfp4(Xd)
    cr, sr = oracle.mxfp4(X)
    assert_exact((host(c), host(s), None), (cr, sr, None), "mxfp4 edges")
    one = np.ones(64, np.float32)
    c, s, y = kq.smoothquant(Xd, dev_f32(one), want_y=True)
    assert_exact((host(c), host(s), host(y)), oracle.smoothquant(X, one, want_y=True), "smooth edges")
    # Hadamard keeps a lone largest-bf16 value finite (/sqrt(32)); skip no row
    c, s, y = kq.hadamard32(Xd, want_y=True)
    assert_exact((host(c), host(s), host(y)), oracle.hadamard32(X, want_y=True), "hadamard edges")


@pytest.mark.parametrize("ab", AB_SPLITS)
def test_edge_blocks_kron(ab):
    a, b = ab
    X = _edge_matrix()
    X = X[np.arange(X.shape[0]) != 5]  # an amplifying transform overflows the largest bf16
    A, B = synth.factors(a, b, 2, seed=3)
    want = oracle.quantize(X, A, B, want_y=True)
    assert_exact(gpu_quantize(X, A, B), want, f"kron edges {ab}")
    assert_mx_close(gpu_quantize(X, A, B, exact=False), want, f"mfma edges {ab}", oracle.transform_f64(X, A, B))
    # identity factors: plain MXFP4 (the -0.0 row excepted, products give +0.0);
    # on the matrix-core path every block max here is a power of two or on a
    # binade edge, so this also drives the exact re-evaluation of tiles
    Ai = np.eye(a, dtype=np.float32)[None]
    Bi = np.eye(b, dtype=np.float32)[None]
    keep = np.arange(X.shape[0]) != 1
    cr, sr = oracle.mxfp4(X[keep])
    for exact in (True, False):
        c, s, _ = gpu_quantize(X[keep], Ai, Bi, exact=exact)
        assert np.array_equal(c, cr) and np.array_equal(s, sr), exact


@pytest.mark.parametrize("ab", AB_SPLITS)
def test_zero_blocks_signed_zeros(ab):
    """All-zero input blocks: the matrix-core paths skip the re-evaluation only
    when the fixed order provably gives +0 everywhere (inputs +0, no factor row
    with every sign bit set); otherwise the signed zeros of the fixed order
    decide the codes.  Codes and scales must equal the oracle exactly here."""
    a, b = ab
    M, d = 70, 2240
    X = synth.activations(M, d, "normal", seed=21)
    X[::3] = 0                       # +0 rows
    X[1::7, 64:160] = 0x8000         # -0 runs
    A, B = synth.factors(a, b, d // 32, seed=22)
    A[3, 0, :] = -np.abs(A[3, 0, :]) - 0.01   # a row of A with every sign bit set (block 3)
    B[5, -1, :] = -np.abs(B[5, -1, :]) - 0.01  # and one of B (block 5)
    for nfac_mode in ("shared", "per_block"):
        Af, Bf = (A[3:4], B[3:4]) if nfac_mode == "shared" else (A, B)
        want = oracle.quantize(X, Af, Bf, want_y=True)
        ye = oracle.transform_f64(X, Af, Bf)
        for got in (gpu_quantize(X, Af, Bf, exact=False), gpu_quantize_packed(X, Af, Bf)):
            assert np.array_equal(got[1], want[1]), f"{ab} {nfac_mode}: scales"
            zero_rows = np.zeros(M, bool)
            zero_rows[::3] = True
            assert np.array_equal(got[0][zero_rows], want[0][zero_rows]), f"{ab} {nfac_mode}: zero-row codes"
            assert_mx_close(got, want, f"{ab} {nfac_mode}", ye)


@pytest.mark.parametrize("ab", [(4, 8), (2, 16)])
def test_binade_edge_stress(ab):
    """Blocks whose fixed-order amax lies within a few binade-edge windows of a
    power of two, gathered from 2M random blocks.  Both matrix-core paths
    re-evaluate those inside their window and must get every other one right
    from the matrix product alone: scales identical to the oracle's."""
    a, b = ab
    A, B = synth.factors(a, b, 1, seed=41)
    pool = synth.activations(8192, 8192, "student_t3", seed=42)     # 2,097,152 blocks
    _, sr, yr = oracle.quantize(pool, A, B, want_y=True)
    amax = np.abs(yr.reshape(-1, 32)).max(-1).astype(np.float32)
    mant = (amax.view(np.uint32) & 0x7FFFFF).astype(np.int64)
    dist = np.minimum(mant, (1 << 23) - mant)                        # to the nearer power of two, in 2^-23 units
    # the packed path's window is T = ceil(2^7 cond_inf) units; take up to 4 T
    A64, B64 = A[0].astype(np.float64), B[0].astype(np.float64)
    cinf = lambda F: np.abs(F).sum(1).max() * np.abs(np.linalg.inv(F)).sum(1).max()
    T = int(np.ceil(128 * 1.01 * cinf(A64) * cinf(B64)))
    pick = np.flatnonzero(dist <= 4 * T)
    assert pick.size >= 512, pick.size
    blocks = pool.reshape(-1, 32)[pick]
    nb = 96
    rows = int(np.ceil(blocks.shape[0] / nb))
    X = np.concatenate([blocks, blocks[: rows * nb - blocks.shape[0]]]).reshape(rows, nb * 32)
    want = oracle.quantize(X, A, B, want_y=True)
    ye = oracle.transform_f64(X, A, B)
    for name, got in (("onthefly", gpu_quantize(X, A, B, exact=False)), ("packed", gpu_quantize_packed(X, A, B))):
        assert_mx_close(got, want, f"{ab} {name} near-edge blocks ({pick.size} picked, T={T})", ye)


def gpu_quantize_lu(X, lu, a):
    c, s, y, y16 = kq.quantize_lu(dev_bf16(X), dev_f32(lu), a, want_y=True, want_y16=True)
    return host(c), host(s), host(y), host(y16.view(torch.int16)).view(np.uint16)


@pytest.mark.parametrize("a", [4, 2, 8, 1])
@pytest.mark.parametrize("per_block", [False, True])
@pytest.mark.parametrize("M,d", [(77, 2240), (256, 1152)])
def test_kroquant_lu_parity(a, per_block, M, d):
    """K2-form factors decoded on chip (kq_quantize_lu) against the oracle's
    fp32 decode + fixed-order quantizer; the bf16 output is the rounding of
    the fp32 values the codes came from."""
    X = synth.activations(M, d, "student_t3", seed=61, chan_frac=0.02, chan_factor=20.0)
    X[3] = 0                                  # an all-zero row
    lu = synth.lu_params(d // 32 if per_block else 1, seed=62 + a)
    cr, sr, yr, y16r = oracle.quantize_lu(X, lu, a, want_y=True)
    c, s, y, y16 = gpu_quantize_lu(X, lu, a)
    assert_mx_close((c, s, y), (cr, sr, yr), f"lu a={a} per_block={per_block}",
                    oracle.transform_f64(X, *oracle.lu_factors_f32(lu, a)))
    assert np.array_equal(y16, oracle.f32_to_bf16(y)), "y16 is not bf16(y)"
    assert (y16 != y16r).mean() <= 1e-3


def test_kroquant_lu_hadamard_init():
    """LU(1/sqrt2, 1/sqrt2, 1) for every factor is the Hadamard init: the
    codes and scales match the Hadamard-32 comparator up to tie flips."""
    X = synth.activations(128, 3072, "normal", seed=63)
    h = np.float32(1 / np.sqrt(2))
    lu = np.array([[[h, h, 1.0]] * 5], dtype=np.float32)
    want = oracle.hadamard32(X, want_y=True)
    for a in (4, 1):
        c, s, y, _ = gpu_quantize_lu(X, lu, a)
        ug, ur = oracle.unpack_codes(c), oracle.unpack_codes(want[0])
        assert np.array_equal(s, want[1])
        assert (ug != ur).mean() <= 1e-4
        assert np.max(np.abs(y - want[2])) <= 1e-5 * np.abs(want[2]).max()


@pytest.mark.parametrize("d", [32, 64, 256, 1024, 2048, 4096, 8192, 16384])
def test_fwht_parity(d):
    """Full-row FWHT comparator: bit-identical to the oracle's butterflies
    (every pass layout, including partial last passes and ragged row counts)."""
    M = {32: 300, 64: 130, 256: 37, 1024: 19, 2048: 9, 4096: 7, 8192: 3, 16384: 2}[d]
    X = synth.activations(M, d, "student_t3", seed=71, chan_frac=0.01, chan_factor=40.0)
    X[M // 2] = 0
    want = oracle.fwht(X, want_y=True)
    c, s_, y = kq.fwht(dev_bf16(X), want_y=True)
    assert_exact((host(c), host(s_), host(y)), want, f"fwht d={d}")


def test_hip_graph_replays_match_eager():
    """The hot-path and comparator launches captured into one HIP graph (as the
    benchmark's power-of-two-d table does) and replayed three times, with eager
    work and synchronizations between the replays: every replay reproduces the
    eager outputs (no allocation, memset or host sync inside the calls)."""
    X = synth.activations(512, 4096, "student_t3", seed=81)
    A, B = synth.factors(4, 8, 1, seed=82)
    lu = synth.lu_params(1, seed=83)
    Xd, Ad, Bd, lud = dev_bf16(X), dev_f32(A), dev_f32(B), dev_f32(lu)
    mult = dev_f32(synth.smoothquant_multipliers(X))
    kpack = kq.pack_factors(Ad, Bd)
    outs = [(torch.empty((512, 2048), dtype=torch.uint8, device="cuda"),
             torch.empty((512, 128), dtype=torch.uint8, device="cuda")) for _ in range(4)]
    calls = [
        lambda c, s: kq.quantize_packed(Xd, Ad, Bd, kpack, codes=c, scales=s),
        lambda c, s: kq.quantize_lu(Xd, lud, 4, codes=c, scales=s),
        lambda c, s: kq.smoothquant(Xd, mult, codes=c, scales=s),
        lambda c, s: kq.fwht(Xd, codes=c, scales=s),
    ]
    for call, (c, s) in zip(calls, outs):
        call(c, s)
    eager = [(host(c).copy(), host(s).copy()) for c, s in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for call, (c, s) in zip(calls, outs):
            call(c, s)
    other = dev_bf16(synth.activations(256, 1024, "normal", seed=84))
    for rep in range(3):
        for c, s in outs:
            c.fill_(0xAB)
            s.fill_(0xCD)
        kq.mxfp4(other)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, (c, s) in enumerate(outs):
            assert np.array_equal(host(c), eager[k][0]) and np.array_equal(host(s), eager[k][1]), (rep, k)


# ------------------------------------------------------------------ layout, guards, determinism
def test_guard_bands_and_full_coverage():
    M, d = 77, 2240
    X = synth.activations(M, d, "normal", seed=1)
    A, B = synth.factors(4, 8, 1, seed=2)
    want = oracle.quantize(X, A, B, want_y=True)
    G = 4096
    for canary in (0xA5, 0x5A):
        cbuf = torch.full((M * d // 2 + 2 * G,), canary, dtype=torch.uint8, device="cuda")
        sbuf = torch.full((M * d // 32 + 2 * G,), canary, dtype=torch.uint8, device="cuda")
        ybuf = torch.full((M * d + 2 * G,), float("nan"), dtype=torch.float32, device="cuda")
        codes = cbuf[G:G + M * d // 2].view(M, d // 2)
        scales = sbuf[G:G + M * d // 32].view(M, d // 32)
        y = ybuf[G:G + M * d].view(M, d)
        kq.quantize_exact(dev_bf16(X), dev_f32(A), dev_f32(B), codes=codes, scales=scales, y=y)
        cb, sb, yb = host(cbuf), host(sbuf), host(ybuf)
        assert np.all(cb[:G] == canary) and np.all(cb[-G:] == canary)
        assert np.all(sb[:G] == canary) and np.all(sb[-G:] == canary)
        assert np.all(np.isnan(yb[:G])) and np.all(np.isnan(yb[-G:]))
        assert_exact((cb[G:-G].reshape(M, -1), sb[G:-G].reshape(M, -1), yb[G:-G].reshape(M, d)), want)
        cbuf.fill_(canary)
        sbuf.fill_(canary)
        ybuf.fill_(float("nan"))
        kq.quantize(dev_bf16(X), dev_f32(A), dev_f32(B), codes=codes, scales=scales, y=y)
        cb, sb, yb = host(cbuf), host(sbuf), host(ybuf)
        assert np.all(cb[:G] == canary) and np.all(cb[-G:] == canary)
        assert np.all(sb[:G] == canary) and np.all(sb[-G:] == canary)
        assert np.all(np.isnan(yb[:G])) and np.all(np.isnan(yb[-G:]))
        assert_mx_close((cb[G:-G].reshape(M, -1), sb[G:-G].reshape(M, -1), yb[G:-G].reshape(M, d)), want,
                        "guard bands", oracle.transform_f64(X, A, B))


def test_flat_and_column_mappings_agree():
    """nfac = 1 runs the flat mapping, nfac = d/32 the column mapping: with
    every per-block pair equal to the shared one they must agree bit for bit."""
    M, d = 300, 3072
    X = synth.activations(M, d, "student_t3", seed=4, chan_frac=0.005, chan_factor=50)
    A, B = synth.factors(4, 8, 1, seed=6)
    for exact in (True, False):
        g1 = gpu_quantize(X, A, B, exact=exact)
        g2 = gpu_quantize(X, np.repeat(A, d // 32, 0), np.repeat(B, d // 32, 0), exact=exact)
        assert_exact(g1, g2)
        g3 = gpu_quantize(X, A, B, exact=exact)
        assert_exact(g1, g3)


def test_non_default_stream():
    M, d = 512, 3072
    X = synth.activations(M, d, "normal", seed=9)
    A, B = synth.factors(4, 8, 1, seed=10)
    s = torch.cuda.Stream()
    Xd, Ad, Bd = dev_bf16(X), dev_f32(A), dev_f32(B)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        c, sc, y = kq.quantize_exact(Xd, Ad, Bd, want_y=True)
        c2, sc2, y2 = kq.quantize(Xd, Ad, Bd, want_y=True)
    s.synchronize()
    want = oracle.quantize(X, A, B, want_y=True)
    assert_exact((c.cpu().numpy(), sc.cpu().numpy(), y.cpu().numpy()), want)
    assert_mx_close((c2.cpu().numpy(), sc2.cpu().numpy(), y2.cpu().numpy()), want, "stream",
                    oracle.transform_f64(X, A, B))


def test_binding_rejects_inconsistent_buffers():
    """Caller-supplied buffers that do not match the call's sizes, factor
    pair counts or device are refused by the binding before any launch."""
    X = dev_bf16(np.zeros((8, 64), np.uint16))
    A, B = synth.factors(4, 8, 1, seed=1)
    Ad, Bd = dev_f32(A), dev_f32(B)
    u8 = lambda n: torch.empty(n, dtype=torch.uint8, device="cuda")
    with pytest.raises(ValueError):
        kq.quantize(X, Ad, Bd, codes=u8(8 * 32 - 16))
    with pytest.raises(ValueError):
        kq.quantize(X, Ad, Bd, scales=u8(8))
    with pytest.raises(ValueError):
        kq.quantize(X, Ad, dev_f32(np.repeat(B, 2, 0)))
    with pytest.raises(TypeError):
        kq.quantize(X, Ad.cpu(), Bd.cpu())          # host factors
    kp = kq.pack_factors(Ad, Bd)
    with pytest.raises(ValueError):
        kq.quantize_packed(X, Ad, Bd, kp[:-16])
    with pytest.raises(ValueError):
        kq.smoothquant(X, dev_f32(np.ones(63, np.float32)))
    with pytest.raises(ValueError):
        kq.quantize_lu(X, dev_f32(np.ones((1, 5, 3), np.float32)), 4, y16=torch.empty((8, 32), dtype=torch.bfloat16,
                                                                                     device="cuda"))
    torch.cuda.synchronize()


# ------------------------------------------------------------------ weight side
@pytest.mark.parametrize("ab", AB_SPLITS)
@pytest.mark.parametrize("per_block", [False, True])
def test_weight_transform(ab, per_block):
    a, b = ab
    o, d = 96, 1152
    W = synth.activations(o, d, "normal", seed=a * 3 + b, chan_frac=0.0)
    A, B = synth.factors(a, b, d // 32 if per_block else 1, seed=a + 11)
    Wt, c, s = kq.weight_transform(dev_bf16(W), torch.from_numpy(A), torch.from_numpy(B))
    got = (host(c), host(s), host(Wt))
    yr, cr, sr = oracle.weight_transform(W, A, B)
    assert_mx_close(got, (cr, sr, yr), f"weight {ab}")
    # eq. (1): <x T, w T^-T> = <x, w>
    X = synth.activations(8, d, "normal", seed=5)
    _, _, y = gpu_quantize(X, A, B, exact=False)
    lhs = y.astype(np.float64) @ got[2].astype(np.float64).T
    xf, wf = oracle.bf16_to_f32(X).astype(np.float64), oracle.bf16_to_f32(W).astype(np.float64)
    assert np.max(np.abs(lhs - xf @ wf.T) / (np.abs(xf) @ np.abs(wf).T)) < 2e-5


# ------------------------------------------------------------------ W4A4 GEMM consumer
def _rand_mx(rows, K, seed):
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 256, (rows, K // 2), dtype=np.uint8)
    scales = rng.integers(110, 140, (rows, K // 32), dtype=np.uint8)
    return codes, scales


def _gemm_tolerance(ac, as_, bc, bs):
    # fp32 accumulation of K exact products in any order: |error| <= K u sum |a||b|
    K = ac.shape[1] * 2
    return K * 2.0 ** -24 * (np.abs(oracle.dequantize(ac, as_)) @ np.abs(oracle.dequantize(bc, bs)).T)


@pytest.mark.parametrize("M,N,K", [(77, 200, 2240), (128, 128, 64), (33, 70, 1120), (300, 257, 3072), (1, 1, 32),
                                   (5, 3, 128), (64, 130, 256), (130, 64, 384), (200, 200, 512), (129, 127, 1280),
                                   (3072, 2304, 128), (3000, 2200, 384), (2500, 2470, 1664)])
def test_mxfp4_gemm_parity(M, N, K):
    """C = deq(A) deq(B)^T on the matrix cores against the oracle's fp64
    product, within the fp32 accumulation bound; ragged tiles, odd block
    counts along K, and the accumulate mode.  The three largest shapes have at
    least 96 tiles of 256 x 256 and so run the large-tile kernel (the last two
    with ragged tiles in both directions; the last one with 13 K stages, so
    every stage buffer is refilled several times and the stage count is not a
    multiple of the three buffers)."""
    ac, as_ = _rand_mx(M, K, seed=M + K)
    bc, bs = _rand_mx(N, K, seed=N + 2 * K)
    ref = oracle.mxfp4_gemm(ac, as_, bc, bs)
    tol = _gemm_tolerance(ac, as_, bc, bs)
    t = lambda a: torch.from_numpy(a).cuda()
    C = host(kq.mxfp4_gemm(t(ac), t(as_), t(bc), t(bs)))
    assert C.shape == (M, N)
    assert np.all(np.abs(C - ref) <= tol), np.max(np.abs(C - ref) - tol)
    C0 = np.random.default_rng(7).normal(size=(M, N)).astype(np.float32)
    Cd = t(C0)
    kq.mxfp4_gemm(t(ac), t(as_), t(bc), t(bs), C=Cd, accumulate=True)
    assert np.all(np.abs(host(Cd) - (ref + C0)) <= tol + 2.0 ** -23 * np.abs(ref + C0))


@pytest.mark.parametrize("M,N,K", [(77, 200, 2240), (33, 70, 1120), (300, 257, 3072), (5, 3, 128), (3000, 2200, 384),
                                   (2500, 2470, 1664)])
def test_mxfp4_gemm_bf16_output(M, N, K):
    """kq_mxfp4_gemm_bf16: the fp32 call's product rounded to bf16 (nearest
    even) element by element -- the same matrix-core sums, one rounding --
    and so within half a bf16 step of the oracle product plus the fp32
    accumulation bound; every kernel the dispatcher picks (small, 128 x 128
    and 256 x 256 tiles, ragged edges)."""
    ac, as_ = _rand_mx(M, K, seed=M + 3 * K)
    bc, bs = _rand_mx(N, K, seed=N + 5 * K)
    t = lambda a: torch.from_numpy(a).cuda()
    C32 = kq.mxfp4_gemm(t(ac), t(as_), t(bc), t(bs))
    C16 = kq.mxfp4_gemm(t(ac), t(as_), t(bc), t(bs), out_dtype=torch.bfloat16)
    c16 = host(C16.view(torch.int16)).view(np.uint16)
    assert np.array_equal(c16, oracle.f32_to_bf16(host(C32)))
    ref = oracle.mxfp4_gemm(ac, as_, bc, bs)
    tol = _gemm_tolerance(ac, as_, bc, bs)
    got = oracle.bf16_to_f32(c16).astype(np.float64)
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * (np.abs(ref) + tol) + tol)


@pytest.mark.parametrize("M,N,K", [(256, 512, 1024), (1024, 768, 3072)])
def test_vendor_mxfp4_gemm_reads_the_same_layout(M, N, K):
    """An independent reading of the operand layout: the vendor's MXFP4
    product (torch._scaled_mm on E2M1 codes, two per byte with element 2i in
    the low nibble, and E8M0 scales per 32-element block, bf16 output) on the
    codes and scales as the quantizers write them, against the oracle's fp64
    product and against kq_mxfp4_gemm_bf16.  The vendor's bf16 results are
    not the nearest bf16 of their sums (they sit up to one bf16 step from the
    exact product, mostly toward zero: a median relative error of 2.6e-3 on
    random operands, against kq_mxfp4_gemm_bf16's correctly rounded fp32
    sums), so the bound is one bf16 step; a misread nibble order, scale or
    row would be off by far more."""
    if not (hasattr(torch, "float4_e2m1fn_x2") and hasattr(torch, "float8_e8m0fnu")):
        pytest.skip("this torch has no MXFP4 dtypes")
    ac, as_ = _rand_mx(M, K, seed=M + 7 * K)
    bc, bs = _rand_mx(N, K, seed=N + 11 * K)
    t = lambda a: torch.from_numpy(a).cuda()
    try:
        V = torch._scaled_mm(t(ac).view(torch.float4_e2m1fn_x2), t(bc).view(torch.float4_e2m1fn_x2).t(),
                             scale_a=t(as_).view(torch.float8_e8m0fnu), scale_b=t(bs).view(torch.float8_e8m0fnu),
                             out_dtype=torch.bfloat16)
        torch.cuda.synchronize()
    except RuntimeError as e:
        pytest.skip(f"the vendor library has no MXFP4 product here: {e!r:.200}")
    got = host(V.float()).astype(np.float64)
    ref = oracle.mxfp4_gemm(ac, as_, bc, bs)
    tol = _gemm_tolerance(ac, as_, bc, bs)
    step = 2.0 ** -7 * (np.abs(ref) + tol)  # one bf16 step at |ref|, or more
    assert np.all(np.abs(got - ref) <= step + tol), np.max(np.abs(got - ref) / (step + tol))
    ours = oracle.bf16_to_f32(host(kq.mxfp4_gemm(t(ac), t(as_), t(bc), t(bs), out_dtype=torch.bfloat16)
                                   .view(torch.int16)).view(np.uint16)).astype(np.float64)
    assert np.all(np.abs(got - ours) <= 1.5 * step + 2 * tol)


def test_w4a4_layer_end_to_end():
    """X -> kq_quantize_packed, W -> kq_weight_transform, then kq_mxfp4_gemm:
    the layer output against the oracle's W4A4 product, and E(T) (Sec. 3.1)
    against the oracle's layer error."""
    M, N, d = 256, 192, 3072
    X = synth.activations(M, d, "student_t3", seed=91, chan_frac=0.005, chan_factor=50.0)
    W = synth.activations(N, d, "normal", seed=92, chan_frac=0.0)
    A, B = synth.factors(4, 8, 1, seed=93)
    Ad, Bd = dev_f32(A), dev_f32(B)
    kpack = kq.pack_factors(Ad, Bd)
    xc, xs, _ = kq.quantize_packed(dev_bf16(X), Ad, Bd, kpack)
    _, wc, ws = kq.weight_transform(dev_bf16(W), torch.from_numpy(A), torch.from_numpy(B))
    C = host(kq.mxfp4_gemm(xc, xs, wc, ws))
    e_ref, (oxc, oxs), (owc, ows), xw = oracle.layer_error(X, W, A, B)
    ref = oracle.mxfp4_gemm(host(xc), host(xs), host(wc), host(ws))
    assert np.all(np.abs(C - ref) <= _gemm_tolerance(host(xc), host(xs), host(wc), host(ws)))
    e_gpu = float(np.linalg.norm(xw - C))
    assert abs(e_gpu - e_ref) <= 1e-3 * e_ref, (e_gpu, e_ref)


# ------------------------------------------------------------------ full-size workloads
FULL = ["pixart_8192x1152", "pixart_8192x4608", "sana_4096x2240", "sana_4096x5600", "flux_4608x3072",
        "flux_4608x12288"]


@pytest.mark.parametrize("name", FULL)
def test_full_size_workloads(name):
    """Every output of the DiT-shaped workloads, KroQuant and the comparators.
    The matrix-core calls run twice, with and without the fp32 output: the
    launch without it is the kernel specialisation the benchmark times, and
    its codes and scales must be byte-identical to those of the launch with
    it and within the tolerance of the oracle (flips at ties of the oracle's y)."""
    w = synth.workload(name)
    Xd = dev_bf16(w.X)
    Ad, Bd = dev_f32(w.A), dev_f32(w.B)
    cr, sr, yr = oracle.quantize(w.X, w.A, w.B, want_y=True)
    ye = oracle.transform_f64(w.X, w.A, w.B)
    c, s, _ = kq.quantize_exact(Xd, Ad, Bd)
    assert_exact((host(c), host(s), None), (cr, sr, None), name)
    kp = kq.pack_factors(Ad, Bd)
    for what, run in (("mfma", lambda wy: kq.quantize(Xd, Ad, Bd, want_y=wy)),
                      ("packed", lambda wy: kq.quantize_packed(Xd, Ad, Bd, kp, want_y=wy))):
        c, s, y = run(True)
        with_y = (host(c), host(s), host(y))
        assert_mx_close(with_y, (cr, sr, yr), f"{name} {what}", ye)
        c, s, _ = run(False)
        c, s = host(c), host(s)
        assert np.array_equal(c, with_y[0]) and np.array_equal(s, with_y[1]), f"{name} {what}: y on/off differ"
        assert_mx_close((c, s, None), (cr, sr, yr), f"{name} {what} (no y output)")
    c, s, _ = kq.smoothquant(Xd, dev_f32(w.mult))
    cr, sr, _ = oracle.smoothquant(w.X, w.mult)
    assert_exact((host(c), host(s), None), (cr, sr, None), name + " smooth")
    c, s, _ = kq.hadamard32(Xd)
    cr, sr, _ = oracle.hadamard32(w.X)
    assert_exact((host(c), host(s), None), (cr, sr, None), name + " hadamard")


@pytest.mark.parametrize("name", ["flux_4608x3072", "flux_4608x12288"])
def test_lu_form_full_size(name):
    """kq_quantize_lu at the FLUX shapes with one shared set of 15 LU
    parameters, launched as the benchmark launches it (codes and scales only)
    and with both 16- and 32-bit outputs: identical codes and scales, within
    the tolerance of the oracle's decode + fixed-order quantizer."""
    w = synth.workload(name)
    lu = synth.lu_params(1, seed=7)
    cr, sr, yr, _ = oracle.quantize_lu(w.X, lu, 4, want_y=True)
    Xd, lud = dev_bf16(w.X), dev_f32(lu)
    c, s, _, _ = kq.quantize_lu(Xd, lud, 4)
    c, s = host(c), host(s)
    assert_mx_close((c, s, None), (cr, sr, yr), f"{name} lu")
    c2, s2, y, y16 = kq.quantize_lu(Xd, lud, 4, want_y=True, want_y16=True)
    assert np.array_equal(host(c2), c) and np.array_equal(host(s2), s), f"{name} lu: outputs on/off differ"
    y = host(y)
    assert_mx_close((c, s, y), (cr, sr, yr), f"{name} lu (with y)", oracle.transform_f64(w.X, *oracle.lu_factors_f32(lu, 4)))
    assert np.array_equal(host(y16.view(torch.int16)).view(np.uint16), oracle.f32_to_bf16(y))


@pytest.mark.parametrize("ab", [(2, 16), (8, 4), (1, 32)])
def test_other_splits_full_size(ab):
    """The (a, b) splits other than the workloads' (4, 8), at FLUX 4608x3072
    (6912 full units) with one shared near-identity pair: every output of the
    fixed-order path bit for bit; the on-the-fly and packed calls launched as
    the benchmark launches the hot path (codes and scales only) and with the
    fp32 output, identical codes and scales either way and within the
    tolerance of the oracle; and the LU form with a = the split's a."""
    a, b = ab
    w = synth.workload("flux_4608x3072")
    A, B = synth.factors(a, b, 1, seed=100 + a)
    Xd, Ad, Bd = dev_bf16(w.X), dev_f32(A), dev_f32(B)
    cr, sr, yr = oracle.quantize(w.X, A, B, want_y=True)
    ye = oracle.transform_f64(w.X, A, B)
    c, s, y = kq.quantize_exact(Xd, Ad, Bd, want_y=True)
    assert_exact((host(c), host(s), host(y)), (cr, sr, yr), f"{ab} exact")
    kp = kq.pack_factors(Ad, Bd)
    for what, run in (("onthefly", lambda wy: kq.quantize(Xd, Ad, Bd, want_y=wy)),
                      ("packed", lambda wy: kq.quantize_packed(Xd, Ad, Bd, kp, want_y=wy))):
        c, s, _ = run(False)
        c, s = host(c), host(s)
        assert_mx_close((c, s, None), (cr, sr, yr), f"{ab} {what} (no y output)")
        c2, s2, y = run(True)
        assert np.array_equal(host(c2), c) and np.array_equal(host(s2), s), f"{ab} {what}: y on/off differ"
        assert_mx_close((c, s, host(y)), (cr, sr, yr), f"{ab} {what}", ye)
    lu = synth.lu_params(1, seed=200 + a)
    cr, sr, yr, _ = oracle.quantize_lu(w.X, lu, a, want_y=True)
    c, s, y, _ = kq.quantize_lu(Xd, dev_f32(lu), a, want_y=True)
    assert_mx_close((host(c), host(s), host(y)), (cr, sr, yr), f"{ab} lu",
                    oracle.transform_f64(w.X, *oracle.lu_factors_f32(lu, a)))


def test_per_block_strips_ragged():
    """Per-block factors on a shape whose strips take two 64-row steps, whose
    last strip has one step, last row block two rows and last column strip
    four column blocks (M = 4610, d = 12160, 380 blocks per row): every row
    against the oracle, and the flat mapping (one shared pair) against the
    column mapping (that pair repeated per block) bit for bit, y included,
    which checks the per-step binade-edge records."""
    M, d = 4610, 12160
    X = synth.activations(M, d, "student_t3", seed=21, chan_frac=0.01, chan_factor=40)
    A, B = synth.factors(4, 8, d // 32, seed=22)
    cr, sr, yr = oracle.quantize(X, A, B, want_y=True)
    ye = oracle.transform_f64(X, A, B)
    Xd, Ad, Bd = dev_bf16(X), dev_f32(A), dev_f32(B)
    c, s, y = kq.quantize(Xd, Ad, Bd, want_y=True)
    assert_mx_close((host(c), host(s), host(y)), (cr, sr, yr), "on the fly", ye)
    c, s, y = kq.quantize_packed(Xd, Ad, Bd, kq.pack_factors(Ad, Bd), want_y=True)
    assert_mx_close((host(c), host(s), host(y)), (cr, sr, yr), "packed", ye)
    del y, ye
    A1, B1 = synth.factors(4, 8, 1, seed=23)
    nb = d // 32
    g1 = gpu_quantize(X, A1, B1, exact=False)
    g2 = gpu_quantize(X, np.repeat(A1, nb, 0), np.repeat(B1, nb, 0), exact=False)
    assert_exact(g1, g2, "on the fly, flat vs column")
    g1 = gpu_quantize_packed(X, A1, B1)
    g2 = gpu_quantize_packed(X, np.repeat(A1, nb, 0), np.repeat(B1, nb, 0))
    # with a pair per block the packed call builds the K terms on chip that the pack holds and takes
    # each pair's window from its pack, so it re-evaluates the same blocks: identical, y included
    assert_exact(g1, g2, "packed, flat vs column")


@pytest.mark.parametrize("a", [4, 1])
def test_per_block_lu_strips_ragged(a):
    """The LU form (15 parameters per pair decoded on chip) on the ragged
    multi-step shape: every row against the oracle's decode + fixed-order
    quantizer, y16 = bf16(y), and one shared parameter set (flat mapping)
    against the same set repeated per block (column mapping) bit for bit."""
    M, d = 4610, 12160
    nb = d // 32
    X = synth.activations(M, d, "student_t3", seed=31, chan_frac=0.01, chan_factor=40)
    lu = synth.lu_params(nb, seed=32 + a)
    cr, sr, yr, _ = oracle.quantize_lu(X, lu, a, want_y=True)
    c, s, y, y16 = gpu_quantize_lu(X, lu, a)
    assert_mx_close((c, s, y), (cr, sr, yr), f"lu a={a}", oracle.transform_f64(X, *oracle.lu_factors_f32(lu, a)))
    assert np.array_equal(y16, oracle.f32_to_bf16(y)), "y16 is not bf16(y)"
    del y, y16, yr
    lu1 = synth.lu_params(1, seed=33 + a)
    g1 = gpu_quantize_lu(X, lu1, a)
    g2 = gpu_quantize_lu(X, np.repeat(lu1, nb, 0), a)
    for u, v, what in zip(g1, g2, ("codes", "scales", "y", "y16")):
        assert np.array_equal(np.ascontiguousarray(u).view(np.uint8), np.ascontiguousarray(v).view(np.uint8)), \
            f"lu a={a}: flat vs column {what}"


@pytest.mark.parametrize("name", ["large_18432x12288", "large_18432x12288_2x16"])
def test_large_per_block_every_row(name):
    """Large per-block-factor workload (18432 x 12288, 384 factor pairs) at
    full size, every output: the fixed-order path bit for bit, and the
    on-the-fly and packed matrix-core calls (as the benchmark launches them,
    without the fp32 output) within the tolerance, each flip checked against
    the oracle's y."""
    w = synth.workload(name)
    cr, sr, yr = oracle.quantize(w.X, w.A, w.B, want_y=True)
    Xd, Ad, Bd = dev_bf16(w.X), dev_f32(w.A), dev_f32(w.B)
    c, s, _ = kq.quantize_exact(Xd, Ad, Bd)
    assert_exact((host(c), host(s), None), (cr, sr, None), name)
    c, s, _ = kq.quantize(Xd, Ad, Bd)
    c, s = host(c), host(s)
    assert_mx_close((c, s, None), (cr, sr, yr), name + " mfma")
    kp = kq.pack_factors(Ad, Bd)
    c, s, _ = kq.quantize_packed(Xd, Ad, Bd, kp)
    assert_mx_close((host(c), host(s), None), (cr, sr, yr), name + " packed")


# ------------------------------------------------------------------ 64-bit indexing
def _assert_mx_close_all(c, s, cr, sr, X, A, B, what):
    """Every code and scale under the tolerance; the flips are then checked
    against the oracle's y, recomputed for the rows that hold them."""
    rep = oracle.mx_compare(c, s, cr, sr)
    assert rep["ok"], f"{what}: {rep}"
    if rep["flips"]:
        rows = np.unique(np.flatnonzero((c != cr).any(axis=1)))
        _, _, yr = oracle.quantize(np.ascontiguousarray(X[rows]), A, B, want_y=True)
        rep = oracle.mx_compare(c[rows], s[rows], cr[rows], sr[rows], y_ref=yr, max_flip_frac=1.0)
        assert rep["off_tie"] == 0 and rep["ok"], f"{what}: {rep}"


def test_index_beyond_2_31_elements():
    """X [262176, 8192] bf16 (2^31 + 2^18 elements, 4.3 GB: the last 32 rows
    lie beyond 2^31 elements and 2^32 bytes of X), FLUX recipe drawn on the
    device: every code and scale of the fixed-order, on-the-fly and packed
    paths, with one shared pair (flat mapping) and per-block pairs (tile
    kernel), against the oracle."""
    M, d = 262176, 8192
    assert M * d > 2 ** 31 and M * d * 2 > 2 ** 32
    Xd = synth.activations_device(M, d, seed=5)
    X = host(Xd.view(torch.int16)).view(np.uint16)
    for nfac in (1, d // 32):
        A, B = synth.factors(4, 8, nfac, seed=17 + nfac)
        cr, sr, _ = oracle.quantize(X, A, B)
        Ad, Bd = dev_f32(A), dev_f32(B)
        c, s, _ = kq.quantize_exact(Xd, Ad, Bd)
        c, s = host(c), host(s)
        assert np.array_equal(s, sr) and np.array_equal(c, cr), f"exact nfac={nfac}"
        c, s, _ = kq.quantize(Xd, Ad, Bd)
        _assert_mx_close_all(host(c), host(s), cr, sr, X, A, B, f"on the fly nfac={nfac}")
        kp = kq.pack_factors(Ad, Bd)
        c, s, _ = kq.quantize_packed(Xd, Ad, Bd, kp)
        _assert_mx_close_all(host(c), host(s), cr, sr, X, A, B, f"packed nfac={nfac}")
        del c, s, cr, sr
        torch.cuda.empty_cache()
