"""Boundary tests that need no GPU: the C-ABI library loads, exports every
symbol include/kroquant.h declares, rejects every invalid argument with its
exact status before any HIP call, and its host helpers match the oracle."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import oracle
import synth
from conftest import ROOT

kq = pytest.importorskip("paper_2607_21446_amd")

SUCCESS, INVALID, NULLP, MISALIGNED, UNSUPPORTED, SINGULAR, HIP = range(7)
FAKE = 1 << 20  # 16-byte aligned fake device address: validation fails before any use


def _declared():
    with open(os.path.join(ROOT, "include", "kroquant.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(kq_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    L = kq.lib()
    declared = _declared()
    assert set(declared) == set(kq.EXPORTED)
    for name in declared:
        assert hasattr(L, name), name
    assert kq.version() >= 100


def test_status_strings_are_stable():
    names = ["KQ_SUCCESS", "KQ_ERROR_INVALID_VALUE", "KQ_ERROR_NULL_POINTER", "KQ_ERROR_MISALIGNED",
             "KQ_ERROR_UNSUPPORTED", "KQ_ERROR_SINGULAR", "KQ_ERROR_HIP"]
    for i, n in enumerate(names):
        assert kq.status_string(i) == n
    assert kq.status_string(99) == "KQ_ERROR_UNKNOWN"


def _q(**kw):
    args = dict(X=FAKE, M=4, d=64, A=FAKE, B=FAKE, a=4, b=8, nfac=1, codes=FAKE, scales=FAKE, y=None)
    args.update(kw)
    L = kq.lib()
    return L.kq_quantize(args["X"], args["M"], args["d"], args["A"], args["B"], args["a"], args["b"],
                         args["nfac"], args["codes"], args["scales"], args["y"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(d=48), INVALID), (dict(d=0), INVALID), (dict(d=-32), INVALID), (dict(M=-1), INVALID),
    (dict(a=4, b=4), UNSUPPORTED), (dict(a=16, b=2), UNSUPPORTED), (dict(a=3, b=8), UNSUPPORTED),
    (dict(nfac=3), UNSUPPORTED), (dict(nfac=0), UNSUPPORTED),
    (dict(X=None), NULLP), (dict(A=None), NULLP), (dict(B=None), NULLP), (dict(codes=None), NULLP),
    (dict(scales=None), NULLP), (dict(X=FAKE + 8), MISALIGNED), (dict(codes=FAKE + 4), MISALIGNED),
    (dict(y=FAKE + 4), MISALIGNED), (dict(A=FAKE + 2), MISALIGNED),
    (dict(M=1 << 40, d=1 << 30), INVALID), (dict(d=1 << 25, nfac=1 << 20), UNSUPPORTED),
    # more workgroups than one launch holds: 2^32 units of 64 blocks, 2^31 tiles of 64 rows x 8 blocks
    (dict(M=1 << 37, d=64), UNSUPPORTED), (dict(M=1 << 36, d=512, nfac=16), UNSUPPORTED),
])
def test_quantize_rejects(kw, status):
    assert _q(**kw) == status
    assert kq.lib().kq_last_error_detail() != b""


def test_timestamp_rejects_before_enqueueing():
    """kq_timestamp checks its destination before anything is enqueued."""
    L = kq.lib()
    assert L.kq_timestamp(None, None) == NULLP
    assert L.kq_timestamp(FAKE + 4, None) == MISALIGNED
    with pytest.raises(TypeError):
        kq.timestamp(torch.zeros(2, dtype=torch.int64))  # a host tensor


def test_zero_rows_is_a_no_op():
    assert _q(M=0) == SUCCESS
    assert _q(M=0, nfac=2) == SUCCESS
    L = kq.lib()
    assert L.kq_mxfp4_quantize(FAKE, 0, 64, FAKE, FAKE, None) == SUCCESS
    assert L.kq_hadamard32_quantize(FAKE, 0, 64, FAKE, FAKE, None, None) == SUCCESS
    assert L.kq_smoothquant_quantize(FAKE, 0, 64, FAKE, FAKE, FAKE, None, None) == SUCCESS
    assert L.kq_e2m1_encode(FAKE, 0, 127, FAKE, None) == SUCCESS


def test_pack_and_packed_reject():
    L = kq.lib()
    assert L.kq_pack_factors(FAKE, FAKE, 4, 4, 1, FAKE, None) == UNSUPPORTED
    assert L.kq_pack_factors(FAKE, FAKE, 4, 8, 0, FAKE, None) == INVALID
    assert L.kq_pack_factors(FAKE, None, 4, 8, 1, FAKE, None) == NULLP
    assert L.kq_pack_factors(FAKE, FAKE, 4, 8, 1, FAKE + 4, None) == MISALIGNED
    assert L.kq_quantize_packed(FAKE, 4, 64, FAKE, FAKE, 4, 8, 1, None, FAKE, FAKE, None, None) == NULLP
    assert L.kq_quantize_packed(FAKE, 4, 64, FAKE, FAKE, 4, 8, 1, FAKE + 8, FAKE, FAKE, None, None) == MISALIGNED
    assert L.kq_quantize_packed(FAKE, 4, 48, FAKE, FAKE, 4, 8, 1, FAKE, FAKE, FAKE, None, None) == INVALID
    assert L.kq_quantize_packed(FAKE, 0, 64, FAKE, FAKE, 4, 8, 1, FAKE, FAKE, FAKE, None, None) == SUCCESS
    assert kq.PACK_BYTES_PER_FACTOR == 6 * 64 * 16 + 16


def test_quantize_lu_rejects():
    L = kq.lib()
    q = lambda **kw: L.kq_quantize_lu(kw.get("X", FAKE), kw.get("M", 4), kw.get("d", 64), kw.get("lu", FAKE),
                                      kw.get("a", 4), kw.get("nfac", 1), kw.get("codes", FAKE), kw.get("scales", FAKE),
                                      kw.get("y", None), kw.get("y16", None), None)
    assert q(a=3) == UNSUPPORTED and q(a=16) == UNSUPPORTED and q(a=0) == UNSUPPORTED
    assert q(nfac=3) == UNSUPPORTED
    assert q(d=1 << 25, nfac=1 << 20) == UNSUPPORTED
    assert q(M=1 << 37, d=64) == UNSUPPORTED and q(M=1 << 36, d=512, nfac=16) == UNSUPPORTED
    assert q(lu=None) == NULLP
    assert q(lu=FAKE + 2) == MISALIGNED
    assert q(y16=FAKE + 8) == MISALIGNED
    assert q(d=48) == INVALID
    assert q(M=0) == SUCCESS
    assert q(M=0, nfac=2) == SUCCESS


def test_fwht_rejects():
    L = kq.lib()
    for d in (96, 3072, 32768, 48):
        st = L.kq_fwht_quantize(FAKE, 4, d, FAKE, FAKE, None, None)
        assert st == (INVALID if d % 32 else UNSUPPORTED), d
    assert L.kq_fwht_quantize(FAKE, 0, 4096, FAKE, FAKE, None, None) == SUCCESS
    assert L.kq_fwht_quantize(FAKE + 8, 4, 4096, FAKE, FAKE, None, None) == MISALIGNED


def test_mxfp4_gemm_rejects():
    L = kq.lib()
    g = lambda **kw: L.kq_mxfp4_gemm(kw.get("ac", FAKE), kw.get("as_", FAKE), kw.get("M", 4), kw.get("bc", FAKE),
                                     kw.get("bs", FAKE), kw.get("N", 4), kw.get("K", 64), kw.get("C", FAKE),
                                     kw.get("ldc", 4), kw.get("acc", 0), None)
    assert g(K=48) == INVALID and g(K=0) == INVALID and g(M=-1) == INVALID
    assert g(ldc=3) == INVALID and g(acc=2) == INVALID
    assert g(M=65535 * 128 + 1) == INVALID
    assert g(ac=None) == NULLP and g(C=None) == NULLP
    assert g(ac=FAKE + 8) == MISALIGNED and g(C=FAKE + 2) == MISALIGNED
    assert g(M=0) == SUCCESS and g(N=0, ldc=0) == SUCCESS
    h = lambda **kw: L.kq_mxfp4_gemm_bf16(kw.get("ac", FAKE), kw.get("as_", FAKE), kw.get("M", 4), kw.get("bc", FAKE),
                                          kw.get("bs", FAKE), kw.get("N", 4), kw.get("K", 64), kw.get("C", FAKE),
                                          kw.get("ldc", 4), None)
    assert h(K=48) == INVALID and h(ldc=3) == INVALID and h(M=-1) == INVALID
    assert h(bs=None) == NULLP and h(C=None) == NULLP
    assert h(bc=FAKE + 4) == MISALIGNED and h(C=FAKE + 1) == MISALIGNED
    assert h(M=0) == SUCCESS and h(N=0, ldc=0) == SUCCESS


def test_comparators_reject():
    L = kq.lib()
    assert L.kq_smoothquant_quantize(FAKE, 4, 64, None, FAKE, FAKE, None, None) == NULLP
    assert L.kq_smoothquant_quantize(FAKE, 4, 64, FAKE + 4, FAKE, FAKE, None, None) == MISALIGNED
    assert L.kq_smoothquant_quantize(FAKE, 4, 40, FAKE, FAKE, FAKE, None, None) == INVALID
    assert L.kq_hadamard32_quantize(FAKE, 4, 64, None, FAKE, None, None) == NULLP
    assert L.kq_mxfp4_quantize(FAKE + 2, 4, 64, FAKE, FAKE, None) == MISALIGNED
    assert L.kq_stream_floor(FAKE + 2, 4, 64, FAKE, FAKE, None) == MISALIGNED
    assert L.kq_stream_floor(FAKE, 4, 48, FAKE, FAKE, None) == INVALID
    assert L.kq_stream_floor(FAKE, 4, 64, None, FAKE, None) == NULLP
    for w, u, g in ((3, 1, 0), (1, 3, 0), (32, 1, 0), (1, 1, -1), (1, 1, 1 << 31)):
        assert L.kq_stream_probe(FAKE, 4, 64, FAKE, FAKE, w, u, g, None) == INVALID
    assert L.kq_stream_probe(FAKE, 0, 64, FAKE, FAKE, 1, 1, 0, None) == SUCCESS
    assert L.kq_stream_floor(FAKE, 0, 64, FAKE, FAKE, None) == 0
    assert L.kq_e2m1_encode(FAKE, 3, 127, FAKE, None) == INVALID
    assert L.kq_e2m1_encode(FAKE, 4, 255, FAKE, None) == INVALID
    assert L.kq_e2m1_encode(FAKE, 4, -1, FAKE, None) == INVALID


def test_weight_transform_rejects_before_any_hip_call():
    L = kq.lib()
    A = np.eye(4, dtype=np.float32)[None].copy()
    B = np.zeros((1, 8, 8), np.float32)  # singular
    pa, pb = A.ctypes.data, B.ctypes.data
    st = L.kq_weight_transform(FAKE, 4, 64, pa, pb, 4, 8, 1, FAKE, None, None, None)
    assert st == SINGULAR
    Bn = np.eye(8, dtype=np.float32)[None].copy()
    st = L.kq_weight_transform(FAKE, 4, 64, pa, Bn.ctypes.data, 4, 8, 1, None, None, None, None)
    assert st == NULLP
    st = L.kq_weight_transform(FAKE, 4, 64, pa, Bn.ctypes.data, 4, 8, 1, FAKE, FAKE, None, None)
    assert st == NULLP  # codes without scales
    st = L.kq_weight_transform(FAKE, 0, 64, pa, Bn.ctypes.data, 4, 8, 1, FAKE, None, None, None)
    assert st == SUCCESS
    Bill = np.diag([1.0] * 7 + [1e-7]).astype(np.float32)[None].copy()  # cond 1e7
    st = L.kq_weight_transform(FAKE, 4, 64, pa, Bill.ctypes.data, 4, 8, 1, FAKE, None, None, None)
    assert st == SINGULAR


@pytest.mark.parametrize("ab", [(4, 8), (2, 16), (8, 4), (1, 32)])
def test_inverse_transpose_matches_oracle(ab):
    a, b = ab
    A, B = synth.factors(a, b, 7, seed=31)
    Ait, Bit = kq.factors_inverse_transpose(torch.from_numpy(A), torch.from_numpy(B))
    Ro, Bo = oracle.factors_inverse_transpose(A, B)
    # both round an fp64 inverse to fp32: at most one fp32 ulp apart
    assert np.allclose(Ait.numpy(), Ro, rtol=2.0**-23, atol=1e-30)
    assert np.allclose(Bit.numpy(), Bo, rtol=2.0**-23, atol=1e-30)


@pytest.mark.parametrize("a", [1, 2, 4, 8])
def test_lu_to_factors_matches_oracle(a):
    rng = np.random.default_rng(5)
    abc = rng.normal(size=(6, 5, 3)).astype(np.float32)
    abc[..., 0] = np.where(np.abs(abc[..., 0]) < 0.3, 0.7, abc[..., 0])
    A, B = kq.lu_to_factors(torch.from_numpy(abc), a)
    Ao, Bo = oracle.lu_to_factors(abc.astype(np.float64), a)
    assert A.shape == Ao.shape and B.shape == Bo.shape
    assert np.allclose(A.numpy(), Ao, rtol=2.0**-22, atol=1e-30)
    assert np.allclose(B.numpy(), Bo, rtol=2.0**-22, atol=1e-30)
    # the Hadamard initialization LU(1/sqrt2, 1/sqrt2, 1) gives H32^T / sqrt(32) = H32 / sqrt(32)
    h = 1 / np.sqrt(2.0)
    Ah, Bh = kq.lu_to_factors(torch.tensor([[h, h, 1.0]] * 5, dtype=torch.float32)[None], a)
    from scipy.linalg import hadamard
    K = np.kron(Ah[0].numpy().astype(np.float64), Bh[0].numpy().astype(np.float64))
    assert np.allclose(K, hadamard(32) / np.sqrt(32.0), atol=1e-6)


def test_lu_rejects():
    L = kq.lib()
    abc = np.zeros((1, 5, 3), np.float32)
    A = np.zeros((1, 4, 4), np.float32)
    B = np.zeros((1, 8, 8), np.float32)
    assert L.kq_lu_to_factors(abc.ctypes.data, 4, 1, A.ctypes.data, B.ctypes.data) == SINGULAR
    assert L.kq_lu_to_factors(abc.ctypes.data, 3, 1, A.ctypes.data, B.ctypes.data) == UNSUPPORTED
    assert L.kq_lu_to_factors(None, 4, 1, A.ctypes.data, B.ctypes.data) == NULLP


def test_product_path_has_no_oracle_dependency():
    """The binding and the HIP sources never reference the oracle."""
    pkg = os.path.join(ROOT, "paper_2607_21446_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".h", ".cpp")):
                with open(os.path.join(dirpath, fn)) as f:
                    text = f.read()
                assert "oracle" not in text.lower(), fn
                assert "kqo_" not in text, fn


def test_calibration_rejects():
    import ctypes
    L = kq.lib()
    n = ctypes.c_size_t(0)
    ws = lambda R=64, o=32, d=64, a=4, nfac=1: L.kq_calib_workspace_size(R, o, d, a, nfac, ctypes.byref(n))
    assert ws() == SUCCESS and n.value > 0
    assert ws(R=0) == INVALID and ws(o=0) == INVALID and ws(d=48) == INVALID
    assert ws(o=65535 * 64 + 1) == INVALID and ws(d=65535 * 64 + 32, nfac=1) == INVALID
    assert ws(a=3) == UNSUPPORTED and ws(nfac=3) == UNSUPPORTED and ws(nfac=2) == SUCCESS
    assert L.kq_calib_workspace_size(64, 32, 64, 4, 1, None) == NULLP
    assert L.kq_calib_reference(FAKE, 4, 64, FAKE, 4, None, None) == NULLP
    assert L.kq_calib_reference(FAKE + 8, 4, 64, FAKE, 4, FAKE, None) == MISALIGNED
    assert ws() == SUCCESS
    need = n.value  # the size for exactly the shape the calls below pass
    step = lambda **kw: L.kq_calib_step(
        kw.get("X", FAKE), 64, 64, FAKE, 32, kw.get("Y", FAKE), FAKE, 4, 1, FAKE, FAKE, FAKE,
        kw.get("m", None), None, kw.get("t", 0), 0.01, kw.get("ws", FAKE), kw.get("wsb", need), None)
    assert step(Y=None) == NULLP and step(X=FAKE + 2) == MISALIGNED
    assert step(t=-1) == INVALID and step(t=1) == NULLP
    assert step(wsb=need - 1) == INVALID and step(ws=FAKE + 16) == MISALIGNED and step(ws=None) == NULLP
    cal = lambda **kw: L.kq_calibrate(FAKE, 64, 64, FAKE, 32, FAKE, FAKE, 4, 1, kw.get("steps", 10), 0.01,
                                      kw.get("losses", FAKE), FAKE, kw.get("wsb", need), None)
    assert cal(steps=-1) == INVALID and cal(losses=None) == NULLP and cal(losses=FAKE + 4) == MISALIGNED
    assert cal(wsb=0) == INVALID


def test_bench_refuses_more_than_one_gpu():
    """bench.py exits with a message before touching a GPU when asked for more than one."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], cwd=ROOT,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr


# ---------------------------------------------------------------- binding argument checks
def test_binding_rejects_wrong_buffer_sizes():
    """The binding checks every caller-supplied buffer against the sizes the
    call will touch before anything reaches the library (an undersized buffer
    would otherwise be written out of bounds)."""
    from paper_2607_21446_amd import binding as bd
    X = torch.zeros((4, 64), dtype=torch.bfloat16)
    c, s, y = bd._outputs(X, None, None, None, True)
    assert c.shape == (4, 32) and s.shape == (4, 2) and y.shape == (4, 64)
    with pytest.raises(ValueError):
        bd._outputs(X, torch.empty(4 * 32 - 1, dtype=torch.uint8), None, None, False)
    with pytest.raises(ValueError):
        bd._outputs(X, None, torch.empty(7, dtype=torch.uint8), None, False)
    with pytest.raises(ValueError):
        bd._outputs(X, None, None, torch.empty((4, 63), dtype=torch.float32), False)
    with pytest.raises(ValueError):
        bd._outputs(torch.zeros(64, dtype=torch.bfloat16), None, None, None, False)
    A, B = torch.zeros((3, 4, 4)), torch.zeros((3, 8, 8))
    assert bd._pairs(A, B) == (4, 8, 3)
    with pytest.raises(ValueError):
        bd._pairs(A, torch.zeros((2, 8, 8)))          # pair counts differ
    with pytest.raises(ValueError):
        bd._pairs(torch.zeros((3, 4, 2)), B)          # A not square
    with pytest.raises(ValueError):
        bd._pairs(A, B, torch.device("cuda", 0))      # factors not on the input's device
    with pytest.raises(ValueError):
        bd._size(torch.zeros(10), 11, "kpack")


def test_binding_rejects_before_the_library_is_called():
    """Public calls with an inconsistent buffer raise ValueError/TypeError
    (on this host the tensors are not device tensors, which is rejected too)."""
    with pytest.raises((TypeError, ValueError)):
        kq.quantize(torch.zeros((4, 64), dtype=torch.bfloat16), torch.zeros((1, 4, 4)), torch.zeros((1, 8, 8)))
    with pytest.raises(ValueError):
        kq.lu_to_factors(torch.zeros(14), 4)


def test_calib_step_noalloc_refuses_before_any_hip_call():
    """Sizes whose workspace exceeds the library's per-GPU scratch are refused
    before any HIP call (so this runs without a GPU)."""
    L = kq.lib()
    st = L.kq_calib_step_noalloc(FAKE, 4096, 1152, FAKE, 1152, FAKE, FAKE, 4, 36, FAKE, FAKE, FAKE, None, None, 0,
                                 0.0, None)
    assert st == INVALID and b"scratch" in L.kq_last_error_detail()
    assert L.kq_calib_step_noalloc(FAKE, 0, 64, FAKE, 8, FAKE, FAKE, 4, 1, FAKE, FAKE, FAKE, None, None, 0, 0.0,
                                   None) == INVALID
    assert kq.CALIB_NOALLOC_MAX_BYTES == 64 << 20
