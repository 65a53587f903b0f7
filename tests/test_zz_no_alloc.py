"""kq_calib_step_noalloc (the calibration step on the library's own per-GPU
scratch, no allocation) against kq_calib_step with a caller workspace.

Two calls in a row, the second on smaller sizes, each compared with the
workspace entry point on the same inputs: losses, gradient and the Adam
update of the parameters and moments must be bit-identical (both run the
same kernels in the same order; the workspace of the reference call is
filled with 0xFF bytes first, so neither result can lean on what a buffer
held before).  The smaller second call runs on scratch that still holds the
larger first call's data."""
import ctypes

import numpy as np
import pytest

import synth

torch = pytest.importorskip("torch")
kq = pytest.importorskip("paper_2607_21446_amd")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    kq.lib()
    yield


def _dev_bf16(X):
    return torch.from_numpy(np.ascontiguousarray(X).view(np.int16)).view(torch.bfloat16).cuda()


def _step_both(R, o, d, a, per_block, seed, t):
    X, W = synth.calib_layer(R, o, d, seed=seed)
    Xd, Wd = _dev_bf16(X), _dev_bf16(W)
    nfac = d // 32 if per_block else 1
    lu0 = torch.from_numpy(synth.lu_params(nfac, seed=seed + 1)).cuda()
    lam = torch.tensor([0.7, 1.3], dtype=torch.float32, device="cuda")
    Yneg = kq.calib_reference(Xd, Wd)
    rng = np.random.default_rng(seed + 2)
    m0 = torch.from_numpy(rng.normal(size=(nfac * 15,)).astype(np.float32) * 1e-3).cuda()
    v0 = torch.from_numpy(np.abs(rng.normal(size=(nfac * 15,))).astype(np.float32) * 1e-6).cuda()
    n = ctypes.c_size_t(0)
    assert kq.lib().kq_calib_workspace_size(R, o, d, a, nfac, ctypes.byref(n)) == 0
    assert n.value <= kq.CALIB_NOALLOC_MAX_BYTES
    ws = torch.full((n.value,), 0xFF, dtype=torch.uint8, device="cuda")
    out = []
    for noalloc in (False, True):
        lu, m, v = lu0.clone(), m0.clone(), v0.clone()
        grad = torch.full((nfac, 5, 3), float("nan"), dtype=torch.float32, device="cuda")
        losses = torch.full((4,), float("nan"), dtype=torch.float64, device="cuda")
        if noalloc:
            kq.calib_step_noalloc(Xd, Wd, Yneg, lu, lam, a=a, adam=(m, v, t, 1e-2), grad=grad, losses=losses)
        else:
            kq.calib_step(Xd, Wd, Yneg, lu, lam, a=a, workspace=ws, adam=(m, v, t, 1e-2), grad=grad, losses=losses)
        torch.cuda.synchronize()
        out.append([x.cpu().numpy() for x in (losses, grad, lu, m, v)])
    return out


@pytest.mark.parametrize("first,second", [((1024, 1152, 1152, 4, True, 11, 1), (300, 96, 640, 2, True, 12, 3)),
                                          ((512, 256, 512, 8, False, 13, 2), (40, 24, 64, 4, True, 14, 1))])
def test_noalloc_step_matches_workspace_step(first, second):
    for case in (first, second):
        ref, got = _step_both(*case)
        for name, u, w in zip(("losses", "grad", "lu", "adam m", "adam v"), ref, got):
            assert np.all(np.isfinite(u)), (case, name)
            assert np.array_equal(u.view(np.uint8), w.view(np.uint8)), (case, name)


def test_noalloc_step_refuses_sizes_beyond_its_scratch():
    X, W = synth.calib_layer(8, 8, 64, seed=1)
    Xd, Wd = _dev_bf16(X), _dev_bf16(W)
    lu = torch.ones((1, 5, 3), dtype=torch.float32, device="cuda")
    lam = torch.zeros(2, dtype=torch.float32, device="cuda")
    # R = 4096, o = d = 1152 needs about 117 MiB: refused (the pointers are never used)
    L = kq.lib()
    st = L.kq_calib_step_noalloc(Xd.data_ptr(), 4096, 1152, Wd.data_ptr(), 1152, lu.data_ptr(), lu.data_ptr(), 4,
                                 36, lam.data_ptr(), lu.data_ptr(), lam.data_ptr(), None, None, 0, 0.0, None)
    assert st == 1 and b"scratch" in L.kq_last_error_detail()
