"""GPU parity of the layer-wise calibration (Sec. 3.3) through the C ABI
against the calibration oracle (oracle/calib.py) on the same seeded layers.

Bar: the quantized operands come from the library's quantizers, which match
the oracle's codes and scales bit for bit (within tie flips), so the losses
agree to the fp32 accumulation error of the residual (L_out, L: 1e-4
relative; L_A, L_W: 1e-5) and the straight-through gradient to 1e-4 of its
largest entry (fp32 sums over o and over the rows on the matrix cores, then
the chain rule in fp32; measured errors are below 1e-6).  Adam is checked against the textbook update on the
library's own gradient.
"""
import numpy as np
import pytest

import oracle
import synth
from oracle import calib

torch = pytest.importorskip("torch")
kq = pytest.importorskip("paper_2607_21446_amd")

pytestmark = pytest.mark.gpu


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


LAM = (float(np.float32(0.7)), float(np.float32(1.3)))

# R, o, d, a, per-block factors, start
CASES = [
    (40, 24, 64, 4, True, "hadamard"),
    (200, 96, 128, 4, False, "random"),
    (300, 160, 320, 2, True, "random"),
    (129, 130, 256, 8, True, "random"),
    (1, 1, 32, 4, False, "random"),
    (520, 72, 96, 1, True, "hadamard"),
]


def _start(nfac, start, seed):
    if start == "hadamard":
        return calib.hadamard_lu(nfac) + np.float32(0.05) * synth.lu_params(nfac, seed=seed)
    return synth.lu_params(nfac, seed=seed)


@pytest.mark.parametrize("R,o,d", [(40, 24, 64), (300, 130, 320), (129, 1, 32), (1, 257, 96)])
def test_calib_reference_parity(R, o, d):
    X, W = synth.calib_layer(R, o, d, seed=R + o)
    Y = host(kq.calib_reference(dev_bf16(X), dev_bf16(W)))
    x = oracle.bf16_to_f32(X).astype(np.float64)
    w = oracle.bf16_to_f32(W).astype(np.float64)
    ref = -(x @ w.T)
    tol = d * 2.0 ** -24 * (np.abs(x) @ np.abs(w).T)
    assert Y.shape == (R, o)
    assert np.all(np.abs(Y - ref) <= tol), np.max(np.abs(Y - ref) - tol)


@pytest.mark.parametrize("R,o,d,a,per_block,start", CASES)
def test_calib_step_parity(R, o, d, a, per_block, start):
    nfac = d // 32 if per_block else 1
    X, W = synth.calib_layer(R, o, d, seed=R + 3 * o + d)
    lu = _start(nfac, start, seed=R + o)
    print(f"calib step R={R} o={o} d={d} a={a} nfac={nfac} start={start}", flush=True)
    Xd, Wd = dev_bf16(X), dev_bf16(W)
    Yneg = kq.calib_reference(Xd, Wd)
    losses, grad = kq.calib_step(Xd, Wd, Yneg, dev_f32(lu), dev_f32(np.array(LAM)), a=a)
    L = host(losses)
    G = host(grad)
    r = calib.objective(X, W, lu, a, *LAM)
    assert L[0] == pytest.approx(r["L_out"], rel=1e-4)
    assert L[1] == pytest.approx(r["L_A"], rel=1e-5)
    assert L[2] == pytest.approx(r["L_W"], rel=1e-5)
    assert L[3] == pytest.approx(r["L"], rel=1e-4)
    scale = np.abs(r["grad"]).max()
    err = np.abs(G - r["grad"]).max()
    print(f"  grad max |err| / max |g| = {err / scale:.3e}", flush=True)
    assert err <= 1e-4 * scale


def test_calib_step_adam_update():
    R, o, d, a = 96, 64, 128, 4
    nfac = d // 32
    X, W = synth.calib_layer(R, o, d, seed=21)
    lu = synth.lu_params(nfac, seed=4)
    Xd, Wd = dev_bf16(X), dev_bf16(W)
    Yneg = kq.calib_reference(Xd, Wd)
    lud = dev_f32(lu)
    m = torch.zeros(nfac * 15, dtype=torch.float32, device="cuda")
    v = torch.zeros_like(m)
    lam = dev_f32(np.array(LAM))
    ws = kq.calib_workspace(R, o, d, a, nfac)
    theta = lu.astype(np.float64)
    mo = np.zeros(theta.shape)
    vo = np.zeros(theta.shape)
    for t in range(1, 4):
        before = host(lud).astype(np.float64)
        _, grad = kq.calib_step(Xd, Wd, Yneg, lud, lam, a=a, workspace=ws, adam=(m, v, t, 1e-2))
        g = host(grad).astype(np.float64)
        want, mo, vo = calib.adam_step(before, g, mo, vo, t, 1e-2)
        got = host(lud)
        np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-7)


def test_calibrate_loop():
    R, o, d, a, steps = 128, 48, 64, 4, 12
    nfac = d // 32
    X, W = synth.calib_layer(R, o, d, seed=5)
    lu0 = calib.hadamard_lu(nfac)
    Xd, Wd = dev_bf16(X), dev_bf16(W)
    lud, losses = kq.calibrate(Xd, Wd, lu=dev_f32(lu0), a=a, steps=steps, lr=1e-2)
    rows = host(losses)
    lu_gpu = host(lud)
    lu_or, rows_or = calib.calibrate(X, W, lu0, a, steps=steps, lr=1e-2)
    assert rows.shape == rows_or.shape == (steps + 2, 4)
    # the first two rows are at the same parameters on both sides
    np.testing.assert_allclose(rows[:2], rows_or[:2], rtol=1e-4)
    assert rows[1, 3] == pytest.approx(3 * rows[0, 0], rel=1e-5)
    assert rows[-1, 3] < rows[1, 3]
    # the final row is the objective at the final parameters
    lam_A, lam_W = calib.auto_lambdas(*rows[0, :3])
    r = calib.objective(X, W, lu_gpu, a, float(np.float32(lam_A)), float(np.float32(lam_W)))
    assert rows[-1, 0] == pytest.approx(r["L_out"], rel=1e-4)
    assert rows[-1, 3] == pytest.approx(r["L"], rel=1e-4)
    print("gpu rows", rows[:, 3], "\noracle rows", rows_or[:, 3], "\nmax |dlu|", np.abs(lu_gpu - lu_or).max())


def test_calibration_graph_replays_match_eager():
    """kq_calib_step (no update) and a whole 3-step kq_calibrate captured into
    HIP graphs and replayed three times, with other work and synchronizations
    between the replays and the parameters reset before each: every replay
    reproduces the eager losses, gradient, parameters and loss rows bit for bit
    (the calls allocate, clear and synchronize nothing; all sums run in a fixed
    order)."""
    R, o, d, a = 300, 160, 256, 4
    nfac = d // 32
    X, W = synth.calib_layer(R, o, d, seed=31)
    lu0 = synth.lu_params(nfac, seed=32)
    Xd, Wd = dev_bf16(X), dev_bf16(W)
    Yneg = kq.calib_reference(Xd, Wd)
    ws = kq.calib_workspace(R, o, d, a, nfac)
    lam = dev_f32(np.array(LAM))
    lud = dev_f32(lu0)
    grad = torch.empty((nfac, 5, 3), dtype=torch.float32, device="cuda")
    losses = torch.empty(4, dtype=torch.float64, device="cuda")
    kq.calib_step(Xd, Wd, Yneg, lud, lam, a=a, workspace=ws, grad=grad, losses=losses)
    e_loss, e_grad = host(losses).copy(), host(grad).copy()
    lu_c = dev_f32(lu0)
    _, e_rows = kq.calibrate(Xd, Wd, lu=lu_c, a=a, steps=3, Yneg=Yneg, workspace=ws)
    e_rows, e_lu = host(e_rows).copy(), host(lu_c).copy()

    g1 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g1):
        kq.calib_step(Xd, Wd, Yneg, lud, lam, a=a, workspace=ws, grad=grad, losses=losses)
    lu_g = dev_f32(lu0)
    rows_g = torch.empty((5, 4), dtype=torch.float64, device="cuda")
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2):
        _, r = kq.calibrate(Xd, Wd, lu=lu_g, a=a, steps=3, Yneg=Yneg, workspace=ws)
        rows_g.copy_(r)
    other = dev_bf16(synth.activations(256, 1024, "normal", seed=33))
    lu0_d = dev_f32(lu0)
    for rep in range(3):
        grad.fill_(7.0)
        losses.fill_(7.0)
        rows_g.fill_(7.0)
        lu_g.copy_(lu0_d)
        kq.mxfp4(other)
        torch.cuda.synchronize()
        g1.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host(losses), e_loss) and np.array_equal(host(grad), e_grad), rep
        g2.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host(rows_g), e_rows) and np.array_equal(host(lu_g), e_lu), rep
