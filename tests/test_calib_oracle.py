"""Pins of the calibration oracle (Sec. 3.3) to things other than itself.

* The straight-through gradient against central finite differences of a
  separately written numpy form of the objective in which the quantizer's
  decisions (codes, scales, clip mask) are frozen at the evaluation point:
  that function is smooth, equals L there, and its exact gradient is the
  straight-through gradient by definition.  It builds every factor as the
  matrix product L_k U_k, the block by numpy.kron and the weight side with a
  LAPACK inverse, so a wrong Kronecker order, transpose, inverse, sign or
  normalisation in the oracle fails it.
* The loss values at exactly representable (dyadic) parameters against the
  layer error E(T) of Sec. 3.1 computed by the oracle's independent
  quantize / weight_transform path (eq. (1)) and the dense fp64 transform.
* The Hadamard initialisation against the Sylvester H_32 / sqrt(32).
* Adam against torch.optim.Adam.
CPU only.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import calib


def _g(a, b, c):
    return np.array([[1.0, 0.0], [c, 1.0]]) @ np.array([[a, b], [0.0, -1.0 / a]])


def _blocks_T(lu64):
    Ts = []
    for blk in lu64:
        T = np.ones((1, 1))
        for k in range(5):
            T = np.kron(T, _g(*blk[k]))
        Ts.append(T)
    return np.array(Ts)


def _apply_np(M, Ts):
    R, d = M.shape
    out = np.empty_like(M)
    for j in range(d // 32):
        T = Ts[0] if len(Ts) == 1 else Ts[j]
        out[:, 32 * j:32 * j + 32] = M[:, 32 * j:32 * j + 32] @ T
    return out


class _Frozen:
    """Objective with the quantizer's decisions frozen at lu0 (numpy, fp64)."""

    def __init__(self, X, W, lu0, a, lam_A, lam_W):
        self.x = oracle.bf16_to_f32(X).astype(np.float64)
        self.w = oracle.bf16_to_f32(W).astype(np.float64)
        self.ref = self.x @ self.w.T
        self.lam_A, self.lam_W = lam_A, lam_W
        lu0 = np.asarray(lu0, np.float32).astype(np.float64)
        Ts = _blocks_T(lu0)
        Us = np.array([np.linalg.inv(T).T for T in Ts])
        self.At0 = _apply_np(self.x, Ts)
        self.Wt0 = _apply_np(self.w, Us)
        ca, sa, _, _ = oracle.quantize_lu(X, np.asarray(lu0, np.float32), a)
        Ai, Bi = oracle.lu_inverse_factors_f32(np.asarray(lu0, np.float32), a)
        cw, sw, _ = oracle.quantize(W, Ai, Bi)
        self.Qa0 = oracle.dequantize(ca, sa)
        self.Qw0 = oracle.dequantize(cw, sw)
        lim_a = 6.0 * np.exp2(np.repeat(sa.astype(np.float64), 32, axis=-1) - 127.0)
        lim_w = 6.0 * np.exp2(np.repeat(sw.astype(np.float64), 32, axis=-1) - 127.0)
        self.ma = (np.abs(self.At0) <= lim_a).astype(np.float64)
        self.mw = (np.abs(self.Wt0) <= lim_w).astype(np.float64)

    def __call__(self, lu64):
        Ts = _blocks_T(lu64)
        Us = np.array([np.linalg.inv(T).T for T in Ts])
        At = _apply_np(self.x, Ts)
        Wt = _apply_np(self.w, Us)
        Qa = self.Qa0 + self.ma * (At - self.At0)
        Qw = self.Qw0 + self.mw * (Wt - self.Wt0)
        R, d = self.x.shape
        o = self.w.shape[0]
        L_out = np.sum((Qa @ Qw.T - self.ref) ** 2) / (R * o)
        L_A = np.sum((Qa - At) ** 2) / (R * d)
        L_W = np.sum((Qw - Wt) ** 2) / (o * d)
        return L_out + self.lam_A * L_A + self.lam_W * L_W


@pytest.mark.parametrize("a,nfac,start", [(4, 1, "hadamard"), (4, 2, "random"), (2, 2, "random"),
                                          (8, 1, "random")])
def test_straight_through_gradient_against_finite_differences(a, nfac, start):
    X, W = synth.calib_layer(40, 24, 64, seed=3)
    lu0 = calib.hadamard_lu(nfac) if start == "hadamard" else synth.lu_params(nfac, seed=5)
    if start == "hadamard":
        lu0 = lu0 + np.float32(0.05) * synth.lu_params(nfac, seed=9)  # off the symmetric point
    lam_A, lam_W = 0.7, 1.3
    r = calib.objective(X, W, lu0, a, lam_A, lam_W)
    f = _Frozen(X, W, lu0, a, lam_A, lam_W)
    base = np.asarray(lu0, np.float32).astype(np.float64)
    assert f(base) == pytest.approx(r["L"], rel=1e-9)
    # the clip mask must matter somewhere for this to pin the straight-through rule
    assert f.ma.min() == 0.0 and f.mw.min() == 0.0
    h = 1e-5
    fd = np.zeros_like(base)
    for idx in np.ndindex(base.shape):
        e = np.zeros_like(base)
        e[idx] = h
        fd[idx] = (f(base + e) - f(base - e)) / (2 * h)
    scale = np.abs(fd).max()
    assert scale > 0
    np.testing.assert_allclose(r["grad"], fd, rtol=0, atol=1e-6 * scale)


def _dyadic_lu(nfac, seed):
    rng = np.random.default_rng(seed)
    lu = np.empty((nfac, 5, 3), np.float32)
    lu[..., 0] = rng.choice([1.0, 2.0, 0.5, -1.0], size=(nfac, 5))
    lu[..., 1] = rng.choice([0.5, 0.25, -0.5, 0.0], size=(nfac, 5))
    lu[..., 2] = rng.choice([0.25, -0.25, 0.5, 0.0], size=(nfac, 5))
    return lu


@pytest.mark.parametrize("a,nfac", [(4, 1), (2, 3)])
def test_losses_against_layer_error(a, nfac):
    """At dyadic parameters every factor entry is exact in fp32 on both
    routes, so L_out R o equals E(T)^2 of the eq. (1) path exactly (up to the
    fp64 sum), and L_A, L_W equal the quantization errors of the dense fp64
    transform and of the weight transform."""
    d = 32 * nfac if nfac > 1 else 64
    X, W = synth.calib_layer(48, 20, d, seed=11)
    lu = _dyadic_lu(nfac, seed=2)
    r = calib.objective(X, W, lu, a, 0.0, 0.0)
    A, B = oracle.lu_to_factors(lu, a)
    A2, B2 = oracle.lu_factors_f32(lu, a)
    assert np.array_equal(A, A2) and np.array_equal(B, B2)
    E, (xc, xs), (wc, ws), _ = oracle.layer_error(X, W, A, B)
    R, o = X.shape[0], W.shape[0]
    assert r["L_out"] * R * o == pytest.approx(E * E, rel=1e-10)
    y = oracle.transform_f64(X, A, B)
    assert r["L_A"] == pytest.approx(np.sum((oracle.dequantize(xc, xs) - y) ** 2) / (R * d), rel=1e-10)
    Wt, _, _ = oracle.weight_transform(W, A, B)
    assert r["L_W"] == pytest.approx(np.sum((oracle.dequantize(wc, ws) - Wt) ** 2) / (o * d), rel=1e-5)
    assert r["L"] == pytest.approx(r["L_out"])


def test_hadamard_initialisation_is_sylvester():
    from scipy.linalg import hadamard
    T = calib.block_transforms(torch.from_numpy(calib.hadamard_lu(2).astype(np.float64)))
    H = hadamard(32) / np.sqrt(32.0)
    for f in range(2):
        np.testing.assert_allclose(T[f].numpy(), H, atol=1e-7)


def test_adam_matches_torch():
    rng = np.random.default_rng(0)
    theta = rng.normal(size=(2, 5, 3))
    p = torch.tensor(theta.copy(), requires_grad=True)
    opt = torch.optim.Adam([p], lr=1e-2)
    m = np.zeros_like(theta)
    v = np.zeros_like(theta)
    for t in range(1, 8):
        g = rng.normal(size=theta.shape) * 10.0 ** rng.integers(-6, 2)
        p.grad = torch.from_numpy(g.copy())
        opt.step()
        theta, m, v = calib.adam_step(theta, g, m, v, t, 1e-2)
        np.testing.assert_allclose(theta, p.detach().numpy(), rtol=1e-12, atol=1e-14)


def test_auto_lambdas_balance_the_terms_at_the_start():
    X, W = synth.calib_layer(32, 16, 64, seed=4)
    lu0 = calib.hadamard_lu(1)
    r0 = calib.objective(X, W, lu0, 4, 0.0, 0.0)
    lam_A, lam_W = calib.auto_lambdas(r0["L_out"], r0["L_A"], r0["L_W"])
    r = calib.objective(X, W, lu0, 4, lam_A, lam_W)
    assert lam_A * r["L_A"] == pytest.approx(r["L_out"], rel=1e-12)
    assert lam_W * r["L_W"] == pytest.approx(r["L_out"], rel=1e-12)
    assert r["L"] == pytest.approx(3 * r["L_out"], rel=1e-12)


def test_calibration_lowers_the_objective():
    X, W = synth.calib_layer(64, 32, 64, seed=6)
    lu, rows = calib.calibrate(X, W, calib.hadamard_lu(2), 4, steps=25, lr=1e-2)
    assert rows.shape == (27, 4)
    assert rows[1, 3] == pytest.approx(3 * rows[0, 0], rel=1e-12)
    assert rows[-1, 3] < rows[1, 3]
