"""Layer-wise calibration oracle (Sec. 3.3) -- TEST INFRASTRUCTURE ONLY.

Plain fp64 PyTorch-CPU form of the per-layer transform optimisation: the
objective

    L_out = || Q(A T) Q(W T^-T)^T - A W^T ||_F^2 / (N m o)
    L_A   = || Q(A T) - A T ||_F^2 / (N m d)
    L_W   = || Q(W T^-T) - W T^-T ||_F^2 / (o d)
    L     = L_out + lambda_A L_A + lambda_W L_W

(the N calibration samples of m tokens stacked into R = N m rows), the
automatic weights lambda_A = L_out(T_0) / L_A(T_0), lambda_W = L_out(T_0) /
L_W(T_0) at the Hadamard initialisation T_0 of Sec. 3.2, the gradient with
respect to the 15 LU parameters (a_k, b_k, c_k) of every block by autograd,
and Adam (Kingma and Ba, Algorithm 1) on it.

Readings where the paper leaves the detail open:
  * Q is the MXFP4 quantizer of Sec. 3.1 evaluated as the product path does:
    Q(A T) = ``quantize_lu`` (factors decoded from the parameters in fp32,
    every output exactly rounded), Q(W T^-T) = ``quantize`` with the
    closed-form inverse factors of ``lu_inverse_factors_f32``.  The autograd
    graph carries T = G_1 (x) ... (x) G_5 in fp64 from the same (fp32)
    parameter values.
  * Straight-through estimator: the E2M1 rounding passes the gradient
    unchanged, the E8M0 scale (a step function of the block maximum) is held
    fixed, and an element clipped at |v| > 6 * scale passes none.  Written
    Q_ste(v) = Q(v) + mask * (v - stop_gradient(v)).  With an identity STE
    everywhere L_A and L_W would have zero gradient, which contradicts their
    stated role of steering both operands.
  * Adam with beta1 = 0.9, beta2 = 0.999, eps = 1e-8 (the method's defaults);
    the paper fixes the learning rate 1e-2 and 100 steps.
It shares no code with the HIP library and never imports it.
"""
from __future__ import annotations

import numpy as np
import torch

from . import bf16_to_f32, dequantize, lu_inverse_factors_f32, quantize, quantize_lu

ADAM_BETA1 = 0.9
ADAM_BETA2 = 0.999
ADAM_EPS = 1e-8


def hadamard_lu(nfac):
    """Hadamard initialisation (Sec. 3.2): every G_k = [[cos, sin], [sin, -cos]]
    at pi/4, which in G = L U with L = [[1, 0], [c, 1]], U = [[a, b], [0, -1/a]]
    is a = b = 1/sqrt(2), c = 1.  Returns fp32 [nfac, 5, 3]."""
    r = np.float32(1.0 / np.sqrt(2.0))
    lu = np.empty((nfac, 5, 3), dtype=np.float32)
    lu[..., 0] = r
    lu[..., 1] = r
    lu[..., 2] = 1.0
    return lu


def factors_of(lu64):
    """G_k = L_k U_k for every block and k (Sec. 3.2): [nfac, 5, 2, 2] fp64."""
    a, b, c = lu64[..., 0], lu64[..., 1], lu64[..., 2]
    row0 = torch.stack([a, b], dim=-1)
    row1 = torch.stack([c * a, c * b - 1.0 / a], dim=-1)
    return torch.stack([row0, row1], dim=-2)


def block_transforms(lu64):
    """T_f = G_1 (x) G_2 (x) ... (x) G_5 per block, [nfac, 32, 32]."""
    G = factors_of(lu64)
    T = G[:, 0]
    for k in range(1, 5):
        n = T.shape[-1]
        T = torch.einsum("fij,fkl->fikjl", T, G[:, k]).reshape(-1, 2 * n, 2 * n)
    return T


def _apply(M, T):
    """Row map of every 32-column block: out[:, 32j + q] = sum_p M[:, 32j + p] T_f(j)[p, q]
    (one T for every block if T has one entry)."""
    R, d = M.shape
    nb = d // 32
    blocks = M.reshape(R, nb, 32)
    if T.shape[0] == 1:
        out = blocks @ T[0]
    else:
        out = torch.einsum("rjp,jpq->rjq", blocks, T)
    return out.reshape(R, d)


def _as_f64(M):
    M = np.asarray(M)
    return bf16_to_f32(M).astype(np.float64) if M.dtype == np.uint16 else M.astype(np.float64)


def objective(X, W, lu, a, lam_A, lam_W):
    """L_out, L_A, L_W, L at the parameters ``lu`` and dL/dlu (straight-through).

    X [R, d], W [o, d]: bf16 bit patterns (uint16).  lu [nfac, 5, 3] (taken as
    fp32).  Returns a dict with the four losses (floats) and ``grad`` (fp64
    [nfac, 5, 3])."""
    lu32 = np.ascontiguousarray(lu, dtype=np.float32).reshape(-1, 5, 3)
    x = torch.from_numpy(_as_f64(X))
    w = torch.from_numpy(_as_f64(W))
    R, d = x.shape
    o = w.shape[0]

    p = torch.tensor(lu32.astype(np.float64), requires_grad=True)
    T = block_transforms(p)
    U = torch.linalg.inv(T).transpose(-1, -2)          # T^-T
    At = _apply(x, T)                                   # A T
    Wt = _apply(w, U)                                   # W T^-T

    ca, sa, _, _ = quantize_lu(X, lu32, a)
    Ai, Bi = lu_inverse_factors_f32(lu32, a)
    cw, sw, _ = quantize(W, Ai, Bi)
    Qa = torch.from_numpy(dequantize(ca, sa))
    Qw = torch.from_numpy(dequantize(cw, sw))
    lim_a = torch.from_numpy(6.0 * np.exp2(np.repeat(sa.astype(np.float64), 32, axis=-1) - 127.0))
    lim_w = torch.from_numpy(6.0 * np.exp2(np.repeat(sw.astype(np.float64), 32, axis=-1) - 127.0))
    mask_a = (At.detach().abs() <= lim_a).to(torch.float64)
    mask_w = (Wt.detach().abs() <= lim_w).to(torch.float64)
    Qa_ste = Qa + mask_a * (At - At.detach())
    Qw_ste = Qw + mask_w * (Wt - Wt.detach())

    L_out = ((Qa_ste @ Qw_ste.T - x @ w.T) ** 2).sum() / (R * o)
    L_A = ((Qa_ste - At) ** 2).sum() / (R * d)
    L_W = ((Qw_ste - Wt) ** 2).sum() / (o * d)
    L = L_out + lam_A * L_A + lam_W * L_W
    L.backward()
    return {"L_out": L_out.item(), "L_A": L_A.item(), "L_W": L_W.item(), "L": L.item(),
            "grad": p.grad.numpy().copy()}


def auto_lambdas(L_out0, L_A0, L_W0):
    """lambda_A = L_out(T_0) / L_A(T_0), lambda_W = L_out(T_0) / L_W(T_0) (0 for a zero denominator)."""
    return (L_out0 / L_A0 if L_A0 > 0 else 0.0), (L_out0 / L_W0 if L_W0 > 0 else 0.0)


def adam_step(theta, g, m, v, t, lr, beta1=ADAM_BETA1, beta2=ADAM_BETA2, eps=ADAM_EPS):
    """One Adam update (Kingma and Ba, Algorithm 1), fp64; returns (theta, m, v)."""
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** t)
    vhat = v / (1.0 - beta2 ** t)
    return theta - lr * mhat / (np.sqrt(vhat) + eps), m, v


def calibrate(X, W, lu0, a, steps=100, lr=1e-2):
    """The per-layer optimisation: lambdas from the losses at lu0, then
    ``steps`` Adam steps on L.  Parameters are kept in fp32 between steps (the
    quantizer decodes fp32 parameters); the moments in fp64.  Returns (lu,
    losses [(steps + 2), 4]) with the rows laid out as kq_calibrate does: row 0
    at lu0 with lambda = 0, row t before update t, the last row at the final lu."""
    lu = np.ascontiguousarray(lu0, dtype=np.float32).reshape(-1, 5, 3).copy()
    r0 = objective(X, W, lu, a, 0.0, 0.0)
    lam_A, lam_W = auto_lambdas(r0["L_out"], r0["L_A"], r0["L_W"])
    rows = [[r0["L_out"], r0["L_A"], r0["L_W"], r0["L"]]]
    m = np.zeros(lu.shape)
    v = np.zeros(lu.shape)
    for t in range(1, steps + 1):
        r = objective(X, W, lu, a, lam_A, lam_W)
        rows.append([r["L_out"], r["L_A"], r["L_W"], r["L"]])
        theta, m, v = adam_step(lu.astype(np.float64), r["grad"], m, v, t, lr)
        lu = theta.astype(np.float32)
    r = objective(X, W, lu, a, lam_A, lam_W)
    rows.append([r["L_out"], r["L_A"], r["L_W"], r["L"]])
    return lu, np.array(rows)
