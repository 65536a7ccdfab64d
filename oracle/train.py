"""CPU oracle for one stage codec's training step (Section III-C: encoder E_phi,
sphere map, sign binarisation with the straight-through estimator, decoder
D_theta; eq. codec_loss and eq. codec_loss_terms), and Adam.

TEST INFRASTRUCTURE ONLY, like the rest of this package. Values are fp64
(numpy); the two decisions a forward pass takes -- the code bits of z = E x
and the ReLU mask of the decoder's hidden layer -- come from the C oracle in
fp32 (orc_train_decisions), the precision the training kernels take them in,
so that both sides agree on every decision.

Parameters of one stage codec, packed in one vector theta (the layout the
training kernels use):
    E [b][d] | W1 [h][b] | b1 [h] | W2 [d][h] | b2 [d]
with the linear encoder z = E x and the symmetric decoder
x_hat = W2 relu(W1 q + b1) + b2.

Forward for a mini-batch of N chunks x_i (the rows of X):
    z_i = E x_i;  u_i = z_i / ||z_i||;  q_i = sign(u_i) / sqrt(b)
    x_hat_i = D(q_ste_i), q_ste = u + (q - u).detach()   (value q, gradient to u)
    L_rec = 1/N sum_i ||x_hat_i - x_i||^2
    L_com = 1/N sum_i ||u_i - sg(q_i)||^2
    p_ij  = [sigma(-t_ij), sigma(t_ij)], t_ij = 2 tau u_ij / sqrt(b)
    pbar_j = 1/N sum_i p_ij
    L_ent = 1/N sum_i sum_j H(p_ij) - gamma sum_j H(pbar_j)
    L = L_rec + lambda_c L_com + lambda_e L_ent
with H the entropy of a two-point distribution (natural log). A chunk with
z = 0 has u = 0 and passes no gradient to E.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from . import code_scale, train_decisions


@dataclass(frozen=True)
class Hyper:
    """Training hyperparameters. The paper names lambda_c, lambda_e, gamma and
    tau without values; these are readings (see the design notes)."""
    lambda_c: float = 0.25
    lambda_e: float = 0.1
    gamma: float = 1.0
    tau: float = 1.0
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8


def param_count(d: int, b: int, h: int) -> int:
    return b * d + h * b + h + d * h + d


def pack(E, W1, b1, W2, b2) -> np.ndarray:
    return np.concatenate([np.ravel(v).astype(np.float64) for v in (E, W1, b1, W2, b2)])


def unpack(theta, d: int, b: int, h: int):
    th = np.asarray(theta, dtype=np.float64)
    o = 0
    out = []
    for shape in ((b, d), (h, b), (h,), (d, h), (d,)):
        n = int(np.prod(shape))
        out.append(th[o:o + n].reshape(shape))
        o += n
    return out


def _entropy2(s):
    """Entropy of the two-point distribution [1 - s, s], natural log."""
    return -(s * np.log(s) + (1.0 - s) * np.log1p(-s))


def loss_and_grad(theta, X, d: int, b: int, h: int, hp: Hyper):
    """(L, L_rec, L_com, L_ent) and dL/dtheta for the chunks X [N, d] (fp32
    values), the straight-through gradient for the encoder."""
    E, W1, b1, W2, b2 = unpack(theta, d, b, h)
    Xf = np.ascontiguousarray(X, dtype=np.float32)
    N = Xf.shape[0]
    codes, masks = train_decisions(b, h, E.astype(np.float32), W1.astype(np.float32), b1.astype(np.float32), Xf)
    X64 = Xf.astype(np.float64)
    mask = masks.astype(np.float64)

    # sphere map and sign binarisation
    z = X64 @ E.T
    nz = np.sqrt(np.sum(z * z, axis=1))
    live = nz > 0
    u = np.zeros_like(z)
    u[live] = z[live] / nz[live, None]
    bits = (codes[:, None].astype(np.int64) >> np.arange(b)[None, :]) & 1
    c = float(code_scale(b))
    q = np.where(bits == 1, c, -c)

    # decoder on the code (the forward value of q_ste)
    pre = q @ W1.T + b1[None, :]
    a = pre * mask
    xh = a @ W2.T + b2[None, :]
    diff = xh - X64

    # the three terms of eq. codec_loss_terms
    L_rec = float(np.sum(diff * diff)) / N
    L_com = float(np.sum((u - q) ** 2)) / N
    t = 2.0 * hp.tau * u / math.sqrt(b)
    s = 1.0 / (1.0 + np.exp(-t))
    sbar = np.mean(s, axis=0)
    L_ent = float(np.sum(_entropy2(s))) / N - hp.gamma * float(np.sum(_entropy2(sbar)))
    L = L_rec + hp.lambda_c * L_com + hp.lambda_e * L_ent

    # backward: decoder
    dxh = 2.0 * diff / N
    dW2 = dxh.T @ a
    db2 = dxh.sum(axis=0)
    dpre = (dxh @ W2) * mask
    dW1 = dpre.T @ q
    db1 = dpre.sum(axis=0)
    # straight-through: the gradient reaching q is passed to u
    du = dpre @ W1
    du += hp.lambda_c * 2.0 * (u - q) / N
    # dH(p)/dt = -t s (1 - s) per chunk; the batch term through pbar_j
    ds_dt = s * (1.0 - s)
    dt = (-t * ds_dt) / N - hp.gamma * np.log((1.0 - sbar) / sbar)[None, :] * ds_dt / N
    du += hp.lambda_e * dt * (2.0 * hp.tau / math.sqrt(b))
    # u = z / ||z||
    dz = np.zeros_like(z)
    dz[live] = (du[live] - u[live] * np.sum(u[live] * du[live], axis=1)[:, None]) / nz[live, None]
    dE = dz.T @ X64
    return (L, L_rec, L_com, L_ent), pack(dE, dW1, db1, dW2, db2)


def adam(theta, grad, m, v, step: int, hp: Hyper):
    """One Adam step (Kingma & Ba 2015) with bias correction; step counts
    from 1. Returns the new (theta, m, v)."""
    g = np.asarray(grad, dtype=np.float64)
    m = hp.beta1 * np.asarray(m, dtype=np.float64) + (1.0 - hp.beta1) * g
    v = hp.beta2 * np.asarray(v, dtype=np.float64) + (1.0 - hp.beta2) * g * g
    mh = m / (1.0 - hp.beta1 ** step)
    vh = v / (1.0 - hp.beta2 ** step)
    return np.asarray(theta, dtype=np.float64) - hp.lr * mh / (np.sqrt(vh) + hp.eps), m, v
