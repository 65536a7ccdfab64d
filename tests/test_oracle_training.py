"""Pins of the codec-training oracle (Section III-C: encoder, sphere map,
sign binarisation with the straight-through estimator, symmetric decoder;
eq. codec_loss and eq. codec_loss_terms; Adam).

Each gradient is checked against central finite differences of a loss
evaluated here from its definition, independently of the oracle's backward
pass: the decoder parameters against the loss itself (smooth in them while no
hidden pre-activation crosses zero), the encoder against the
straight-through surrogate in which the decoder reads u + (q0 - u0) (the
estimator's forward value with the offset held fixed). Closed forms pin the
loss terms (zero temperature, codes on the sphere's vertices) and the first
Adam step; a short run pins that training lowers the loss.
"""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
import oracle.train as T
import synth


def _setup(d, b, h, seed, n=256, scale=0.5):
    dec = synth.decoder_params(synth.DEC_MLP, d, b, h, 1, seed=seed, encoder=True)[0]
    theta = T.pack(dec.E, dec.W1, dec.b1, dec.W2, dec.b2)
    X = np.random.default_rng(seed).normal(0, scale, (n, d)).astype(np.float32)
    return theta, X


def _loss_fixed(theta, X, d, b, h, hp, q0, u0, masks, encoder_surrogate):
    """The loss from its definition, fp64, with the decisions held fixed: the
    decoder reads q0 (or, for the encoder surrogate, u + (q0 - u0)); the ReLU
    mask is `masks`."""
    E, W1, b1, W2, b2 = T.unpack(theta, d, b, h)
    X64 = X.astype(np.float64)
    N = len(X)
    z = X64 @ E.T
    u = z / np.linalg.norm(z, axis=1, keepdims=True)
    qin = (u + (q0 - u0)) if encoder_surrogate else q0
    a = (qin @ W1.T + b1) * masks
    xh = a @ W2.T + b2
    L_rec = np.sum((xh - X64) ** 2) / N
    L_com = np.sum((u - q0) ** 2) / N
    t = 2 * hp.tau * u / math.sqrt(b)
    s = 1 / (1 + np.exp(-t))
    H = -(s * np.log(s) + (1 - s) * np.log(1 - s))
    sb = s.mean(axis=0)
    Hb = -(sb * np.log(sb) + (1 - sb) * np.log(1 - sb))
    return L_rec + hp.lambda_c * L_com + hp.lambda_e * (H.sum() / N - hp.gamma * Hb.sum())


def _decisions(theta, X, d, b, h):
    E, W1, b1, _, _ = T.unpack(theta, d, b, h)
    codes, masks = oracle.train_decisions(b, h, E, W1, b1, X)
    bits = (codes[:, None].astype(np.int64) >> np.arange(b)) & 1
    c = oracle.code_scale(b)
    q0 = np.where(bits == 1, c, -c)
    z = X.astype(np.float64) @ E.T
    u0 = z / np.linalg.norm(z, axis=1, keepdims=True)
    return q0, u0, masks.astype(np.float64)


@pytest.mark.parametrize("d,b,h", [(8, 8, 8), (8, 16, 12), (16, 8, 5)])
def test_gradient_against_finite_differences(d, b, h):
    hp = T.Hyper(lambda_c=0.3, lambda_e=0.2, gamma=0.7, tau=1.5)
    theta, X = _setup(d, b, h, seed=10 + d + b + h)
    (L, *_), g = T.loss_and_grad(theta, X, d, b, h, hp)
    q0, u0, masks = _decisions(theta, X, d, b, h)
    assert abs(_loss_fixed(theta, X, d, b, h, hp, q0, u0, masks, False) - L) <= 1e-12 * max(1.0, abs(L))
    n_enc = b * d
    r = np.random.default_rng(3)
    for idx in list(r.choice(n_enc, 12, replace=False)) + list(n_enc + r.choice(len(theta) - n_enc, 24, replace=False)):
        eps = 1e-6 * max(1.0, abs(theta[idx]))
        tp, tm = theta.copy(), theta.copy()
        tp[idx] += eps
        tm[idx] -= eps
        sur = idx < n_enc
        if not sur:   # the decisions must not move for a decoder parameter's finite difference
            assert np.array_equal(_decisions(tp, X, d, b, h)[2], masks)
            assert np.array_equal(_decisions(tm, X, d, b, h)[2], masks)
        fd = (_loss_fixed(tp, X, d, b, h, hp, q0, u0, masks, sur) -
              _loss_fixed(tm, X, d, b, h, hp, q0, u0, masks, sur)) / (2 * eps)
        assert abs(fd - g[idx]) <= 1e-6 * max(1.0, abs(fd)), (idx, fd, g[idx])


def test_zero_temperature_and_vertex_codes_closed_forms():
    """tau = 0: every bit probability is 1/2, so L_ent = b ln 2 (1 - gamma)
    and the entropy passes no gradient. Chunks with E = I whose entries are
    +-a (the scaled vertices of the cube): u = q exactly, so L_com = 0 and
    the commitment passes no gradient; then the encoder gradient is the
    decoder's straight-through gradient projected off u, divided by ||z||."""
    d = b = h = 8
    hp = T.Hyper(lambda_c=1.0, lambda_e=1.0, gamma=0.4, tau=0.0)
    theta, X = _setup(d, b, h, seed=20)
    (L, L_rec, L_com, L_ent), g = T.loss_and_grad(theta, X, d, b, h, hp)
    assert abs(L_ent - b * math.log(2) * (1 - hp.gamma)) <= 1e-12
    hp0 = T.Hyper(lambda_c=1.0, lambda_e=0.0, gamma=0.4, tau=0.0)
    (_, _, _, _), g0 = T.loss_and_grad(theta, X, d, b, h, hp0)
    np.testing.assert_allclose(g, g0, rtol=0, atol=1e-15)
    E, W1, b1, W2, b2 = T.unpack(theta, d, b, h)
    sgn = np.where(np.random.default_rng(21).random((64, d)) < 0.5, -1.0, 1.0)
    Xv = (0.25 * sgn).astype(np.float32)
    th = T.pack(np.eye(d), W1, b1, W2, b2)
    (_, _, L_com, _), gv = T.loss_and_grad(th, Xv, d, b, h, T.Hyper(lambda_c=1.0, lambda_e=0.0))
    c32 = oracle.code_scale(b)          # the stored code entry, fp32(1 / sqrt(b))
    assert L_com <= b * (c32 - 1 / math.sqrt(b)) ** 2 * (1 + 1e-9)
    u = sgn / math.sqrt(b)
    q = sgn * c32
    _, masks = oracle.train_decisions(b, h, np.eye(d), W1, b1, Xv)
    dxh = 2 * (((q @ W1.T + b1) * masks) @ W2.T + b2 - Xv.astype(np.float64)) / len(Xv)
    du = ((dxh @ W2) * masks) @ W1 + 2 * (u - q) / len(Xv)
    dz = (du - u * np.sum(u * du, axis=1, keepdims=True)) / (0.25 * math.sqrt(d))
    np.testing.assert_allclose(gv[:b * d].reshape(b, d), dz.T @ Xv.astype(np.float64), rtol=1e-12, atol=1e-15)


def test_first_adam_step_is_the_sign_step():
    """With zero moments, the bias-corrected first step is
    theta - lr g / (|g| + eps) (Kingma & Ba 2015, Algorithm 1)."""
    hp = T.Hyper(lr=0.01)
    g = np.array([3.0, -2e-3, 0.0, 1e-12, -5.0])
    th = np.array([1.0, 2.0, 3.0, 4.0, 5.0])
    new, m, v = T.adam(th, g, np.zeros(5), np.zeros(5), 1, hp)
    np.testing.assert_allclose(new, th - hp.lr * g / (np.abs(g) + hp.eps), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(m, (1 - hp.beta1) * g)
    np.testing.assert_allclose(v, (1 - hp.beta2) * g * g)


def test_training_lowers_the_loss_on_weight_chunks():
    """Category-batched training (Section III-G: the chunks of several layers
    of one category as one batch) lowers L over 200 Adam steps."""
    d = b = h = 8
    hp = T.Hyper(lr=3e-3)
    dec = synth.decoder_params(synth.DEC_MLP, d, b, h, 1, seed=30, encoder=True)[0]
    theta = T.pack(dec.E, dec.W1, dec.b1, dec.W2, dec.b2)
    layers = [np.random.default_rng(31 + li).normal(0, 0.02, (64, 128)).astype(np.float32) for li in range(4)]
    X = np.concatenate([w.reshape(-1, d) for w in layers])      # the category's chunks, stacked
    m = np.zeros_like(theta)
    v = np.zeros_like(theta)
    L0 = T.loss_and_grad(theta, X, d, b, h, hp)[0][0]
    for step in range(1, 201):
        (L, *_), g = T.loss_and_grad(theta, X, d, b, h, hp)
        theta, m, v = T.adam(theta, g, m, v, step, hp)
    L1 = T.loss_and_grad(theta, X, d, b, h, hp)[0][0]
    assert L1 < 0.5 * L0
