"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a library
routine (numpy's binary16 rounding, numpy's least-squares solver), a brute-force
enumeration, a closed form, an invariant, or a special case that reduces to a
known map. Together they are meant to catch a dropped term, a flipped sign, a
wrong index or a transposed operand anywhere in the encoder, decoder assembly,
protected-channel path or product routes.
"""
import itertools
import math
import os

import numpy as np
import pytest

import oracle
import synth
from oracle import KIND_IDENTITY, KIND_LINEAR, KIND_MLP, Config

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _unpack(code, d):
    return np.array([(int(code) >> j) & 1 for j in range(d)], dtype=np.int64)


def _f16(bits):
    return oracle.f16_bits_to_f32(np.asarray(bits, dtype=np.uint16))


# ---------------------------------------------------------------- binary16
def test_f16_rounding_matches_numpy():
    """The oracle's RNE fp32->fp16 agrees with numpy's conversion bit for bit,
    including subnormals, exact ties, the overflow boundary and signed zero."""
    L = oracle.lib()
    r = _rng(0)
    vals = np.concatenate([
        r.normal(0, 1, 20000), r.normal(0, 1e-5, 20000), r.normal(0, 3e4, 5000),
        np.ldexp(r.integers(1, 2 ** 13, 5000).astype(np.float64) + 0.5, -24),  # subnormal ties
        np.ldexp(r.integers(1024, 2048, 5000).astype(np.float64) + 0.5, -10),  # normal ties
        [0.0, -0.0, 65504.0, 65519.99, 65520.0, -65520.0, 6.0e-8, 5.96e-8, 2.98e-8, 1e-40],
    ]).astype(np.float32)
    ref = vals.astype(np.float16).view(np.uint16)
    got = np.array([L.orc_f32_to_f16(float(v)) for v in vals], dtype=np.uint16)
    np.testing.assert_array_equal(got, ref)
    back = np.array([L.orc_f16_to_f32(int(b)) for b in ref[:3000]], dtype=np.float32)
    np.testing.assert_array_equal(back, ref[:3000].view(np.float16).astype(np.float32))


def test_gain_saturates_to_max_finite():
    L = oracle.lib()
    assert L.orc_gain_to_f16(1e6) == 0x7BFF
    assert L.orc_gain_to_f16(-1e6) == 0xFBFF
    assert L.orc_gain_to_f16(65520.0) == 0x7BFF
    assert L.orc_gain_to_f16(1.0) == 0x3C00


# ---------------------------------------------------------------- codes
@pytest.mark.parametrize("b", list(range(1, 17)))
def test_codes_have_unit_norm(b):
    """Every spherical code q = sign(u)/sqrt(b) has ||q||_2 = 1 (Sec. III-C):
    exactly for b in {1, 4, 16}, within one fp32 rounding otherwise."""
    cfg = Config(d=b, b=b, stages=1, kind=KIND_IDENTITY, protect_num=0)
    tab = oracle.decoder_table(cfg, [synth.StageDecoder()])[0].astype(np.float64)
    norms = np.sqrt((tab * tab).sum(axis=1))
    if b in (1, 4, 16):
        assert np.all(norms == 1.0)
    assert np.max(np.abs(norms - 1.0)) <= 2 ** -23
    # every entry is +-1/sqrt(b) rounded once to fp32
    np.testing.assert_array_equal(np.unique(np.abs(tab)), [np.float32(1 / math.sqrt(b))])


@pytest.mark.parametrize("d", list(range(1, 13)))
def test_sign_is_nearest_vertex_bruteforce(d):
    """q = sign(u)/sqrt(b) is the nearest vertex of {+-1/sqrt(b)}^b to u, checked
    against all 2^b vertices; exact zeros (ties) take the + vertex."""
    r = _rng(100 + d)
    n = 64
    w = r.normal(0, 1, (n, d)).astype(np.float32)
    w[r.random((n, d)) < 0.15] = 0.0            # exact ties
    w[0, :] = 0.0                               # the all-zero chunk
    w[1, :] = -0.0
    cfg = Config(d=d, b=d, stages=1, kind=KIND_IDENTITY, protect_num=0)
    enc = oracle.encode(cfg, [synth.StageDecoder()], w)
    verts = np.array(list(itertools.product([-1.0, 1.0], repeat=d))) / math.sqrt(d)
    for i in range(n):
        bits = _unpack(enc.codes[0][i, 0], d)
        q = (2.0 * bits - 1.0) / math.sqrt(d)
        z = w[i].astype(np.float64)
        nz = np.linalg.norm(z)
        u = z / nz if nz > 0 else z
        dist = ((verts - u) ** 2).sum(axis=1)
        assert ((q - u) ** 2).sum() <= dist.min() + 1e-12
        np.testing.assert_array_equal(bits[z == 0], 1)
    assert enc.codes[0][0, 0] == (1 << d) - 1 and enc.codes[0][1, 0] == (1 << d) - 1
    assert enc.gains[0][0, 0] == 0 and enc.gains[0][1, 0] == 0


@pytest.mark.parametrize("d", [8, 16])
def test_pack_patterns_and_round_trip(d):
    """LSB-first packing: all-positive -> all ones; only element j negative ->
    bit j clear; unpacking recovers the sign pattern of every chunk."""
    rows = [np.ones(d, np.float32)]
    for j in range(d):
        v = np.ones(d, np.float32)
        v[j] = -1.0
        rows.append(v)
    r = _rng(7)
    rows += list(r.normal(0, 1, (40, d)).astype(np.float32))
    w = np.stack(rows)
    cfg = Config(d=d, b=d, stages=1, kind=KIND_IDENTITY, protect_num=0)
    enc = oracle.encode(cfg, [synth.StageDecoder()], w)
    full = (1 << d) - 1
    assert enc.codes[0][0, 0] == full
    for j in range(d):
        assert enc.codes[0][1 + j, 0] == full & ~(1 << j)
    for i in range(len(rows)):
        np.testing.assert_array_equal(_unpack(enc.codes[0][i, 0], d), (w[i] >= 0).astype(np.int64))
    assert enc.codes[0].dtype == (np.uint8 if d == 8 else np.uint16)


# ---------------------------------------------------------------- stages
def _stage_terms(cfg, tabs, enc, i, c):
    """Per-stage fp64 reconstructions alpha_s * D_s(code_s) of chunk (i, c)."""
    out = []
    for s in range(cfg.stages):
        code = int(enc.codes[s][i, c])
        a = float(_f16(enc.gains[s][i, c]))
        out.append(a * tabs[s][code].astype(np.float64))
    return out


@pytest.mark.parametrize("kind", [KIND_IDENTITY, KIND_LINEAR, KIND_MLP])
@pytest.mark.parametrize("d", [4, 8, 12, 16])
def test_residual_stage_never_increases_error(kind, d):
    """err_2 <= err_1 <= ||x||^2 for every chunk (Sec. III-D), evaluated in fp64
    from the stored gains and decoded vectors, for any decoder."""
    stages = 3 if d == 4 else 2
    cfg = Config(d=d, b=d, stages=stages, kind=kind, hidden=d, protect_num=0)
    decs = synth.decoder_params(kind, d, d, d, stages, seed=11 + d)
    r = _rng(20 + d + kind)
    w = r.normal(0, 0.02, (64, 4 * d)).astype(np.float32)
    tabs = oracle.decoder_table(cfg, decs)
    enc = oracle.encode(cfg, decs, w, tables=tabs)
    for i in range(w.shape[0]):
        for c in range(4):
            x = w[i, c * d:(c + 1) * d].astype(np.float64)
            errs = [float(x @ x)]
            acc = np.zeros(d)
            for t in _stage_terms(cfg, tabs, enc, i, c):
                acc = acc + t
                errs.append(float(((x - acc) ** 2).sum()))
            for a, b in zip(errs, errs[1:]):
                assert b <= a * (1 + 1e-5) + 1e-30


@pytest.mark.parametrize("d", [8, 16])
def test_identity_decoder_closed_form(d):
    """One identity stage reconstructs x by (||x||_1 / d) sign(x), the
    least-squares binary approximation with one scale per block; the fp64
    error then equals ||x||^2 - ||x||_1^2 / d up to the fp16 gain rounding."""
    cfg = Config(d=d, b=d, stages=1, kind=KIND_IDENTITY, protect_num=0)
    r = _rng(31 + d)
    w = r.normal(0, 0.05, (200, 2 * d)).astype(np.float32)
    enc = oracle.encode(cfg, [synth.StageDecoder()], w)
    w_hat = oracle.decode(cfg, [synth.StageDecoder()], enc)
    for i in range(w.shape[0]):
        for c in range(2):
            x = w[i, c * d:(c + 1) * d].astype(np.float64)
            closed = (np.abs(x).sum() / d) * np.where(x >= 0, 1.0, -1.0)
            got = w_hat[i, c * d:(c + 1) * d].astype(np.float64)
            np.testing.assert_allclose(got, closed, rtol=2 ** -10, atol=0)
            err_closed = x @ x - np.abs(x).sum() ** 2 / d
            err_got = ((x - got) ** 2).sum()
            assert err_got >= err_closed * (1 - 1e-9) - 1e-18       # LS optimum is a floor
            assert err_got <= err_closed + (x @ x) * 2 ** -18 + 1e-18


@pytest.mark.parametrize("kind", [KIND_LINEAR, KIND_MLP])
def test_gain_is_least_squares_solution(kind):
    """The stored gain equals numpy's least-squares solution of
    min_a ||r - a y||^2 over the unprotected positions, up to fp16 rounding."""
    d = 8
    cfg = Config(d=d, b=d, stages=2, kind=kind, hidden=8, protect_num=0)
    decs = synth.decoder_params(kind, d, d, 8, 2, seed=5)
    tabs = oracle.decoder_table(cfg, decs)
    r = _rng(40 + kind)
    w = r.normal(0, 0.02, (100, d)).astype(np.float32)
    enc = oracle.encode(cfg, decs, w)
    for i in range(w.shape[0]):
        target = w[i].astype(np.float64)
        for s in range(2):
            y = tabs[s][int(enc.codes[s][i, 0])].astype(np.float64)
            a_ls = np.linalg.lstsq(y[:, None], target, rcond=None)[0][0]
            a = float(_f16(enc.gains[s][i, 0]))
            assert abs(a - a_ls) <= abs(a_ls) * 2 ** -10 + 1e-7 * abs(a_ls) + 1e-30
            target = target - a * y


def test_mlp_special_cases_reduce_to_known_maps():
    """MLP decoder y = W2 relu(W1 q + b1) + b2:
    (a) W1 = P, b1 = 4, W2 = P^T, b2 = -P^T b1 gives y = q (a transposed W1 or
        W2 would not); (b) W1 = I, b1 = 0, W2 = I, b2 = 0 gives y = relu(q);
    (c) W2 = 0 gives y = b2."""
    d = 8
    cfg = Config(d=d, b=d, stages=1, kind=KIND_MLP, hidden=d, protect_num=0)
    ident = oracle.decoder_table(Config(d=d, b=d, stages=1, kind=KIND_IDENTITY), [synth.StageDecoder()])[0]
    perm = np.array([3, 0, 7, 1, 6, 2, 5, 4])
    P = np.eye(d, dtype=np.float32)[perm]           # (P q)_k = q_perm[k]
    b1 = np.full(d, 4.0, np.float32)
    dec = synth.StageDecoder(W1=P, b1=b1, W2=P.T.copy(), b2=-(P.T @ b1).astype(np.float32))
    tab = oracle.decoder_table(cfg, [dec])[0]
    np.testing.assert_allclose(tab, ident, atol=1e-6, rtol=0)
    bad = synth.StageDecoder(W1=P.T.copy(), b1=b1, W2=P.T.copy(), b2=dec.b2)
    assert np.abs(oracle.decoder_table(cfg, [bad])[0] - ident).max() > 0.5
    I = np.eye(d, dtype=np.float32)
    z = np.zeros(d, np.float32)
    tab = oracle.decoder_table(cfg, [synth.StageDecoder(W1=I, b1=z, W2=I, b2=z)])[0]
    np.testing.assert_array_equal(tab, np.maximum(ident, 0.0))
    b2 = np.arange(d, dtype=np.float32) - 3.5
    tab = oracle.decoder_table(cfg, [synth.StageDecoder(W1=P, b1=b1, W2=np.zeros((d, d), np.float32), b2=b2)])[0]
    np.testing.assert_array_equal(tab, np.broadcast_to(b2, tab.shape))


def test_linear_special_cases():
    d = 8
    cfg = Config(d=d, b=d, stages=1, kind=KIND_LINEAR, protect_num=0)
    ident = oracle.decoder_table(Config(d=d, b=d, stages=1, kind=KIND_IDENTITY), [synth.StageDecoder()])[0]
    perm = np.array([3, 0, 7, 1, 6, 2, 5, 4])
    P = np.eye(d, dtype=np.float32)[perm]
    beta = np.zeros(d, np.float32)
    tab = oracle.decoder_table(cfg, [synth.StageDecoder(W1=P, b1=beta)])[0]
    np.testing.assert_array_equal(tab, ident[:, perm])


def _all_codes_q(b):
    """q for every b-bit code, [2^b, b]: q_j = +-1/sqrt(b) by bit j (LSB first),
    built here from the definition of the sphere map (Section III-C)."""
    codes = np.arange(1 << b, dtype=np.int64)
    bits = (codes[:, None] >> np.arange(b)[None, :]) & 1
    return np.where(bits == 1, 1.0, -1.0) / math.sqrt(b)


def _fma_chain_bound(n_terms, *mags):
    """Bound on |fp32 fmaf chain - exact| for a sum of n_terms products
    started from a bias: each step rounds once (relative 2^-24), so the
    error is at most (n + 1) 2^-24 times the sum of the magnitudes."""
    return (n_terms + 1) * 2.0 ** -24 * sum(mags)


@pytest.mark.parametrize("d,b", [(8, 8), (16, 16), (8, 12), (12, 8)])
def test_linear_decoder_with_bias_against_numpy(d, b):
    """Linear decoder y = beta + M q (M is d x b, beta nonzero), every code,
    against an fp64 numpy evaluation written from the definition: a dropped or
    mis-indexed beta, a transposed M or a row stride of d instead of b fails."""
    cfg = Config(d=d, b=b, stages=1, kind=KIND_LINEAR, protect_num=0)
    r = _rng(300 + d + b)
    M = r.uniform(-0.5, 0.5, (d, b)).astype(np.float32)
    beta = r.uniform(-1.0, 1.0, d).astype(np.float32)
    tab = oracle.decoder_table(cfg, [synth.StageDecoder(W1=M, b1=beta)])[0]
    q = _all_codes_q(b)
    qf = q.astype(np.float32).astype(np.float64)   # the oracle's fp32 code values
    want = beta.astype(np.float64)[None, :] + qf @ M.astype(np.float64).T
    bound = _fma_chain_bound(b, np.abs(beta)[None, :], np.abs(qf) @ np.abs(M.astype(np.float64)).T)
    assert np.all(np.abs(tab - want) <= bound)
    # the bias alone (M = 0) comes back exactly, for every code
    tab0 = oracle.decoder_table(cfg, [synth.StageDecoder(W1=np.zeros((d, b), np.float32), b1=beta)])[0]
    np.testing.assert_array_equal(tab0, np.broadcast_to(beta, tab0.shape))


def test_linear_permutation_plus_bias_is_one_rounding():
    """M a permutation and beta nonzero: each output is beta_m + q_perm(m)
    rounded once to fp32 (the chain adds exact zeros and one product), so the
    table equals numpy's fp32 sum bit for bit."""
    d = 8
    cfg = Config(d=d, b=d, stages=1, kind=KIND_LINEAR, protect_num=0)
    perm = np.array([3, 0, 7, 1, 6, 2, 5, 4])
    P = np.eye(d, dtype=np.float32)[perm]
    beta = (np.arange(d, dtype=np.float32) - 3.25) * np.float32(0.37)
    tab = oracle.decoder_table(cfg, [synth.StageDecoder(W1=P, b1=beta)])[0]
    c = np.float32(oracle.lib().orc_code_scale(d))
    q32 = np.where(_all_codes_q(d) > 0, c, -c).astype(np.float32)
    want = beta[None, :] + q32[:, perm]
    np.testing.assert_array_equal(tab.view(np.uint32), want.astype(np.float32).view(np.uint32))


@pytest.mark.parametrize("d,b,h", [(8, 8, 5), (8, 8, 16), (16, 16, 5), (8, 12, 16), (12, 8, 3)])
def test_mlp_decoder_hidden_width_against_numpy(d, b, h):
    """Symmetric decoder at hidden widths other than d: every code against an
    fp64 numpy evaluation of W2 relu(W1 q + b1) + b2. The bound propagates the
    fp32 rounding of each hidden unit through relu (1-Lipschitz) and W2, so a
    W2 stride of d instead of h, a hidden loop bound of d, or a W1 stride of d
    instead of b fails."""
    cfg = Config(d=d, b=b, stages=1, kind=KIND_MLP, hidden=h, protect_num=0)
    decs = synth.decoder_params(KIND_MLP, d, b, h, 1, seed=400 + h)
    dec = decs[0]
    tab = oracle.decoder_table(cfg, decs)[0]
    q = _all_codes_q(b).astype(np.float32).astype(np.float64)
    W1, b1, W2, b2 = (v.astype(np.float64) for v in (dec.W1, dec.b1, dec.W2, dec.b2))
    pre = q @ W1.T + b1[None, :]
    a = np.maximum(pre, 0.0)
    want = a @ W2.T + b2[None, :]
    ea = _fma_chain_bound(b, np.abs(b1)[None, :], np.abs(q) @ np.abs(W1).T)
    bound = ea @ np.abs(W2).T + _fma_chain_bound(h, np.abs(b2)[None, :], (np.abs(a) + ea) @ np.abs(W2).T)
    assert np.all(np.abs(tab - want) <= bound)
    assert np.abs(want).max() > 10 * bound.max()   # the bound is far below the values it guards


def test_mlp_decoder_selector_closed_form():
    """h = 16 > d = 8 with one-hot W1 and W2: hidden unit k is b1_k + q_(k mod b)
    (one fp32 rounding), and output m reads only hidden unit 15 - m, all of
    them past index d. So y_m = relu(fp32(b1_(15-m) + q_((15-m) mod 8))) bit
    for bit; a loop over d hidden units or a W2 stride of d gives b2 = 0 or
    the wrong unit."""
    d, b, h = 8, 8, 16
    cfg = Config(d=d, b=b, stages=1, kind=KIND_MLP, hidden=h, protect_num=0)
    W1 = np.zeros((h, b), np.float32)
    W1[np.arange(h), np.arange(h) % b] = 1.0
    b1 = np.array([0.5, -0.5, 0.25, -1.0, 0.125, -0.25, 0.75, -0.125,
                   0.3, -0.3, 0.1, -0.6, 0.45, -0.05, 0.2, -0.4], np.float32)
    sel = h - 1 - np.arange(d)
    W2 = np.zeros((d, h), np.float32)
    W2[np.arange(d), sel] = 1.0
    b2 = np.zeros(d, np.float32)
    tab = oracle.decoder_table(cfg, [synth.StageDecoder(W1=W1, b1=b1, W2=W2, b2=b2)])[0]
    c = np.float32(oracle.lib().orc_code_scale(b))
    q32 = np.where(_all_codes_q(b) > 0, c, -c).astype(np.float32)
    pre = b1[sel][None, :] + q32[:, sel % b]                 # fp32 sums, one rounding each
    want = np.where(pre > 0, pre, np.float32(0.0)).astype(np.float32)
    np.testing.assert_array_equal(tab.view(np.uint32), want.view(np.uint32))
    assert (want > 0).mean() > 0.3 and (want == 0).mean() > 0.3


def test_mlp_relu_gives_positive_zero():
    """relu(a) is +0 for a <= 0, including a = -0: with W1 = 0 and b1 = -0 the
    pre-activation of code 0 is -0 (every product is -0), with b1 = -1 it is
    negative; W2 = 1 and b2 = -0 then give y = +0 only if relu returned +0
    (-0 + -0 would stay -0). The sign bit is checked on every code."""
    d = 8
    cfg = Config(d=d, b=d, stages=1, kind=KIND_MLP, hidden=d, protect_num=0)
    for b1v in (-0.0, -1.0):
        dec = synth.StageDecoder(W1=np.zeros((d, d), np.float32), b1=np.full(d, b1v, np.float32),
                                 W2=np.ones((d, d), np.float32), b2=np.full(d, -0.0, np.float32))
        tab = oracle.decoder_table(cfg, [dec])[0]
        assert np.all(tab == 0.0)
        assert not np.signbit(tab).any(), f"b1 = {b1v}: relu returned -0"


# ---------------------------------------------------------------- protected path
def test_q8_bounds_and_symmetry():
    r = _rng(50)
    w = r.normal(0, 0.02, (300, 64)).astype(np.float32)
    w[:, 10] *= 10
    w[:, 20] = 0.0
    idx = np.array([3, 10, 20, 63], np.int32)
    q, s = oracle.q8(w, idx)
    for p, j in enumerate(idx):
        col = w[:, j].astype(np.float64)
        if s[p] == 0:
            assert np.all(q[:, p] == 0) and np.all(col == 0)
            continue
        deq = q[:, p].astype(np.float64) * s[p]
        assert np.all(np.abs(deq - col) <= s[p] * (0.5 + 1e-6))
        am = np.argmax(np.abs(col))
        assert abs(int(q[am, p])) == 127
    qn, sn = oracle.q8(-w, idx)
    np.testing.assert_array_equal(qn, -q)
    np.testing.assert_array_equal(sn, s)


def test_topk_recovers_planted_outliers():
    """With ceil(d_in/100) input columns scaled x10, the protected set is exactly
    the planted set (eq. protected_channel_selection with g = 1)."""
    import torch
    for d_in, seed in ((512, 1), (1024, 2), (768, 3)):
        k = synth.n_outliers(d_in)
        w, cols = synth.weight(256, d_in, seed, k_outliers=k, dtype=torch.bfloat16)
        idx = oracle.protect_select(oracle.to_f32(w), k)
        np.testing.assert_array_equal(idx, cols)


def test_topk_ties_and_bruteforce():
    r = _rng(60)
    w = r.normal(0, 1, (50, 40)).astype(np.float32)
    keys = (w.astype(np.float64) ** 2).sum(axis=0)
    for k in range(0, 41, 7):
        want = np.sort(sorted(range(40), key=lambda j: (-keys[j], j))[:k])
        np.testing.assert_array_equal(oracle.protect_select(w, k), want)
    # exact ties: columns 5 and 9 identical and both at the boundary -> lower index wins
    w2 = np.ones((8, 12), np.float32)
    w2[:, 5] = 3.0
    w2[:, 9] = 3.0
    w2[:, 2] = 5.0
    np.testing.assert_array_equal(oracle.protect_select(w2, 2), [2, 5])
    # activation statistic g re-ranks columns: key = g^2 * sum w^2
    g = np.ones(12, np.float32)
    g[9] = 2.0
    np.testing.assert_array_equal(oracle.protect_select(w2, 2, g=g), [2, 9])


def test_protected_columns_leave_bsq_and_come_back_from_q8():
    """Assembly (eq. protected_8bit_scatter): W_hat[:, P] = Q8 exactly; the BSQ
    gains ignore the protected positions (a huge protected value does not
    change the BSQ part of its chunk)."""
    d = 8
    cfg = Config(d=d, b=d, stages=2, kind=KIND_MLP, hidden=8, protect_num=1, protect_den=16)
    decs = synth.decoder_params(KIND_MLP, d, d, 8, 2, seed=9)
    r = _rng(70)
    w = r.normal(0, 0.02, (64, 64)).astype(np.float32)
    w[:, 17] *= 50
    w[:, 40] *= 50
    w[:, 41] *= 40
    w[:, 60] *= 30
    enc = oracle.encode(cfg, decs, w)
    np.testing.assert_array_equal(enc.idx, [17, 40, 41, 60])
    w_hat = oracle.decode(cfg, decs, enc)
    for p, j in enumerate(enc.idx):
        np.testing.assert_array_equal(w_hat[:, j], enc.q8[:, p].astype(np.float32) * enc.scale[p])
    w2 = w.copy()
    w2[:, 17] *= 1000.0
    enc2 = oracle.encode(cfg, decs, w2)
    for s in range(2):
        np.testing.assert_array_equal(enc2.codes[s], enc.codes[s])
        np.testing.assert_array_equal(enc2.gains[s], enc.gains[s])


# ---------------------------------------------------------------- assembly, products
def test_decode_equals_fp64_assembly():
    d = 16
    cfg = Config(d=d, b=d, stages=2, kind=KIND_MLP, hidden=16, protect_num=1, protect_den=50)
    decs = synth.decoder_params(KIND_MLP, d, d, 16, 2, seed=13)
    tabs = oracle.decoder_table(cfg, decs)
    r = _rng(80)
    w = r.normal(0, 0.02, (40, 96)).astype(np.float32)
    enc = oracle.encode(cfg, decs, w, tables=tabs)
    w_hat = oracle.decode(cfg, decs, enc, tables=tabs)
    ref = np.zeros(w.shape)
    mag = np.zeros(w.shape)
    for s in range(2):
        codes = enc.codes[s][:, :96 // d].astype(np.int64)
        gains = _f16(enc.gains[s][:, :96 // d]).astype(np.float64)
        term = (gains[:, :, None] * tabs[s][codes].astype(np.float64)).reshape(40, 96)
        ref += term
        mag += np.abs(term)
    for p, j in enumerate(enc.idx):
        ref[:, j] = enc.q8[:, p].astype(np.float64) * enc.scale[p]
        mag[:, j] = np.abs(ref[:, j])
    # two fp32 roundings (the stage-1 product, the fused stage-2 update)
    assert np.all(np.abs(w_hat - ref) <= 2 ** -23 * 2 * mag + 1e-38)


@pytest.mark.parametrize("d", [8, 16])
def test_two_product_routes_agree(d):
    cfg = Config(d=d, b=d, stages=2, kind=KIND_MLP, hidden=d)
    decs = synth.decoder_params(KIND_MLP, d, d, d, 2, seed=17)
    r = _rng(90 + d)
    w = r.normal(0, 0.02, (96, 512)).astype(np.float32)
    w[:, [3, 100, 300, 301, 511]] *= 10
    enc = oracle.encode(cfg, decs, w)
    x = r.normal(0, 1, 512).astype(np.float32)
    A = r.normal(0, 0.01, (16, 512)).astype(np.float32)
    B = r.normal(0, 0.01, (96, 16)).astype(np.float32)
    y_dense = oracle.gemv(cfg, decs, enc, x, lora=(A, B))
    y_fused = oracle.gemv_fused(cfg, decs, enc, x, lora=(A, B))
    scale = np.sqrt(np.mean(y_dense ** 2))
    assert np.max(np.abs(y_dense - y_fused)) <= 1e-6 * scale
    # the LoRA term is really there
    assert np.max(np.abs(y_dense - oracle.gemv(cfg, decs, enc, x))) > 1e-3 * scale


def test_encode_rejects_nonfinite_and_ragged_chunks():
    cfg = Config(d=8, b=8, stages=2, kind=KIND_IDENTITY, protect_num=0)
    w = np.zeros((4, 16), np.float32)
    w[1, 3] = np.nan
    with pytest.raises(oracle.OracleError):
        oracle.encode(cfg, [synth.StageDecoder()] * 2, w)
    w[1, 3] = np.inf
    with pytest.raises(oracle.OracleError):
        oracle.encode(cfg, [synth.StageDecoder()] * 2, w)
    with pytest.raises(oracle.OracleError):
        oracle.encode(cfg, [synth.StageDecoder()] * 2, np.zeros((4, 12), np.float32))


def test_ragged_pitch_padding_is_zero():
    """Rows are padded to 16 chunks; padding holds code 0 and gain +0."""
    cfg = Config(d=8, b=8, stages=2, kind=KIND_MLP, hidden=8, protect_num=0)
    decs = synth.decoder_params(KIND_MLP, 8, 8, 8, 2, seed=1)
    w = _rng(3).normal(0, 1, (5, 8 * 21)).astype(np.float32)
    enc = oracle.encode(cfg, decs, w)
    assert enc.pitch == 32
    for s in range(2):
        assert np.all(enc.codes[s][:, 21:] == 0) and np.all(enc.gains[s][:, 21:] == 0)


def test_row_parallel_oracle_is_bit_identical():
    cfg = Config(d=8, b=8, stages=2, kind=KIND_MLP, hidden=8)
    decs = synth.decoder_params(KIND_MLP, 8, 8, 8, 2, seed=2)
    w = _rng(4).normal(0, 0.02, (300, 256)).astype(np.float32)
    e1 = oracle.encode(cfg, decs, w, nthreads=1)
    e4 = oracle.encode(cfg, decs, w, nthreads=4)
    for s in range(2):
        np.testing.assert_array_equal(e1.codes[s], e4.codes[s])
        np.testing.assert_array_equal(e1.gains[s], e4.gains[s])


# ---------------------------------------------------------------- accounting
def _golden():
    vals = {}
    with open(os.path.join(GOLDEN, "paper_rate_arithmetic.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                name, value = line.split()[:2]
                vals[name] = float(value)
    return vals


def test_rate_arithmetic_matches_paper():
    g = _golden()
    one = oracle.sizes(Config(d=32, b=32, stages=1, kind=KIND_IDENTITY, protect_num=0), 4096, 4096)
    two = oracle.sizes(Config(d=32, b=32, stages=2, kind=KIND_IDENTITY, protect_num=0), 4096, 4096)
    assert one["bpw_nominal"] == g["bpw_stage_b32_d32"]
    assert two["bpw_nominal"] == g["bpw_two_stage_b32_d32"]
    assert one["chunks"] == g["chunks_q_proj_4096x4096_d32"] == 2 ** 19
    assert abs(524286 / 2 ** 64 - g["occupied_fraction_524286_of_2p64"]) < 0.005e-14
    # S_code of one stage at b = d = 32 is exactly 1 bit per weight
    assert one["S_code"] * 8 == 4096 * 4096


def test_real_size_is_the_sum_of_its_parts():
    cfg = Config(d=8, b=8, stages=2, kind=KIND_MLP, hidden=8)
    s = oracle.sizes(cfg, 4096, 4096, lora_rank=16)
    assert s["S_tot"] == s["S_code"] + s["S_dec"] + s["S_8bit"] + s["S_LoRA"] + s["S_meta"]
    C = 4096 // 8
    assert s["S_code"] == 2 * 4096 * C                     # one byte per chunk per stage
    assert s["S_8bit"] == 4096 * 41                        # ceil(1% of 4096) = 41 columns
    assert s["S_LoRA"] == 2 * 16 * (4096 + 4096)
    assert s["S_dec"] == 2 * 4 * (8 * 8 + 8 + 8 * 8 + 8)
