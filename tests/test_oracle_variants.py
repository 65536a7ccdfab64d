"""Pins of the oracle's codec variants from the paper's component ablation
(Section IV-D, Table "BSQ codec components"): the symmetric decoder with one
residual block, the FP8-E4M3 / FP8-E5M2 formats of the protected path, and a
linear encoder z = E r (Section III-C's E_phi), which also allows code
lengths b other than the chunk length d (the b/d settings of Section III-D).

Each pin checks the oracle against something other than itself: torch's own
float8 conversions (a library routine), closed forms of the two formats,
special cases of the residual block that reduce to the pinned decoder without
one, an fp64 numpy evaluation of the decoder written from its definition,
encoders whose codes have a closed form (identity, positive scaling,
permutation, stacked and summed maps), and the signs of E r in fp64.
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import FMT_E4M3, FMT_E5M2, FMT_INT8, KIND_MLP, KIND_MLP_RES1, Config

TORCH_FP8 = {FMT_E4M3: torch.float8_e4m3fn, FMT_E5M2: torch.float8_e5m2}
FMAX = {FMT_INT8: 127.0, FMT_E4M3: 448.0, FMT_E5M2: 57344.0}
MBITS = {FMT_E4M3: 3, FMT_E5M2: 2}
EMIN = {FMT_E4M3: -6, FMT_E5M2: -14}     # exponent of the smallest normal


def _rng(seed):
    return np.random.default_rng(seed)


def _all_codes_q(b):
    """q for every b-bit code: +-1/sqrt(b) by bit j, LSB first (Section III-C)."""
    codes = np.arange(1 << b, dtype=np.int64)
    bits = (codes[:, None] >> np.arange(b)[None, :]) & 1
    return np.where(bits == 1, 1.0, -1.0) / math.sqrt(b)


def _torch_values(fmt):
    """fp32 value of every byte 0..255 under torch's float8 dtype."""
    raw = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    return raw.view(TORCH_FP8[fmt]).to(torch.float32).numpy()


def _torch_quant(v, fmt):
    return torch.from_numpy(np.asarray(v, np.float32)).to(TORCH_FP8[fmt]).view(torch.uint8).numpy()


# ---------------------------------------------------------------- FP8 payloads
@pytest.mark.parametrize("fmt", [FMT_E4M3, FMT_E5M2])
def test_fp8_byte_values_match_torch(fmt):
    """Every byte's value (finite, infinite or NaN) equals torch's float8
    reading of the same byte."""
    want = _torch_values(fmt)
    got = np.array([oracle.payload_value(v, fmt) for v in range(256)], dtype=np.float32)
    nan = np.isnan(want)
    np.testing.assert_array_equal(np.isnan(got), nan)
    np.testing.assert_array_equal(got[~nan], want[~nan])
    np.testing.assert_array_equal(np.signbit(got[~nan]), np.signbit(want[~nan]))


def test_fp8_closed_forms():
    v = oracle.payload_value
    assert v(0x7E, FMT_E4M3) == 448.0 and v(0xFE, FMT_E4M3) == -448.0
    assert math.isnan(v(0x7F, FMT_E4M3)) and math.isnan(v(0xFF, FMT_E4M3))
    assert v(0x01, FMT_E4M3) == 2.0 ** -9 and v(0x08, FMT_E4M3) == 2.0 ** -6
    assert v(0x38, FMT_E4M3) == 1.0 and v(0x3F, FMT_E4M3) == 1.875
    assert v(0x7B, FMT_E5M2) == 57344.0 and v(0x7C, FMT_E5M2) == math.inf
    assert v(0x01, FMT_E5M2) == 2.0 ** -16 and v(0x04, FMT_E5M2) == 2.0 ** -14
    assert v(0x3C, FMT_E5M2) == 1.0 and v(0x3F, FMT_E5M2) == 1.75
    assert oracle.payload_max(FMT_E4M3) == 448.0 and oracle.payload_max(FMT_E5M2) == 57344.0
    assert oracle.payload_max(FMT_INT8) == 127.0
    # int8 bytes are two's complement
    assert v(0x81, FMT_INT8) == -127.0 and v(0x7F, FMT_INT8) == 127.0


@pytest.mark.parametrize("fmt", [FMT_E4M3, FMT_E5M2])
def test_fp8_rounding_matches_torch(fmt):
    """In range (|v| <= largest finite), the stored byte is torch's cast:
    every representable value, every midpoint between neighbours (ties to
    the even code), points a quarter of a step off, signed zeros, and random
    values spread over the whole exponent range."""
    vals = _torch_values(fmt)[:128]
    fin = vals[np.isfinite(vals)]
    fin = fin[fin <= FMAX[fmt]]
    mids = (fin[:-1].astype(np.float64) + fin[1:]) / 2
    quarter = fin[:-1].astype(np.float64) + (fin[1:] - fin[:-1]) / 4
    r = _rng(7 + fmt)
    rand = np.exp(r.uniform(math.log(2.0 ** (EMIN[fmt] - MBITS[fmt] - 2)), math.log(FMAX[fmt]), 4000))
    pts = np.concatenate([fin, mids, quarter, rand, [0.0]]).astype(np.float32)
    pts = np.concatenate([pts, -pts])
    got = np.array([oracle.payload_quant(float(p), fmt) for p in pts], dtype=np.uint8)
    np.testing.assert_array_equal(got, _torch_quant(pts, fmt))
    # ties really go to the even code (both neighbours at equal distance)
    gm = np.array([oracle.payload_quant(float(p), fmt) for p in mids.astype(np.float32)])
    assert np.all(gm % 2 == 0)


@pytest.mark.parametrize("fmt", [FMT_E4M3, FMT_E5M2])
def test_fp8_saturates_and_keeps_sign(fmt):
    """Reading: magnitudes beyond the largest finite value store that value
    (the scale makes them rare: only fp32 rounding of the scale reaches past
    it); negative values that round to zero store the negative zero code."""
    top = 0x7E if fmt == FMT_E4M3 else 0x7B
    for m in (1.0000001, 1.03, 2.0, 1e6):
        assert oracle.payload_quant(FMAX[fmt] * m, fmt) == top
        assert oracle.payload_quant(-FMAX[fmt] * m, fmt) == 0x80 | top
    assert oracle.payload_quant(-1e-30, fmt) == 0x80
    assert oracle.payload_quant(-0.0, fmt) == 0x80
    assert oracle.payload_quant(0.0, fmt) == 0x00


@pytest.mark.parametrize("fmt", [FMT_INT8, FMT_E4M3, FMT_E5M2])
def test_protected_columns_in_each_format(fmt):
    """Q8 of protected columns in each format: scale = column max / the
    format's largest finite value; the column's largest magnitude stores that
    value; every stored value is within half a step of w / scale (steps from
    the format's definition); negating w negates every stored value."""
    r = _rng(60 + fmt)
    w = r.normal(0, 0.02, (300, 64)).astype(np.float32)
    w[:, 10] *= 10
    w[:, 20] = 0.0
    w[5, 30] = 1e-30           # tiny entries fall in the subnormal range of the format
    idx = np.array([3, 10, 20, 30, 63], np.int32)
    q, s = oracle.q8(w, idx, fmt)
    np.testing.assert_array_equal(s, np.abs(w[:, idx]).max(axis=0) / np.float32(FMAX[fmt]))
    vals = oracle.payload_values(q, fmt).astype(np.float64)
    for p, j in enumerate(idx):
        col = w[:, j].astype(np.float64)
        if s[p] == 0:
            assert np.all(q[:, p] == 0) and np.all(col == 0)
            continue
        t = col / np.float64(s[p])
        if fmt == FMT_INT8:
            step = np.ones_like(t)
        else:
            e = np.floor(np.log2(np.maximum(np.abs(t), 2.0 ** EMIN[fmt])))
            step = 2.0 ** (e - MBITS[fmt])
        assert np.all(np.abs(vals[:, p] - t) <= 0.5 * step * (1 + 1e-6))
        am = np.argmax(np.abs(col))
        assert abs(vals[am, p]) == FMAX[fmt]
    qn, sn = oracle.q8(-w, idx, fmt)
    np.testing.assert_array_equal(oracle.payload_values(qn, fmt), -oracle.payload_values(q, fmt))
    np.testing.assert_array_equal(sn, s)


@pytest.mark.parametrize("fmt", [FMT_E4M3, FMT_E5M2])
@pytest.mark.parametrize("axis", [0, 1])
def test_fp8_payload_reaches_decode_and_products(fmt, axis):
    """Encode with an FP8 protected path on either axis: the decoded protected
    slices are torch's reading of the stored bytes times the scale (one fp32
    product), the BSQ part equals the int8-path encoding (the format does not
    touch the codes), and the two product routes agree."""
    d = 8
    base = Config(d=d, b=d, stages=2, kind=KIND_MLP, hidden=8, protect_num=1, protect_den=16,
                  protect_axis=axis)
    cfg = Config(**{**base.__dict__, "protect_format": fmt})
    decs = synth.decoder_params(KIND_MLP, d, d, 8, 2, seed=9)
    r = _rng(70 + fmt)
    w = r.normal(0, 0.02, (64, 64)).astype(np.float32)
    w[:, [17, 40]] *= 50
    w[[5, 33], :] *= 30
    enc = oracle.encode(cfg, decs, w)
    enc8 = oracle.encode(base, decs, w)
    np.testing.assert_array_equal(enc.idx, enc8.idx)
    for s in range(2):
        np.testing.assert_array_equal(enc.codes[s], enc8.codes[s])
        np.testing.assert_array_equal(enc.gains[s], enc8.gains[s])
    w_hat = oracle.decode(cfg, decs, enc)
    tv = _torch_values(fmt)
    for p, j in enumerate(enc.idx):
        if axis == 0:
            np.testing.assert_array_equal(w_hat[:, j], tv[enc.q8[:, p].view(np.uint8)] * enc.scale[p])
        else:
            np.testing.assert_array_equal(w_hat[j, :], tv[enc.q8[p].view(np.uint8)] * enc.scale[p])
    x = r.normal(0, 1, 64).astype(np.float32)
    y_dense = oracle.gemv(cfg, decs, enc, x)
    y_fused = oracle.gemv_fused(cfg, decs, enc, x)
    assert np.max(np.abs(y_dense - y_fused)) <= 1e-6 * np.sqrt(np.mean(y_dense ** 2))


# ---------------------------------------------------------------- res1 decoder
def _res1(d, h, seed, R=None, c=None):
    dec = synth.decoder_params(synth.DEC_MLP_RES1, d, d, h, 1, seed=seed)[0]
    if R is not None:
        dec.R = np.asarray(R, np.float32)
    if c is not None:
        dec.c = np.asarray(c, np.float32)
    return dec


def _cfg(d, h, kind=KIND_MLP_RES1):
    return Config(d=d, b=d, stages=1, kind=kind, hidden=h, protect_num=0)


@pytest.mark.parametrize("d,h", [(8, 8), (8, 5), (16, 16)])
def test_res1_with_a_dead_block_is_the_plain_decoder(d, h):
    """R = 0, c = 0, and R = -I, c = 0 (relu(-a) = +0 for a >= 0): the block
    adds +0 to every hidden unit, so the table is the plain symmetric decoder's
    bit for bit."""
    dec = _res1(d, h, 500 + h)
    plain = synth.StageDecoder(W1=dec.W1, b1=dec.b1, W2=dec.W2, b2=dec.b2)
    want = oracle.decoder_table(_cfg(d, h, KIND_MLP), [plain])[0]
    for R in (np.zeros((h, h)), -np.eye(h)):
        got = oracle.decoder_table(_cfg(d, h), [_res1(d, h, 500 + h, R=R, c=np.zeros(h))])[0]
        np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("d,h", [(8, 8), (8, 16), (16, 16)])
def test_res1_identity_block_doubles_the_hidden_layer(d, h):
    """R = I, c = 0: the block adds relu(a) = a, so a' = 2a exactly, and the
    table is the plain decoder's with W2 doubled (W2 (2a) and (2 W2) a are
    the same exact products), bit for bit."""
    dec = _res1(d, h, 600 + h, R=np.eye(h), c=np.zeros(h))
    plain2 = synth.StageDecoder(W1=dec.W1, b1=dec.b1, W2=(2 * dec.W2).astype(np.float32), b2=dec.b2)
    want = oracle.decoder_table(_cfg(d, h, KIND_MLP), [plain2])[0]
    got = oracle.decoder_table(_cfg(d, h), [dec])[0]
    np.testing.assert_array_equal(got, want)


def _numpy_res1(dec, b):
    q = _all_codes_q(b).astype(np.float32).astype(np.float64)
    W1, b1, W2, b2, R, c = (v.astype(np.float64) for v in (dec.W1, dec.b1, dec.W2, dec.b2, dec.R, dec.c))
    pre = q @ W1.T + b1[None, :]
    a = np.maximum(pre, 0.0)
    t = np.maximum(a @ R.T + c[None, :], 0.0)
    ap = a + t
    y = ap @ W2.T + b2[None, :]
    # propagated fp32 rounding: each chain rounds once per step (relative
    # 2^-24 of its magnitudes), relu is 1-Lipschitz, the block's add rounds once
    u = 2.0 ** -24
    h = W1.shape[0]
    ea = (b + 1) * u * (np.abs(b1)[None, :] + np.abs(q) @ np.abs(W1).T)
    et = ea @ np.abs(R).T + (h + 1) * u * (np.abs(c)[None, :] + (a + ea) @ np.abs(R).T)
    eap = ea + et + u * (ap + ea + et)
    ey = eap @ np.abs(W2).T + (h + 1) * u * (np.abs(b2)[None, :] + (ap + eap) @ np.abs(W2).T)
    return y, ey


@pytest.mark.parametrize("d,h", [(8, 8), (8, 5), (8, 16), (16, 16), (16, 7)])
def test_res1_against_numpy(d, h):
    """Random parameters, every code, against an fp64 numpy evaluation of
    W2 (a + relu(R a + c)) + b2 with a = relu(W1 q + b1). A transposed R, a
    dropped c, the relu of the block left out or put after the add, or the
    skip connection dropped all fail the bound, which sits far below the
    values it guards."""
    dec = _res1(d, h, 700 + 10 * d + h)
    got = oracle.decoder_table(_cfg(d, h), [dec])[0]
    want, bound = _numpy_res1(dec, d)
    assert np.all(np.abs(got - want) <= bound)
    assert np.abs(want).max() > 100 * bound.max()
    # the planted mistakes, evaluated in numpy, all sit far outside the bound
    q = _all_codes_q(d)
    W1, b1, W2, b2, R, c = (v.astype(np.float64) for v in (dec.W1, dec.b1, dec.W2, dec.b2, dec.R, dec.c))
    a = np.maximum(q @ W1.T + b1, 0.0)
    wrong = {
        "R transposed": a + np.maximum(a @ R + c, 0.0),
        "c dropped": a + np.maximum(a @ R.T, 0.0),
        "no block relu": a + (a @ R.T + c),
        "relu after add": np.maximum(a + a @ R.T + c, 0.0),
        "no skip": np.maximum(a @ R.T + c, 0.0),
    }
    for name, ap in wrong.items():
        yw = ap @ W2.T + b2
        assert np.max(np.abs(yw - want) - bound) > 0, name


def test_res1_permutation_block_closed_form():
    """R a permutation matrix (not its own inverse) and c = 0: a'_k =
    a_k + a_perm(k), each output an fmaf chain over exact products. Compared
    against numpy with the permutation applied explicitly."""
    d = h = 8
    perm = np.array([1, 2, 3, 4, 5, 6, 7, 0])      # a cycle: perm != perm^-1
    R = np.eye(h, dtype=np.float32)[perm]           # (R a)_k = a_perm(k)
    dec = _res1(d, h, 800, R=R, c=np.zeros(h))
    got = oracle.decoder_table(_cfg(d, h), [dec])[0]
    q = _all_codes_q(d).astype(np.float32).astype(np.float64)
    W1, b1, W2, b2 = (v.astype(np.float64) for v in (dec.W1, dec.b1, dec.W2, dec.b2))
    a = np.maximum(q @ W1.T + b1, 0.0)
    want = (a + a[:, perm]) @ W2.T + b2
    bound = 40 * 2.0 ** -24 * (np.abs(a + a[:, perm]) @ np.abs(W2).T + np.abs(b2) + 1e-30)
    assert np.all(np.abs(got - want) <= bound)
    inv = np.argsort(perm)
    assert np.max(np.abs((a + a[:, inv]) @ W2.T + b2 - want) - bound) > 0


def test_res1_storage_counts_the_block():
    cfg = Config(d=8, b=8, stages=2, kind=KIND_MLP_RES1, hidden=8)
    plain = Config(d=8, b=8, stages=2, kind=KIND_MLP, hidden=8)
    assert oracle.decoder_param_count(cfg) == oracle.decoder_param_count(plain) + 8 * 8 + 8
    assert oracle.sizes(cfg, 64, 64)["S_dec"] == 2 * 4 * oracle.decoder_param_count(cfg)


# ---------------------------------------------------------------- linear encoder, b != d
from oracle import ENC_LINEAR, KIND_LINEAR  # noqa: E402


def _enc_cfg(d, b, stages=1, kind=KIND_MLP, h=None, **kw):
    return Config(d=d, b=b, stages=stages, kind=kind, hidden=h or b, encoder=ENC_LINEAR, **kw)


def _with_E(decs, Es):
    out = []
    for dec, E in zip(decs, Es):
        nd = synth.StageDecoder(W1=dec.W1, b1=dec.b1, W2=dec.W2, b2=dec.b2)
        nd.E = np.asarray(E, np.float32)
        out.append(nd)
    return out


def _bits_of(codes, b):
    c = np.asarray(codes).astype(np.int64)
    return (c[..., None] >> np.arange(b)) & 1


@pytest.mark.parametrize("d", [8, 16])
def test_encoder_identity_and_positive_scaling_are_the_plain_encoder(d):
    """E = I, and E = a positive diagonal (sign(E r) = sign(r)), reproduce the
    identity-encoder encoding bit for bit: codes, gains, payload, every stage."""
    plain_cfg = Config(d=d, b=d, stages=2, kind=KIND_MLP, hidden=d)
    decs = synth.decoder_params(KIND_MLP, d, d, d, 2, seed=31)
    r = _rng(900 + d)
    w = r.normal(0, 0.02, (96, 512)).astype(np.float32)
    w[:, [5, 300]] *= 10
    want = oracle.encode(plain_cfg, decs, w)
    scales = r.uniform(0.01, 50.0, d).astype(np.float32)
    for E in (np.eye(d), np.diag(scales)):
        got = oracle.encode(_enc_cfg(d, d, stages=2, h=d), _with_E(decs, [E, E]), w)
        for s in range(2):
            np.testing.assert_array_equal(got.codes[s], want.codes[s])
            np.testing.assert_array_equal(got.gains[s], want.gains[s])
        np.testing.assert_array_equal(got.q8, want.q8)


def test_encoder_permutation_permutes_the_code_bits():
    """E a permutation (b = d = 8, one stage): bit m of the code is bit
    perm(m) of the identity encoder's code."""
    d = 8
    perm = np.array([3, 0, 7, 1, 6, 2, 5, 4])
    decs = synth.decoder_params(KIND_MLP, d, d, d, 1, seed=32)
    w = _rng(910).normal(0, 0.02, (64, 256)).astype(np.float32)
    ident = oracle.encode(Config(d=d, b=d, stages=1, kind=KIND_MLP, hidden=d), decs, w)
    got = oracle.encode(_enc_cfg(d, d), _with_E(decs, [np.eye(d)[perm]]), w)
    np.testing.assert_array_equal(_bits_of(got.codes[0], d), _bits_of(ident.codes[0], d)[..., perm])


@pytest.mark.parametrize("d,b", [(8, 16), (16, 8)])
def test_encoder_stacked_and_summed_maps(d, b):
    """b = 2d with E = [I; -I]: the high byte is the complement of the low
    one, which is the identity code. b = d/2 with E summing pairs
    (z_m = r_2m + r_2m+1, one rounding): bit m is the sign of that sum,
    computed here in fp32 from the definition. No protected columns and no
    zeros, so every z is nonzero."""
    decs = synth.decoder_params(KIND_LINEAR, d, b, b, 1, seed=33)
    w = _rng(920 + d).normal(0, 0.02, (64, 256)).astype(np.float32)
    C = 256 // d
    chunks = w.reshape(64, C, d)
    if b == 2 * d:
        E = np.vstack([np.eye(d), -np.eye(d)])
        got = oracle.encode(_enc_cfg(d, b, kind=KIND_LINEAR, protect_num=0), _with_E(decs, [E]), w)
        lo = (chunks >= 0).astype(np.int64)
        want = (lo * (1 << np.arange(d))).sum(-1) | (((1 - lo) * (1 << np.arange(d, 2 * d))).sum(-1))
    else:
        E = np.zeros((b, d), np.float32)
        E[np.arange(b), 2 * np.arange(b)] = 1
        E[np.arange(b), 2 * np.arange(b) + 1] = 1
        got = oracle.encode(_enc_cfg(d, b, kind=KIND_LINEAR, protect_num=0), _with_E(decs, [E]), w)
        z = chunks[..., 0::2] + chunks[..., 1::2]          # fp32 sums, one rounding each
        want = ((z >= 0).astype(np.int64) * (1 << np.arange(b))).sum(-1)
    np.testing.assert_array_equal(got.codes[0][:, :C].astype(np.int64), want)


@pytest.mark.parametrize("d,b", [(8, 16), (16, 8), (8, 8)])
def test_random_encoder_codes_are_the_signs_of_E_r(d, b):
    """A random E: every code bit is the sign of z = E r evaluated in fp64
    wherever |z| exceeds the fmaf chain's rounding bound (the sphere map's
    sign rule of Section III-C applied to the encoder output), at both
    stages, with the stage-2 residual recomputed from the stage-1 code and
    gain by the definition."""
    cfg = _enc_cfg(d, b, stages=2, h=b, protect_num=0)
    decs = synth.decoder_params(KIND_MLP, d, b, b, 2, seed=34, encoder=True)
    w = _rng(930 + d + b).normal(0, 0.02, (48, 128)).astype(np.float32)
    tabs = oracle.decoder_table(cfg, decs)
    enc = oracle.encode(cfg, decs, w, tables=tabs)
    C = 128 // d
    r = w.reshape(48, C, d).astype(np.float32)
    checked = 0
    for s in range(2):
        E = decs[s].E.astype(np.float64)
        z = r.astype(np.float64) @ E.T
        bound = (d + 1) * 2.0 ** -24 * (np.abs(r).astype(np.float64) @ np.abs(E).T)
        sure = np.abs(z) > bound
        bits = _bits_of(enc.codes[s][:, :C], b)
        assert np.all(bits[sure] == (z[sure] >= 0))
        checked += int(sure.sum())
        # next stage's target: r - a y with the stage's code and gain (fmaf per element)
        codes = enc.codes[s][:, :C].astype(np.int64)
        a = oracle.f16_bits_to_f32(enc.gains[s][:, :C]).astype(np.float32)
        y = tabs[s][codes]
        r = (r.astype(np.float64) - a[..., None].astype(np.float64) * y.astype(np.float64)).astype(np.float32)
    assert checked > 0.99 * 2 * 48 * C * b


@pytest.mark.parametrize("d,b", [(8, 16), (16, 8)])
def test_b_ne_d_routes_agree_and_residual_never_increases(d, b):
    """b != d: the decode assembly and the two product routes agree, and each
    stage's least-squares gain keeps the reconstruction error from growing
    (whatever the encoder picked); code planes are 8-bit for b = 8 and 16-bit
    for b = 16; sizes count b bits per chunk and stage and the encoder."""
    cfg = _enc_cfg(d, b, stages=2, h=b, protect_num=1, protect_den=32)
    decs = synth.decoder_params(KIND_MLP, d, b, b, 2, seed=35, encoder=True)
    r = _rng(940 + d)
    w = r.normal(0, 0.02, (80, 512)).astype(np.float32)
    w[:, [17, 400]] *= 10
    enc = oracle.encode(cfg, decs, w)
    assert enc.codes[0].dtype == (np.uint8 if b == 8 else np.uint16)
    x = r.normal(0, 1, 512).astype(np.float32)
    y_dense = oracle.gemv(cfg, decs, enc, x)
    y_fused = oracle.gemv_fused(cfg, decs, enc, x)
    assert np.max(np.abs(y_dense - y_fused)) <= 1e-6 * np.sqrt(np.mean(y_dense ** 2))
    one = _enc_cfg(d, b, stages=1, h=b, protect_num=1, protect_den=32)
    e1 = oracle.encode(one, decs, w)
    keep = np.ones(512, bool)
    keep[enc.idx] = False
    err0 = float(np.sum(w[:, keep].astype(np.float64) ** 2))
    err1 = float(np.sum((oracle.decode(one, decs, e1) - w)[:, keep].astype(np.float64) ** 2))
    err2 = float(np.sum((oracle.decode(cfg, decs, enc) - w)[:, keep].astype(np.float64) ** 2))
    assert err1 <= err0 * (1 + 1e-6) and err2 <= err1 * (1 + 1e-6)
    sz = oracle.sizes(cfg, 80, 512)
    assert sz["S_code"] == 2 * 80 * (512 // d) * b / 8
    assert sz["S_dec"] == 2 * 4 * (oracle.decoder_param_count(cfg) + b * d)
    assert sz["bpw_nominal"] == 2 * b / d


def test_encoder_required_for_b_ne_d():
    decs = synth.decoder_params(KIND_MLP, 8, 16, 16, 1, seed=36)
    w = np.ones((8, 64), np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.encode(Config(d=8, b=16, stages=1, kind=KIND_MLP, hidden=16), decs, w)
    with pytest.raises(oracle.OracleError):
        oracle.encode(_enc_cfg(8, 16), decs, w)       # encoder config but no E
