"""Pins of the oracle's output-row and coupled MLP protection.

Covered: the coupled score of eq. mlp_coupled_protection, row protection
(eq. protected_channel_selection applied to output channels, eq.
protected_8bit_scatter with row slices) and encode with a given protected set.
Each test checks the oracle against something other than itself: a closed
form with exactly representable norms, a reduction to the column path pinned
in test_oracle_pins.py, a transpose identity, or bit-identity with the
unprotected encoding of the same rows.
"""
import numpy as np
import pytest

import oracle
import synth
from oracle import KIND_MLP, Config


def _rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- coupled score
def test_coupled_score_closed_form_and_ties():
    """S_j = |g_gate| ||gate row j|| + |g_up| ||up row j|| + |g_down| ||down col j||
    on rows and columns with integer norms (3-4-5, 6-8-10, 1-2-2-3), so every
    term is exact; a tie goes to the lower channel; a negative statistic
    counts by its magnitude."""
    d_model, d_ffn = 4, 6
    a = np.array([1, 0, 2, 1, 0, 3], np.float64)   # gate row j = (3a, 4a, 0, 0): norm 5|a|
    b = np.array([0, 1, 1, 0, 2, 0], np.float64)   # up row j = (0, 0, 6b, 8b): norm 10|b|
    c = np.array([2, 1, 0, 4, 1, 0], np.float64)   # down column j = (c, 2c, 2c, 0): norm 3|c|
    wg = np.zeros((d_ffn, d_model), np.float32)
    wu = np.zeros((d_ffn, d_model), np.float32)
    wd = np.zeros((d_model, d_ffn), np.float32)
    wg[:, 0], wg[:, 1] = 3 * a, 4 * a
    wu[:, 2], wu[:, 3] = 6 * b, -8 * b
    wd[0, :], wd[1, :], wd[2, :] = c, -2 * c, 2 * c
    gg = np.array([1, 2, 1, 0.5, 1, 1], np.float32)
    gu = np.array([1, 1, -2, 1, 0.25, 1], np.float32)
    gd = np.array([0.5, 1, 1, 1, 4, 1], np.float32)
    want = np.abs(gg) * 5 * a + np.abs(gu) * 10 * b + np.abs(gd) * 3 * c
    # channels: 0 -> 5+0+3 = 8; 1 -> 0+10+3 = 13; 2 -> 10+20+0 = 30;
    #           3 -> 2.5+0+12 = 14.5; 4 -> 0+5+12 = 17; 5 -> 15+0+0 = 15
    idx, score = oracle.coupled_select(wg, wu, wd, 3, gg, gu, gd)
    np.testing.assert_array_equal(score, want)
    np.testing.assert_array_equal(idx, [2, 4, 5])
    # ties at the cut go to the lower channel: gate norms 5a with up = down = 0
    for a2, k, want_idx in (([2, 4, 4, 1], 1, [1]), ([4, 4, 4, 1], 2, [0, 1]), ([1, 3, 2, 3], 1, [1])):
        a2 = np.array(a2, np.float32)
        wg2 = np.zeros((4, d_model), np.float32)
        wg2[:, 0], wg2[:, 1] = 3 * a2, 4 * a2
        z = np.zeros((4, d_model), np.float32)
        idx2, score2 = oracle.coupled_select(wg2, z, np.zeros((d_model, 4), np.float32), k)
        np.testing.assert_array_equal(score2, 5.0 * a2.astype(np.float64))
        np.testing.assert_array_equal(idx2, want_idx)


def test_coupled_score_defaults_and_brute_force():
    """g = NULL means ones; on random data the score agrees with an
    independent fp64 numpy evaluation to rounding, and the set is the k
    channels of largest score."""
    r = _rng(5)
    d_model, d_ffn, k = 24, 80, 7
    wg = r.normal(0, 1, (d_ffn, d_model)).astype(np.float32)
    wu = r.normal(0, 1, (d_ffn, d_model)).astype(np.float32)
    wd = r.normal(0, 1, (d_model, d_ffn)).astype(np.float32)
    idx, score = oracle.coupled_select(wg, wu, wd, k)
    ref = (np.linalg.norm(wg.astype(np.float64), axis=1) + np.linalg.norm(wu.astype(np.float64), axis=1)
           + np.linalg.norm(wd.astype(np.float64), axis=0))
    np.testing.assert_allclose(score, ref, rtol=1e-14)
    np.testing.assert_array_equal(idx, np.sort(np.argsort(-ref, kind="stable")[:k]))
    ones = np.ones(d_ffn, np.float32)
    idx1, score1 = oracle.coupled_select(wg, wu, wd, k, ones, ones, ones)
    np.testing.assert_array_equal(score1, score)
    np.testing.assert_array_equal(idx1, idx)


def test_coupled_reduces_to_single_matrix_selection():
    """With gate = up = 0 the coupled set is down's own input-column set
    (column keys g^2 sum w^2 rank like |g| ||w||); with up = down = 0 it is
    gate's own output-row set."""
    r = _rng(6)
    d_model, d_ffn, k = 32, 96, 5
    wd = r.normal(0, 1, (d_model, d_ffn)).astype(np.float32)
    gd = r.uniform(0.5, 2.0, d_ffn).astype(np.float32)
    z = np.zeros((d_ffn, d_model), np.float32)
    idx, _ = oracle.coupled_select(z, z, wd, k, None, None, gd)
    np.testing.assert_array_equal(idx, oracle.protect_select(wd, k, g=gd))
    wg = r.normal(0, 1, (d_ffn, d_model)).astype(np.float32)
    idx_g, _ = oracle.coupled_select(wg, z, np.zeros((d_model, d_ffn), np.float32), k)
    np.testing.assert_array_equal(idx_g, oracle.topk(oracle.row_keys(wg), k))


def test_row_keys_are_column_keys_of_the_transpose():
    """The same fp64 sums in the same element order: bit-identical."""
    r = _rng(7)
    w = r.normal(0, 1, (33, 70)).astype(np.float32)
    g = r.uniform(0, 2, 33).astype(np.float32)
    np.testing.assert_array_equal(oracle.row_keys(w, g), oracle.column_keys(np.ascontiguousarray(w.T), g))


def test_topk_matches_sort_with_index_tiebreak():
    r = _rng(8)
    key = r.integers(0, 6, 200).astype(np.float64)  # many ties
    for k in (0, 1, 13, 200):
        want = np.sort(sorted(range(200), key=lambda j: (-key[j], j))[:k])
        np.testing.assert_array_equal(oracle.topk(key, k), want)


# ---------------------------------------------------------------- row Q8
def test_q8_rows_is_column_q8_of_the_transpose_and_bounded():
    r = _rng(9)
    w = r.normal(0, 0.05, (40, 72)).astype(np.float32)
    w[11] = 0.0  # an all-zero protected row: scale 0, codes 0
    idx = np.array([2, 11, 19, 39], np.int32)
    q, s = oracle.q8_rows(w, idx)
    qt, st = oracle.q8(np.ascontiguousarray(w.T), idx)
    np.testing.assert_array_equal(q, qt.T)
    np.testing.assert_array_equal(s, st)
    assert s[1] == 0.0 and not q[1].any()
    for p, i in enumerate(idx):
        if s[p] == 0:
            continue
        assert np.abs(q[p]).max() == 127
        err = np.abs(q[p].astype(np.float64) * s[p] - w[i])
        assert err.max() <= 0.5 * s[p] * (1 + 1e-6)


# ---------------------------------------------------------------- encode / decode with rows
def _setup(d=8, seed=11):
    decs = synth.decoder_params(KIND_MLP, d, d, d, 2, seed=seed)
    return decs


@pytest.mark.parametrize("d", [8, 16])
def test_row_protection_leaves_other_rows_bit_identical(d):
    """Protecting rows masks no position, so every other row encodes exactly
    as with no protection at all; protected rows carry code 0 / gain +0 and
    come back from Q8 in the decode."""
    decs = _setup(d)
    r = _rng(12)
    w = r.normal(0, 0.02, (48, 128)).astype(np.float32)
    idx = np.array([3, 17, 40], np.int32)
    cfg_rows = Config(d=d, b=d, stages=2, kind=KIND_MLP, hidden=d, protect_num=1, protect_den=16,
                      protect_axis=1)
    cfg_none = Config(d=d, b=d, stages=2, kind=KIND_MLP, hidden=d, protect_num=0, protect_den=1)
    enc = oracle.encode_set(cfg_rows, decs, w, idx)
    ref = oracle.encode(cfg_none, decs, w)
    keep = np.setdiff1d(np.arange(48), idx)
    for s in range(2):
        np.testing.assert_array_equal(enc.codes[s][keep], ref.codes[s][keep])
        np.testing.assert_array_equal(enc.gains[s][keep], ref.gains[s][keep])
        assert not enc.codes[s][idx].any() and not enc.gains[s][idx].any()
    q, sc = oracle.q8_rows(w, idx)
    np.testing.assert_array_equal(enc.q8, q)
    np.testing.assert_array_equal(enc.scale, sc)
    w_hat = oracle.decode(cfg_rows, decs, enc)
    w_ref = oracle.decode(cfg_none, decs, ref)
    np.testing.assert_array_equal(w_hat[keep], w_ref[keep])
    for p, i in enumerate(idx):
        np.testing.assert_array_equal(w_hat[i], q[p].astype(np.float32) * sc[p])


def test_row_axis_self_selection_finds_planted_rows():
    decs = _setup(8)
    r = _rng(13)
    w = r.normal(0, 0.02, (48, 64)).astype(np.float32)
    w[5] *= 40
    w[30] *= 30
    cfg = Config(d=8, b=8, stages=2, kind=KIND_MLP, hidden=8, protect_num=1, protect_den=24,
                 protect_axis=1)
    assert cfg.k_for(48, 64) == 2
    enc = oracle.encode(cfg, decs, w)
    np.testing.assert_array_equal(enc.idx, [5, 30])
    assert enc.axis == 1 and enc.q8.shape == (2, 64)


def test_given_column_set_equals_self_selected_encode():
    """Column axis: encode with the set the self-selecting encoder picked is
    bit-identical to it (codes, gains, int8 payload, scales)."""
    decs = _setup(8)
    r = _rng(14)
    w = r.normal(0, 0.02, (40, 256)).astype(np.float32)
    w[:, [7, 99, 200]] *= 30
    cfg = Config(d=8, b=8, stages=2, kind=KIND_MLP, hidden=8, protect_num=1, protect_den=100)
    enc = oracle.encode(cfg, decs, w)
    enc2 = oracle.encode_set(cfg, decs, w, enc.idx)
    for s in range(2):
        np.testing.assert_array_equal(enc2.codes[s], enc.codes[s])
        np.testing.assert_array_equal(enc2.gains[s], enc.gains[s])
    np.testing.assert_array_equal(enc2.q8, enc.q8)
    np.testing.assert_array_equal(enc2.scale, enc.scale)


def test_row_protection_product_routes_agree():
    """The fused route (coded rows + scale_p <q8_p, x> + LoRA) and the dense
    route (decode, fp64 matmul) agree; a protected row is the plain int8 dot."""
    decs = _setup(8)
    r = _rng(15)
    w = r.normal(0, 0.02, (64, 128)).astype(np.float32)
    idx = np.array([0, 9, 63], np.int32)
    cfg = Config(d=8, b=8, stages=2, kind=KIND_MLP, hidden=8, protect_num=1, protect_den=22,
                 protect_axis=1)
    enc = oracle.encode_set(cfg, decs, w, idx)
    x = r.normal(0, 1, 128)
    A = r.normal(0, 0.05, (4, 128))
    B = r.normal(0, 0.05, (64, 4))
    y1 = oracle.gemv_fused(cfg, decs, enc, x, (A, B))
    y2 = oracle.gemv(cfg, decs, enc, x, (A, B))
    # the dense route rounds W_hat to fp32 (as the column-path test allows)
    scale = np.sqrt(np.mean(y2 ** 2))
    assert np.max(np.abs(y1 - y2)) <= 1e-6 * scale
    for p, i in enumerate(idx):
        want = sum(float(enc.scale[p]) * float(enc.q8[p, j]) * x[j] for j in range(128)) + B[i] @ (A @ x)
        assert abs(y1[i] - want) <= 1e-9 * (1 + abs(want))


def test_encode_set_rejects_invalid_sets():
    decs = _setup(8)
    w = np.zeros((16, 32), np.float32)
    cfg = Config(d=8, b=8, stages=2, kind=KIND_MLP, hidden=8, protect_num=1, protect_den=8,
                 protect_axis=1)
    for bad in ([3, 3], [5, 2], [-1, 4], [4, 16]):
        with pytest.raises(oracle.OracleError):
            oracle.encode_set(cfg, decs, w, np.array(bad, np.int32))


def test_row_protection_size_accounting():
    """eq. real_size with row slices: the protected rows hold d_in int8 values
    each and no BSQ codes or gains."""
    cfg = Config(d=8, b=8, stages=2, kind=KIND_MLP, hidden=8, protect_num=1, protect_den=100,
                 protect_axis=1)
    s = oracle.sizes(cfg, 12288, 4096)
    k = (12288 + 99) // 100
    assert s["k"] == k == 123
    assert s["S_8bit"] == k * 4096
    assert s["S_code"] == 2 * (12288 - k) * 512
    assert s["S_meta"] == 2 * (12288 - k) * 512 * 2 + 8 * k
    assert s["S_tot"] == s["S_code"] + s["S_dec"] + s["S_8bit"] + s["S_LoRA"] + s["S_meta"]
