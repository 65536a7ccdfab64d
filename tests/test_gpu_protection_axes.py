"""Protected output rows and the coupled MLP channel set on the GPU, against
the oracle through the C ABI (bsq_encode / bsq_encode_with_set with
protect_axis = 1, bsq_coupled_select, and the products over row-protected
layers).

Bar as for the column axis: codes, gains, indices, int8 rows and scales
bit-exact; coupled scores bit-exact (fp64, same order); fp32 decode
bit-exact; products within 2e-2 relative (bf16 activations) or 1e-4 (fp32)
with the derived floors of tests/parity_bounds.py.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_08643_amd as bsq
import synth
from test_gpu_parity import OFMT, OKIND, check_product, decoders, gemv_kind, np_codes, np_gains, say

pytestmark = pytest.mark.gpu


def ocfg(cfg: bsq.Config) -> oracle.Config:
    return oracle.Config(d=cfg.d, b=cfg.d, stages=cfg.stages, kind=OKIND[cfg.kind], hidden=cfg.hidden,
                         protect_num=cfg.protect_num, protect_den=cfg.protect_den, protect_axis=cfg.protect_axis,
                         protect_format=OFMT[cfg.protect_format])


def planted_rows(d_out, k, seed):
    """k distinct rows (seeded) that the test scales up, so that the row
    energy TopK has a clear answer."""
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(d_out, size=k, replace=False)).astype(np.int32)


def row_weight(d_out, d_in, seed, k, dtype, n_mats=1):
    W, _ = synth.weight(d_out, d_in, seed, dtype=torch.float32, n_mats=n_mats)
    W = W.reshape(n_mats, d_out, d_in).clone()
    for m in range(n_mats):
        if k:
            W[m, torch.as_tensor(planted_rows(d_out, k, seed + m))] *= 10.0
    W = W.to(dtype)
    return W[0] if n_mats == 1 else W


def assert_rows_layer_equal(L, enc, cfg):
    for s in range(cfg.stages):
        np.testing.assert_array_equal(np_codes(L, L.codes[s]), enc.codes[s], err_msg=f"codes stage {s}")
        np.testing.assert_array_equal(np_gains(L, L.gains[s]), enc.gains[s], err_msg=f"gains stage {s}")
    k = L.k
    assert k == len(enc.idx)
    if not k:
        return
    np.testing.assert_array_equal(L.idx.cpu().numpy(), enc.idx, err_msg="protected rows")
    q8 = L.q8.cpu().numpy()
    np.testing.assert_array_equal(q8[:, :L.d_in], enc.q8, err_msg="int8 rows")
    assert not q8[:, L.d_in:].any(), "int8 row padding"
    np.testing.assert_array_equal(L.scale.cpu().numpy().view(np.uint32), enc.scale.view(np.uint32),
                                  err_msg="row scales")


# (name, d_out, d_in, cfg kwargs, dtype, n_mats, with_g)
ROWS = [
    ("rows-333x296-d8", 333, 296, dict(d=8, hidden=8), torch.bfloat16, 1, False),
    ("rows-130x512-d16-fp32", 130, 512, dict(d=16, hidden=16), torch.float32, 1, False),
    ("rows-200x384-d8-rho5", 200, 384, dict(d=8, hidden=8, protect_num=1, protect_den=20), torch.bfloat16, 1, True),
    ("rows-stack2-96x640-d16", 96, 640, dict(d=16, hidden=16), torch.bfloat16, 2, False),
    ("rows-64x256-d8-identity", 64, 256, dict(d=8, kind=bsq.DEC_IDENTITY, hidden=0, protect_num=1,
                                               protect_den=8), torch.bfloat16, 1, False),
    ("rows-e4m3-200x512-d8", 200, 512, dict(d=8, hidden=8, protect_format=bsq.PROT_E4M3), torch.bfloat16, 1, False),
    ("rows-e5m2-res1-96x640-d16", 96, 640, dict(d=16, hidden=16, kind=bsq.DEC_MLP_RES1,
                                                 protect_format=bsq.PROT_E5M2), torch.bfloat16, 1, False),
]


def _make_rows(name, d_out, d_in, kw, dtype, n_mats, with_g, gpu, seed=21):
    cfg = bsq.Config(protect_axis=1, **kw)
    decs = decoders(cfg, seed)
    k = cfg.k(d_out)
    W = row_weight(d_out, d_in, seed, k, dtype, n_mats)
    g = None
    if with_g:
        g = torch.rand((n_mats, d_out) if n_mats > 1 else (d_out,),
                       generator=torch.Generator().manual_seed(seed)) + 0.5
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer = bsq.bsq_encode(cfg, codec, W.to(gpu), g=None if g is None else g.to(gpu))
    torch.cuda.synchronize()
    oc = ocfg(cfg)
    tabs = oracle.decoder_table(oc, decs)
    Wf = oracle.to_f32(W)
    encs = []
    for m in range(n_mats):
        gm = None if g is None else (g[m] if n_mats > 1 else g).numpy()
        encs.append(oracle.encode(oc, decs, Wf[m] if n_mats > 1 else Wf, g=gm, tables=tabs))
    return cfg, decs, codec, layer, W, encs, tabs


@pytest.mark.parametrize("case", ROWS, ids=[c[0] for c in ROWS])
def test_row_protected_encode_decode_bit_exact(case, gpu):
    say(f"case {case[0]}")
    cfg, decs, codec, layer, W, encs, tabs = _make_rows(*case, gpu)
    oc = ocfg(cfg)
    n_mats = case[5]
    for m, enc in enumerate(encs):
        assert_rows_layer_equal(layer.mat(m), enc, cfg)
        if not case[6]:
            # with no statistic the planted rows are the protected set
            np.testing.assert_array_equal(enc.idx, planted_rows(case[1], cfg.k(case[1]), 21 + m))
    w32 = bsq.bsq_decode(cfg, codec, layer, dtype=torch.float32)
    w16 = bsq.bsq_decode(cfg, codec, layer, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    for m, enc in enumerate(encs):
        ref = oracle.decode(oc, decs, enc, tables=tabs)
        got = (w32[m] if n_mats > 1 else w32).cpu().numpy()
        np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32), err_msg=f"decode fp32 m={m}")
        got16 = (w16[m] if n_mats > 1 else w16).float().cpu().numpy()
        want16 = torch.from_numpy(ref).to(torch.bfloat16).float().numpy()
        np.testing.assert_array_equal(got16.view(np.uint32), want16.view(np.uint32), err_msg=f"decode bf16 m={m}")


@pytest.mark.parametrize("case", ROWS, ids=[c[0] for c in ROWS])
@pytest.mark.parametrize("with_lora", [False, True], ids=["nolora", "lora"])
def test_row_protected_gemv(case, with_lora, gpu):
    say(f"case {case[0]} lora={with_lora}")
    cfg, decs, codec, layer, W, encs, tabs = _make_rows(*case, gpu)
    oc = ocfg(cfg)
    name, d_out, d_in, _, dtype, n_mats, _ = case
    x = synth.activation(d_in, seed=5, dtype=dtype)
    xf = oracle.to_f32(x)
    for m, enc in enumerate(encs):
        lora = synth.lora(d_out, d_in, 16 if m == 0 else 5, seed=9 + m) if with_lora else None
        lora_dev = None if lora is None else (lora[0].to(gpu), lora[1].to(gpu))
        lref = None if lora is None else (oracle.to_f32(lora[0]), oracle.to_f32(lora[1]))
        w_hat = oracle.decode(oc, decs, enc, tables=tabs)
        y_ref = oracle.dense_product(w_hat, xf, lref)
        for ydt in (torch.float32, torch.bfloat16):
            y = bsq.bsq_gemv(cfg, codec, layer.mat(m), x.to(gpu), loras=lora_dev, y_dtype=ydt)
            torch.cuda.synchronize()
            check_product(y.float().cpu().numpy(), y_ref, gemv_kind(dtype), cfg, enc, tabs, w_hat, xf, lref,
                          f"gemv m={m} y={ydt}", ydt)


@pytest.mark.parametrize("d", [8, 16])
def test_row_protected_grouped_gemv(d, gpu):
    """q/k/v-like group with different d_out (so different k) sharing x."""
    cfg = bsq.Config(d=d, hidden=d, protect_axis=1)
    decs = decoders(cfg, 4)
    oc = ocfg(cfg)
    tabs = oracle.decoder_table(oc, decs)
    d_in = 512
    shapes = [256, 64, 64]
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layers, encs, loras = [], [], []
    for i, d_out in enumerate(shapes):
        W = row_weight(d_out, d_in, 40 + i, cfg.k(d_out), torch.bfloat16)
        layers.append(bsq.bsq_encode(cfg, codec, W.to(gpu)))
        encs.append(oracle.encode(oc, decs, oracle.to_f32(W), tables=tabs))
        loras.append(synth.lora(d_out, d_in, 16, seed=50 + i))
    torch.cuda.synchronize()
    x = synth.activation(d_in, seed=8)
    ys = bsq.bsq_gemv(cfg, [codec] * 3, layers, x.to(gpu), loras=[(a.to(gpu), b.to(gpu)) for a, b in loras],
                      y_dtype=torch.float32)
    torch.cuda.synchronize()
    xf = oracle.to_f32(x)
    for i, enc in enumerate(encs):
        assert_rows_layer_equal(layers[i], enc, cfg)
        lref = (oracle.to_f32(loras[i][0]), oracle.to_f32(loras[i][1]))
        w_hat = oracle.decode(oc, decs, enc, tables=tabs)
        check_product(ys[i].cpu().numpy(), oracle.dense_product(w_hat, xf, lref), "gemv", cfg, enc, tabs, w_hat, xf,
                      lref, f"group member {i}", torch.float32)


GEMM_ROWS = [ROWS[0], ROWS[1], ROWS[2], ROWS[5], ROWS[6]]


@pytest.mark.parametrize("case", GEMM_ROWS, ids=[c[0] for c in GEMM_ROWS])
@pytest.mark.parametrize("M", [1, 5, 16, 64, 100])
def test_row_protected_gemm(case, M, gpu):
    say(f"case {case[0]} M={M}")
    cfg, decs, codec, layer, W, encs, tabs = _make_rows(*case, gpu)
    oc = ocfg(cfg)
    name, d_out, d_in = case[:3]
    X = synth.activation(d_in, seed=6, dtype=torch.bfloat16, batch=M)
    lora = synth.lora(d_out, d_in, 16, seed=3)
    Y = bsq.bsq_gemm(cfg, codec, layer, X.to(gpu), lora=(lora[0].to(gpu), lora[1].to(gpu)), y_dtype=torch.float32)
    Yb = bsq.bsq_gemm(cfg, codec, layer, X.to(gpu), y_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    Xf = oracle.to_f32(X)
    w_hat = oracle.decode(oc, decs, encs[0], tables=tabs)
    lref = (oracle.to_f32(lora[0]), oracle.to_f32(lora[1]))
    check_product(Y.cpu().numpy(), oracle.dense_product(w_hat, Xf, lref), "gemm", cfg, encs[0], tabs, w_hat, Xf,
                  lref, "gemm fp32 out", torch.float32)
    check_product(Yb.float().cpu().numpy(), oracle.dense_product(w_hat, Xf), "gemm", cfg, encs[0], tabs, w_hat, Xf,
                  None, "gemm bf16 out", torch.bfloat16)


@pytest.mark.parametrize("axis", [0, 1], ids=["cols", "rows"])
@pytest.mark.parametrize("d,dtype", [(8, torch.bfloat16), (16, torch.float32)])
def test_encode_with_given_set(axis, d, dtype, gpu):
    cfg = bsq.Config(d=d, hidden=d, protect_axis=axis, protect_num=1, protect_den=16)
    decs = decoders(cfg, 12)
    oc = ocfg(cfg)
    d_out, d_in = 150, 512
    W, _ = synth.weight(d_out, d_in, 33, dtype=dtype)
    k = cfg.k(d_out if axis == 1 else d_in)
    n = d_out if axis == 1 else d_in
    idx = np.sort(np.random.default_rng(2).choice(n, size=k, replace=False)).astype(np.int32)
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer = bsq.bsq_encode_with_set(cfg, codec, W.to(gpu), torch.from_numpy(idx))
    torch.cuda.synchronize()
    enc = oracle.encode_set(oc, decs, oracle.to_f32(W), idx)
    if axis == 1:
        assert_rows_layer_equal(layer, enc, cfg)
    else:
        from test_gpu_parity import assert_layer_equal
        assert_layer_equal(layer, enc, cfg)
    w32 = bsq.bsq_decode(cfg, codec, layer)
    torch.cuda.synchronize()
    ref = oracle.decode(oc, decs, enc)
    np.testing.assert_array_equal(w32.cpu().numpy().view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("axis", [0, 1], ids=["cols", "rows"])
def test_encode_with_invalid_set_flags_error(axis, gpu):
    """A set that is not strictly ascending, or leaves the axis, sets bit 2 of
    the error word (the kernels skip such entries; no access leaves its
    buffer)."""
    cfg = bsq.Config(d=8, hidden=8, protect_axis=axis, protect_num=1, protect_den=32)
    decs = decoders(cfg, 1)
    W, _ = synth.weight(64, 256, 3)
    k = cfg.k(64 if axis == 1 else 256)
    assert k >= 2
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    for bad in ([1, 1], [3, 2], [0, 1 << 20], [-1, 4]):
        idx = torch.tensor((bad + list(range(10, 10 + k)))[:k], dtype=torch.int32)
        err = torch.zeros(1, dtype=torch.int32, device=gpu)
        bsq.bsq_encode_with_set(cfg, codec, W.to(gpu), idx, err=err)
        torch.cuda.synchronize()
        assert int(err.item()) & 2, f"set {idx.tolist()} not flagged"


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("with_g", [False, True], ids=["no-g", "g"])
def test_coupled_select_matches_oracle(dtype, with_g, gpu):
    d_model, d_ffn = 256, 1000
    Wg, _ = synth.weight(d_ffn, d_model, 61, dtype=dtype)
    Wu, _ = synth.weight(d_ffn, d_model, 62, dtype=dtype)
    Wd, _ = synth.weight(d_model, d_ffn, 63, dtype=dtype)
    gs = [None] * 3
    if with_g:
        gs = [torch.randn(d_ffn, generator=torch.Generator().manual_seed(70 + i)) for i in range(3)]
    cfg = bsq.Config(d=8, hidden=8)
    k = cfg.k(d_ffn)
    idx, scores = bsq.bsq_coupled_select(cfg, Wg.to(gpu), Wu.to(gpu), Wd.to(gpu),
                                         *[None if g is None else g.to(gpu) for g in gs], with_scores=True)
    torch.cuda.synchronize()
    ref_idx, ref_s = oracle.coupled_select(oracle.to_f32(Wg), oracle.to_f32(Wu), oracle.to_f32(Wd), k,
                                           *[None if g is None else g.numpy() for g in gs])
    np.testing.assert_array_equal(scores.cpu().numpy().view(np.uint64), ref_s.view(np.uint64))
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)


def test_coupled_mlp_protection_end_to_end(gpu):
    """The coupled set applied as the paper's MLP scheme: rows of gate and up
    (axis 1) and columns of down (axis 0), encoded with the given set, and the
    three products against the oracle."""
    d_model, d_ffn = 256, 768
    Wg, _ = synth.weight(d_ffn, d_model, 81)
    Wu, _ = synth.weight(d_ffn, d_model, 82)
    Wd, _ = synth.weight(d_model, d_ffn, 83)
    base = dict(d=8, hidden=8)
    rows_cfg, cols_cfg = bsq.Config(protect_axis=1, **base), bsq.Config(protect_axis=0, **base)
    decs = decoders(rows_cfg, 5)
    idx = bsq.bsq_coupled_select(rows_cfg, Wg.to(gpu), Wu.to(gpu), Wd.to(gpu))
    codec_r = bsq.bsq_codec_prepare(rows_cfg, decs, device=gpu)
    codec_c = bsq.bsq_codec_prepare(cols_cfg, decs, device=gpu)
    Lg = bsq.bsq_encode_with_set(rows_cfg, codec_r, Wg.to(gpu), idx)
    Lu = bsq.bsq_encode_with_set(rows_cfg, codec_r, Wu.to(gpu), idx)
    Ld = bsq.bsq_encode_with_set(cols_cfg, codec_c, Wd.to(gpu), idx)
    x = synth.activation(d_model, seed=1)
    yg, yu = bsq.bsq_gemv(rows_cfg, [codec_r] * 2, [Lg, Lu], x.to(gpu), y_dtype=torch.float32)
    h = synth.activation(d_ffn, seed=2)
    yd = bsq.bsq_gemv(cols_cfg, codec_c, Ld, h.to(gpu), y_dtype=torch.float32)
    torch.cuda.synchronize()
    ref_idx, _ = oracle.coupled_select(oracle.to_f32(Wg), oracle.to_f32(Wu), oracle.to_f32(Wd), rows_cfg.k(d_ffn))
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
    for W, L, y, v, oc_axis in ((Wg, Lg, yg, x, 1), (Wu, Lu, yu, x, 1), (Wd, Ld, yd, h, 0)):
        cfg = rows_cfg if oc_axis == 1 else cols_cfg
        oc = ocfg(cfg)
        enc = oracle.encode_set(oc, decs, oracle.to_f32(W), ref_idx)
        if oc_axis == 1:
            assert_rows_layer_equal(L, enc, cfg)
        tabs = oracle.decoder_table(oc, decs)
        w_hat = oracle.decode(oc, decs, enc, tables=tabs)
        vf = oracle.to_f32(v)
        check_product(y.cpu().numpy(), oracle.dense_product(w_hat, vf), "gemv", cfg, enc, tabs, w_hat, vf, None,
                      f"axis {oc_axis} product", torch.float32)


@pytest.mark.parametrize("d", [8, 16])
def test_row_axis_degenerate_cases(d, gpu):
    """Row axis with no protected rows (rho = 0, and a matrix too small for
    k > 0 is impossible: k = ceil(rho d_out) >= 1 for d_out >= 1), an empty
    batch, and every row protected (rho = 1: no row is BSQ-coded)."""
    decs = None
    for num, den in ((0, 1), (1, 1)):
        cfg = bsq.Config(d=d, hidden=d, protect_axis=1, protect_num=num, protect_den=den)
        decs = decoders(cfg, 2)
        oc = ocfg(cfg)
        W, _ = synth.weight(70, 256, 17)
        codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
        layer = bsq.bsq_encode(cfg, codec, W.to(gpu))
        tabs = oracle.decoder_table(oc, decs)
        enc = oracle.encode(oc, decs, oracle.to_f32(W), tables=tabs)
        torch.cuda.synchronize()
        assert_rows_layer_equal(layer, enc, cfg)
        w_hat = oracle.decode(oc, decs, enc, tables=tabs)
        got = bsq.bsq_decode(cfg, codec, layer)
        x = synth.activation(256, seed=3)
        y = bsq.bsq_gemv(cfg, codec, layer, x.to(gpu), y_dtype=torch.float32)
        X = synth.activation(256, seed=4, batch=7)
        Y = bsq.bsq_gemm(cfg, codec, layer, X.to(gpu), y_dtype=torch.float32)
        Y0 = bsq.bsq_gemm(cfg, codec, layer, X[:0].to(gpu), y_dtype=torch.float32)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(got.cpu().numpy().view(np.uint32), w_hat.view(np.uint32))
        xf, Xf = oracle.to_f32(x), oracle.to_f32(X)
        check_product(y.cpu().numpy(), oracle.dense_product(w_hat, xf), "gemv", cfg, enc, tabs, w_hat, xf, None,
                      f"gemv rho={num}/{den}", torch.float32)
        check_product(Y.cpu().numpy(), oracle.dense_product(w_hat, Xf), "gemm", cfg, enc, tabs, w_hat, Xf, None,
                      f"gemm rho={num}/{den}", torch.float32)
        assert Y0.shape == (0, 70)
        if num == den:
            # every row protected: the planes hold only zeros
            for s in range(cfg.stages):
                assert int(layer.codes[s].abs().sum()) == 0 and int(layer.gains[s].abs().sum()) == 0
