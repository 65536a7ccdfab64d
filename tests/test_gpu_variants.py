"""The FP8 protected payloads on the GPU at the values where a conversion can
go wrong: a protected slice whose scale is exactly 1 (its largest magnitude is
the format's largest finite value) and whose entries are every non-negative
finite value of the format, every midpoint between neighbours (ties to the
even code), points a quarter step off, values below the smallest subnormal
and signed zeros, each with both signs. The stored bytes must equal the
oracle's (found there by trying every code) and torch's own float8 cast, and
the decoded slice must be torch's reading of those bytes, on the input-column
axis and on the output-row axis. A second test writes all 256 bytes, NaN and
infinity codes included, into a layer's payload and decodes them.

The linear encoder z = E r (Section III-C) and code lengths b other than the
chunk length d: encode, stage-parallel and sequential decode bit-exact, GEMV
(bf16 and fp32 x) and GEMM against the oracle with LoRA.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_08643_amd as bsq
import synth
from parity_bounds import say
from test_gpu_parity import OFMT, OKIND, check_product, decoders, gemv_kind

pytestmark = pytest.mark.gpu

TORCH_FP8 = {bsq.PROT_E4M3: torch.float8_e4m3fn, bsq.PROT_E5M2: torch.float8_e5m2}
FMAX = {bsq.PROT_E4M3: 448.0, bsq.PROT_E5M2: 57344.0}


def crafted_values(fmt):
    raw = torch.arange(128, dtype=torch.int32).to(torch.uint8)
    vals = raw.view(TORCH_FP8[fmt]).to(torch.float64).numpy()
    fin = vals[np.isfinite(vals) & (vals <= FMAX[fmt])]
    mids = (fin[:-1] + fin[1:]) / 2
    quarter = fin[:-1] + (fin[1:] - fin[:-1]) / 4
    tiny = fin[1] * np.array([0.25, 0.5, 0.75])
    v = np.concatenate([fin, mids, quarter, tiny]).astype(np.float32)
    v = np.concatenate([v, -v])
    assert np.abs(v).max() == FMAX[fmt]
    return v


def ocfg(cfg):
    return oracle.Config(d=cfg.d, b=cfg.d, stages=cfg.stages, kind=OKIND[cfg.kind], hidden=cfg.hidden,
                         protect_num=cfg.protect_num, protect_den=cfg.protect_den, protect_axis=cfg.protect_axis,
                         protect_format=OFMT[cfg.protect_format])


@pytest.mark.parametrize("fmt", [bsq.PROT_E4M3, bsq.PROT_E5M2], ids=["e4m3", "e5m2"])
@pytest.mark.parametrize("axis", [0, 1], ids=["cols", "rows"])
@pytest.mark.parametrize("d", [8, 16])
def test_fp8_payload_at_every_code_and_tie(fmt, axis, d, gpu):
    vals = crafted_values(fmt)
    n = len(vals)
    slice_len = (n + 63) // 64 * 64
    r = np.random.default_rng(5 + fmt + 2 * axis)
    if axis == 0:
        d_out, d_in, j0 = slice_len, 256, 37
        W = r.normal(0, 0.02, (d_out, d_in)).astype(np.float32)
        W[:, j0] = 0.0
        W[:n, j0] = vals
    else:
        d_out, d_in, j0 = 96, slice_len, 41
        W = r.normal(0, 0.02, (d_out, d_in)).astype(np.float32)
        W[j0, :] = 0.0
        W[j0, :n] = vals
    cfg = bsq.Config(d=d, hidden=d, protect_axis=axis, protect_format=fmt, protect_num=1,
                     protect_den=(d_in if axis == 0 else d_out))     # k = 1: the planted slice
    say(f"fp8 crafted slice fmt={fmt} axis={axis} d={d} n={n}")
    decs = decoders(cfg, seed=13)
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer = bsq.bsq_encode(cfg, codec, torch.from_numpy(W).to(gpu))
    w_hat = bsq.bsq_decode(cfg, codec, layer, dtype=torch.float32)
    torch.cuda.synchronize()
    oc = ocfg(cfg)
    enc = oracle.encode(oc, decs, W)
    assert list(enc.idx) == [j0]
    assert float(enc.scale[0]) == 1.0
    got_idx = layer.idx.cpu().numpy()
    assert list(got_idx) == [j0]
    assert float(layer.scale.cpu()[0]) == 1.0
    q = layer.q8.cpu().numpy()
    stored = (q[:n, 0] if axis == 0 else q[0, :n]).view(np.uint8)
    want_oracle = (enc.q8[:n, 0] if axis == 0 else enc.q8[0, :n]).view(np.uint8)
    want_torch = torch.from_numpy(vals).to(TORCH_FP8[fmt]).view(torch.uint8).numpy()
    np.testing.assert_array_equal(stored, want_oracle, err_msg="bytes vs oracle")
    np.testing.assert_array_equal(stored, want_torch, err_msg="bytes vs torch")
    wh = w_hat.cpu().numpy()
    dec = wh[:n, j0] if axis == 0 else wh[j0, :n]
    want = torch.from_numpy(stored.copy()).view(TORCH_FP8[fmt]).to(torch.float32).numpy()
    np.testing.assert_array_equal(dec.view(np.uint32), want.view(np.uint32), err_msg="decoded slice")
    np.testing.assert_array_equal(wh.view(np.uint32), oracle.decode(oc, decs, enc).view(np.uint32))
    # the product over the crafted slice
    x = synth.activation(d_in, seed=8, dtype=torch.bfloat16)
    y = bsq.bsq_gemv(cfg, codec, layer, x.to(gpu), y_dtype=torch.float32)
    torch.cuda.synchronize()
    tabs = oracle.decoder_table(oc, decs)
    w_ref = oracle.decode(oc, decs, enc, tables=tabs)
    xf = oracle.to_f32(x)
    check_product(y.cpu().numpy(), oracle.dense_product(w_ref, xf), gemv_kind(torch.bfloat16), cfg, enc, tabs,
                  w_ref, xf, None, "gemv over the crafted slice", torch.float32)


@pytest.mark.parametrize("fmt", [bsq.PROT_E4M3, bsq.PROT_E5M2], ids=["e4m3", "e5m2"])
@pytest.mark.parametrize("d", [8, 16])
def test_every_stored_byte_decodes_to_its_value(fmt, d, gpu):
    """All 256 bytes, NaN and infinity codes included, written into the
    payload of an encoded layer (scale 1): the decoded protected column is
    torch's float8 reading of each byte."""
    say(f"every byte fmt={fmt} d={d}")
    d_out, d_in = 256, 128
    cfg = bsq.Config(d=d, hidden=d, protect_format=fmt, protect_num=1, protect_den=d_in)
    W = synth.weight(d_out, d_in, seed=3, k_outliers=1, dtype=torch.float32)[0]
    codec = bsq.bsq_codec_prepare(cfg, decoders(cfg, seed=2), device=gpu)
    layer = bsq.bsq_encode(cfg, codec, W.to(gpu))
    torch.cuda.synchronize()
    j0 = int(layer.idx.cpu()[0])
    layer.q8[:, 0] = torch.arange(256, device=gpu, dtype=torch.int32).to(torch.uint8).view(torch.int8)
    layer.scale.fill_(1.0)
    w_hat = bsq.bsq_decode(cfg, codec, layer, dtype=torch.float32)
    torch.cuda.synchronize()
    got = w_hat[:, j0].cpu().numpy()
    want = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(TORCH_FP8[fmt]).to(torch.float32).numpy()
    nan = np.isnan(want)
    np.testing.assert_array_equal(np.isnan(got), nan)
    np.testing.assert_array_equal(got[~nan].view(np.uint32), want[~nan].view(np.uint32))


# ---------------------------------------------------------------- linear encoder, b != d
from test_gpu_parity import assert_layer_equal  # noqa: E402

# (name, d_out, d_in, d, b, decoder kind, hidden, W dtype)
ENC_CASES = [
    ("enc-d8-b16", 96, 512, 8, 16, bsq.DEC_MLP, 16, torch.bfloat16),
    ("enc-d16-b8", 80, 640, 16, 8, bsq.DEC_MLP, 8, torch.bfloat16),
    ("enc-d8-b8", 120, 512, 8, 8, bsq.DEC_MLP, 8, torch.bfloat16),
    ("enc-d16-b16-linear", 64, 512, 16, 16, bsq.DEC_LINEAR, 16, torch.float32),
    ("enc-d8-b16-res1-e4m3", 70, 384, 8, 16, bsq.DEC_MLP_RES1, 12, torch.bfloat16),
]


def _make_enc(case, gpu, seed=41):
    name, d_out, d_in, d, b, kind, h, dtype = case
    fmt = bsq.PROT_E4M3 if "e4m3" in name else bsq.PROT_INT8
    cfg = bsq.Config(d=d, codebook_bits=b, kind=kind, hidden=h, encoder=bsq.ENC_LINEAR, protect_format=fmt)
    decs = synth.decoder_params(kind, d, b, h, cfg.stages, seed=seed, encoder=True)
    W, _ = synth.weight(d_out, d_in, seed, k_outliers=cfg.k(d_in), dtype=dtype, device="cpu")
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer = bsq.bsq_encode(cfg, codec, W.to(gpu))
    torch.cuda.synchronize()
    oc = oracle.Config(d=d, b=b, stages=cfg.stages, kind=OKIND[kind], hidden=h, protect_format=OFMT[fmt],
                       encoder=oracle.ENC_LINEAR)
    tabs = oracle.decoder_table(oc, decs)
    enc = oracle.encode(oc, decs, oracle.to_f32(W), tables=tabs)
    return cfg, oc, decs, codec, layer, W, enc, tabs


@pytest.mark.parametrize("case", ENC_CASES, ids=[c[0] for c in ENC_CASES])
def test_linear_encoder_encode_decode_bit_exact(case, gpu):
    say(f"encoder case {case[0]}")
    cfg, oc, decs, codec, layer, W, enc, tabs = _make_enc(case, gpu)
    assert layer.codes[0].dtype == (torch.uint8 if cfg.b == 8 else torch.int16)
    assert_layer_equal(layer, enc, cfg)
    w32 = bsq.bsq_decode(cfg, codec, layer, dtype=torch.float32)
    w16 = bsq.bsq_decode(cfg, codec, layer, dtype=torch.bfloat16)
    seq = torch.full_like(w32, float("nan"))
    for s in range(cfg.stages):
        bsq.bsq_decode_stage(cfg, codec, layer, s, s > 0, seq)
    torch.cuda.synchronize()
    ref = oracle.decode(oc, decs, enc, tables=tabs)
    np.testing.assert_array_equal(w32.cpu().numpy().view(np.uint32), ref.view(np.uint32))
    assert torch.equal(w16.cpu().view(torch.int16), torch.from_numpy(ref).to(torch.bfloat16).view(torch.int16))
    assert torch.equal(seq.view(torch.int32), w32.view(torch.int32))


@pytest.mark.parametrize("case", ENC_CASES, ids=[c[0] for c in ENC_CASES])
def test_linear_encoder_products_match_oracle(case, gpu):
    say(f"encoder case {case[0]} products")
    cfg, oc, decs, codec, layer, W, enc, tabs = _make_enc(case, gpu)
    name, d_out, d_in = case[:3]
    w_hat = oracle.decode(oc, decs, enc, tables=tabs)
    A, Bm = synth.lora(d_out, d_in, 16, seed=43)
    lref = (oracle.to_f32(A), oracle.to_f32(Bm))
    fp32_path = cfg.b != cfg.d
    for xdt in (torch.bfloat16, torch.float32):
        x = synth.activation(d_in, seed=44, dtype=xdt)
        y = bsq.bsq_gemv(cfg, codec, layer, x.to(gpu), loras=(A.to(gpu), Bm.to(gpu)), y_dtype=torch.float32)
        torch.cuda.synchronize()
        xf = oracle.to_f32(x)
        kind = "fp32" if (fp32_path or xdt == torch.float32) else "gemv"
        check_product(y.cpu().numpy(), oracle.dense_product(w_hat, xf, lref), kind, cfg, enc, tabs, w_hat, xf, lref,
                      f"gemv x={xdt}", torch.float32)
    for M in (1, 16, 100):
        X = synth.activation(d_in, seed=45, dtype=torch.bfloat16, batch=M)
        Y = bsq.bsq_gemm(cfg, codec, layer, X.to(gpu), lora=(A.to(gpu), Bm.to(gpu)), y_dtype=torch.float32)
        torch.cuda.synchronize()
        Xf = oracle.to_f32(X)
        check_product(Y.cpu().numpy(), oracle.dense_product(w_hat, Xf, lref), "fp32" if fp32_path else "gemm", cfg,
                      enc, tabs, w_hat, Xf, lref, f"gemm M={M}", torch.float32)
