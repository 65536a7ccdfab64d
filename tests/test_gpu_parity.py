"""HIP path vs the CPU oracle, element by element, through the C ABI.

Bar: codes, gains, protected indices, int8 payload, scales and the bitmap
bit-exact; fp32 decode bit-exact (bf16 decode = the oracle's fp32 value
rounded to nearest even); products within 2e-2 relative per output for bf16
activations and 1e-4 for fp32 activations, with an absolute floor per output
derived from the rounding the GPU path does (tests/parity_bounds.py: a
sub-Gaussian bound on the bf16 roundings of the decoded terms, 3.78 u
sqrt(sum t^2), plus fp32 accumulation). Separate checks take the LoRA term
and the int8 protected term out of the product (the difference of two calls
that differ only in that term) and compare each with the oracle's value of
the term, so that a dropped or partly wrong term cannot hide under the floor.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2607_08643_amd as bsq
import synth
from parity_bounds import check_close, product_floor, say, term_bar

pytestmark = pytest.mark.gpu

OKIND = {bsq.DEC_IDENTITY: oracle.KIND_IDENTITY, bsq.DEC_LINEAR: oracle.KIND_LINEAR, bsq.DEC_MLP: oracle.KIND_MLP,
         bsq.DEC_MLP_RES1: oracle.KIND_MLP_RES1}
OFMT = {bsq.PROT_INT8: oracle.FMT_INT8, bsq.PROT_E4M3: oracle.FMT_E4M3, bsq.PROT_E5M2: oracle.FMT_E5M2}


def ocfg(cfg: bsq.Config) -> oracle.Config:
    return oracle.Config(d=cfg.d, b=cfg.d, stages=cfg.stages, kind=OKIND[cfg.kind], hidden=cfg.hidden,
                         protect_num=cfg.protect_num, protect_den=cfg.protect_den,
                         protect_format=OFMT[cfg.protect_format])


def np_codes(L, t):
    a = L.rowmajor(t).contiguous().cpu().numpy()
    return a.view(np.uint16) if a.dtype == np.int16 else a


def np_gains(L, t):
    return L.rowmajor(t).contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def decoders(cfg, seed=7):
    return synth.decoder_params(cfg.kind, cfg.d, cfg.d, cfg.hidden, cfg.stages, seed=seed)


def assert_layer_equal(layer, enc, cfg, m=None):
    L = layer.mat(m) if m is not None else layer
    for s in range(cfg.stages):
        np.testing.assert_array_equal(np_codes(L, L.codes[s]), enc.codes[s], err_msg=f"codes stage {s}")
        np.testing.assert_array_equal(np_gains(L, L.gains[s]), enc.gains[s], err_msg=f"gains stage {s}")
        # padding rows of the last 64-row group hold code 0 and gain +0
        pad = L.row_groups * 64 - L.d_out
        if pad:
            full = L.codes[s].transpose(-3, -2).reshape(L.row_groups * 64, L.pitch)
            assert int(full[L.d_out:].abs().sum()) == 0
    if cfg.k(L.d_in):
        np.testing.assert_array_equal(L.idx.cpu().numpy(), enc.idx, err_msg="protected indices")
        q8 = L.q8.cpu().numpy()
        np.testing.assert_array_equal(q8[:, :enc.q8.shape[1]], enc.q8, err_msg="protected payload")
        assert not q8[:, enc.q8.shape[1]:].any(), "protected payload padding"
        np.testing.assert_array_equal(L.scale.cpu().numpy().view(np.uint32), enc.scale.view(np.uint32),
                                      err_msg="scales")
        # bitmap over the padded columns: exactly the oracle's protected set
        want = np.zeros(L.pitch * cfg.d, dtype=np.uint8)
        want[enc.idx] = 1
        want = np.packbits(want, bitorder="little").view(np.uint32)
        np.testing.assert_array_equal(L.bits.cpu().numpy().view(np.uint32), want, err_msg="protected bitmap")


def gemv_kind(x_dtype):
    """The arithmetic of the GEMV path bsq_gemv takes for this activation
    dtype: fp32 throughout for fp32 x, else bf16 decoded terms."""
    return "fp32" if x_dtype == torch.float32 else "gemv"


def check_product(y, y_ref, kind, cfg, enc, tabs, w_hat, X, lref, what, y_dtype):
    """The product bar: 1e-4 relative for fp32 activations with fp32 output,
    else 2e-2, with the derived floor of the path and the output rounding."""
    rel = 1e-4 if (kind == "fp32" and y_dtype == torch.float32) else 2e-2
    floor = product_floor(kind, cfg.d, enc, tabs, w_hat, X, lref)
    check_close(np.asarray(y, dtype=np.float64), y_ref, rel, what, floor, out_bf16=(y_dtype == torch.bfloat16))


# (name, d_out, d_in, cfg kwargs, dtype, n_mats, with_g)
SMALL = [
    ("tiny-256x256-fp32-d8", 256, 256, dict(d=8, hidden=8, protect_num=0), torch.float32, 1, False),
    ("ragged-333x296-d8", 333, 296, dict(d=8, hidden=8), torch.bfloat16, 1, False),
    ("ragged-77x592-d16", 77, 592, dict(d=16, hidden=16, protect_num=1, protect_den=50), torch.bfloat16, 1, False),
    ("identity-128x512-d8", 128, 512, dict(d=8, kind=bsq.DEC_IDENTITY, hidden=0), torch.bfloat16, 1, False),
    ("linear-64x512-d16-3stage", 64, 512, dict(d=16, kind=bsq.DEC_LINEAR, stages=3), torch.float32, 1, False),
    ("mlp-1stage-200x384-d8", 200, 384, dict(d=8, stages=1, hidden=8), torch.bfloat16, 1, False),
    ("mlp-4stage-50x1024-d8-h16", 50, 1024, dict(d=8, stages=4, hidden=16), torch.bfloat16, 1, False),
    ("mlp-h5-96x320-d16", 96, 320, dict(d=16, hidden=5), torch.bfloat16, 1, False),
    ("stack3-96x1024-d8", 96, 1024, dict(d=8, hidden=8), torch.bfloat16, 3, False),
    ("stack2-40x640-d16-fp32", 40, 640, dict(d=16, hidden=16), torch.float32, 2, False),
    ("g-128x640-d8", 128, 640, dict(d=8, hidden=8), torch.bfloat16, 1, True),
    ("rho25-64x256-d8", 64, 256, dict(d=8, hidden=8, protect_num=1, protect_den=4), torch.bfloat16, 1, False),
    ("mlp-3stage-100x768-d16", 100, 768, dict(d=16, hidden=16, stages=3), torch.bfloat16, 1, False),
    ("stack2-130x1056-d16", 130, 1056, dict(d=16, hidden=16), torch.bfloat16, 2, False),
    # the component ablation's variants: decoder with one residual block, FP8 protected payloads
    ("res1-160x512-d8", 160, 512, dict(d=8, hidden=8, kind=bsq.DEC_MLP_RES1), torch.bfloat16, 1, False),
    ("res1-h12-96x640-d16", 96, 640, dict(d=16, hidden=12, kind=bsq.DEC_MLP_RES1), torch.bfloat16, 1, False),
    ("e4m3-200x512-d8", 200, 512, dict(d=8, hidden=8, protect_format=bsq.PROT_E4M3, protect_num=1, protect_den=32),
     torch.bfloat16, 1, False),
    ("e5m2-77x592-d16", 77, 592, dict(d=16, hidden=16, protect_format=bsq.PROT_E5M2, protect_num=1, protect_den=50),
     torch.bfloat16, 1, False),
    ("res1-e4m3-fp32-64x256-d8", 64, 256, dict(d=8, hidden=8, kind=bsq.DEC_MLP_RES1, protect_format=bsq.PROT_E4M3),
     torch.float32, 1, False),
]


def _make(name, d_out, d_in, kw, dtype, n_mats, with_g, gpu, seed=11):
    cfg = bsq.Config(**kw)
    decs = decoders(cfg, seed)
    k = cfg.k(d_in)
    W, _ = synth.weight(d_out, d_in, seed, k_outliers=k, dtype=dtype, device="cpu", n_mats=n_mats)
    g = None
    if with_g:
        g = torch.rand((n_mats, d_in) if n_mats > 1 else (d_in,), generator=torch.Generator().manual_seed(seed)) + 0.5
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer = bsq.bsq_encode(cfg, codec, W.to(gpu), g=None if g is None else g.to(gpu))
    torch.cuda.synchronize()
    Wf = oracle.to_f32(W)
    oc = ocfg(cfg)
    tabs = oracle.decoder_table(oc, decs)
    encs = []
    for m in range(n_mats):
        Wm = Wf[m] if n_mats > 1 else Wf
        gm = None if g is None else (g[m] if n_mats > 1 else g).numpy()
        encs.append(oracle.encode(oc, decs, Wm, g=gm, tables=tabs))
    return cfg, decs, codec, layer, W, encs, tabs


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_encode_decode_bit_exact(case, gpu):
    say(f"case {case[0]}")
    cfg, decs, codec, layer, W, encs, tabs = _make(*case, gpu)
    oc = ocfg(cfg)
    n_mats = case[5]
    for m, enc in enumerate(encs):
        assert_layer_equal(layer, enc, cfg, m if n_mats > 1 else None)
    w32 = bsq.bsq_decode(cfg, codec, layer, dtype=torch.float32)
    w16 = bsq.bsq_decode(cfg, codec, layer, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    for m, enc in enumerate(encs):
        ref = oracle.decode(oc, decs, enc, tables=tabs)
        got = (w32[m] if n_mats > 1 else w32).cpu().numpy()
        np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))
        got16 = (w16[m] if n_mats > 1 else w16).cpu()
        ref16 = torch.from_numpy(ref).to(torch.bfloat16)
        assert torch.equal(got16.view(torch.int16), ref16.view(torch.int16))


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_sequential_stage_decode_equals_stage_parallel(case, gpu):
    """Decoding the residual stages one launch after the other
    (bsq_decode_stage, accumulating in fp32) gives the bits of the
    stage-parallel decode of eq. parallel_stage_decode (bsq_decode), which
    the oracle's decode pins."""
    say(f"case {case[0]} sequential stages")
    cfg, decs, codec, layer, W, encs, tabs = _make(*case, gpu)
    par = bsq.bsq_decode(cfg, codec, layer, dtype=torch.float32)
    seq = torch.full_like(par, float("nan"))
    for s in range(cfg.stages):
        bsq.bsq_decode_stage(cfg, codec, layer, s, s > 0, seq)
    torch.cuda.synchronize()
    assert torch.equal(seq.view(torch.int32), par.view(torch.int32))


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
@pytest.mark.parametrize("with_lora", [False, True], ids=["nolora", "lora"])
def test_gemv_matches_oracle(case, with_lora, gpu):
    say(f"case {case[0]} lora={with_lora}")
    cfg, decs, codec, layer, W, encs, tabs = _make(*case, gpu)
    oc = ocfg(cfg)
    name, d_out, d_in, _, dtype, n_mats, _ = case
    x = synth.activation(d_in, seed=5, dtype=dtype)
    for m, enc in enumerate(encs):
        lora = synth.lora(d_out, d_in, 16 if m % 2 == 0 else 3, seed=9 + m) if with_lora else None
        lora_dev = None if lora is None else (lora[0].to(gpu), lora[1].to(gpu))
        for ydt in (torch.float32, torch.bfloat16):
            y = bsq.bsq_gemv(cfg, codec, layer.mat(m), x.to(gpu), loras=lora_dev, y_dtype=ydt)
            torch.cuda.synchronize()
            lref = None if lora is None else (oracle.to_f32(lora[0]), oracle.to_f32(lora[1]))
            xf = oracle.to_f32(x)
            w_hat = oracle.decode(oc, decs, enc, tables=tabs)
            y_ref = oracle.dense_product(w_hat, xf, lref)
            check_product(y.float().cpu().numpy(), y_ref, gemv_kind(dtype), cfg, enc, tabs, w_hat, xf, lref,
                          f"gemv m={m} y={ydt}", ydt)


@pytest.mark.parametrize("scale", [2.0 ** 24, 2.0 ** -24], ids=["huge", "tiny"])
def test_gemv_d16_activation_range(scale, gpu):
    """The d = 16 decoder path folds W2 into x and keeps the result in fp16
    with a power-of-two scale per chunk: activations far outside fp16's range
    must still give the oracle's product within tolerance."""
    case = ("range-192x1024-d16", 192, 1024, dict(d=16, hidden=16), torch.bfloat16, 1, False)
    say(f"case {case[0]} x scale {scale}")
    cfg, decs, codec, layer, W, encs, tabs = _make(*case, gpu)
    oc = ocfg(cfg)
    x = (synth.activation(1024, seed=5, dtype=torch.float32) * scale).to(torch.bfloat16)
    y = bsq.bsq_gemv(cfg, codec, layer, x.to(gpu), y_dtype=torch.float32)
    torch.cuda.synchronize()
    xf = oracle.to_f32(x)
    w_hat = oracle.decode(oc, decs, encs[0], tables=tabs)
    y_ref = oracle.dense_product(w_hat, xf, None)
    check_product(y.float().cpu().numpy(), y_ref, "gemv", cfg, encs[0], tabs, w_hat, xf, None, f"gemv x*{scale}",
                  torch.float32)


# Long rows: the K steps of a tile are split over several blocks (ragged
# split sizes, a partial last step) and summed in split order by a second launch.
SPLITK = [
    ("splitk-200x2600-d8", 200, 2600, dict(d=8, hidden=8), torch.bfloat16, 1, False),
    ("splitk-130x2608-d16", 130, 2608, dict(d=16, hidden=16), torch.bfloat16, 1, False),
]
# Stage counts 1 and 3 at d = 8 and 3 and 4 at d = 16, so that every kernel
# shape of the GEMM (token tile x row block x stages) runs at some M.
GEMM_STAGES = [
    ("mlp-3stage-70x1000-d8", 70, 1000, dict(d=8, hidden=8, stages=3), torch.bfloat16, 1, False),
    ("mlp-4stage-90x640-d16", 90, 640, dict(d=16, hidden=16, stages=4), torch.bfloat16, 1, False),
]
GEMM_CASES = ([SMALL[1], SMALL[2], SMALL[3], SMALL[5], SMALL[6], SMALL[11], SMALL[12], SMALL[14], SMALL[15], SMALL[16],
               SMALL[17]] + GEMM_STAGES + SPLITK)


@pytest.mark.parametrize("case", GEMM_CASES, ids=[c[0] for c in GEMM_CASES])
@pytest.mark.parametrize("M", [1, 5, 16, 20, 40, 64, 100, 256])
def test_gemm_matches_oracle(case, M, gpu):
    say(f"case {case[0]} M={M}")
    cfg, decs, codec, layer, W, encs, tabs = _make(*case, gpu)
    oc = ocfg(cfg)
    name, d_out, d_in, _, dtype, n_mats, _ = case
    X = synth.activation(d_in, seed=6, dtype=torch.bfloat16, batch=M)
    lora = synth.lora(d_out, d_in, 16, seed=3)
    Y = bsq.bsq_gemm(cfg, codec, layer, X.to(gpu), lora=(lora[0].to(gpu), lora[1].to(gpu)), y_dtype=torch.float32)
    Yb = bsq.bsq_gemm(cfg, codec, layer, X.to(gpu), y_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    Xf = oracle.to_f32(X)
    w_hat = oracle.decode(oc, decs, encs[0], tables=tabs)
    lref = (oracle.to_f32(lora[0]), oracle.to_f32(lora[1]))
    Y_ref = oracle.dense_product(w_hat, Xf, lref)
    check_product(Y.cpu().numpy(), Y_ref, "gemm", cfg, encs[0], tabs, w_hat, Xf, lref, "gemm fp32 out",
                  torch.float32)
    Yb_ref = oracle.dense_product(w_hat, Xf)
    check_product(Yb.float().cpu().numpy(), Yb_ref, "gemm", cfg, encs[0], tabs, w_hat, Xf, None, "gemm bf16 out",
                  torch.bfloat16)


@pytest.mark.parametrize("d", [8, 16])
def test_gemm_workspace_reuse(d, gpu):
    """One workspace for calls of different token counts: each result equals
    the one from a fresh workspace, and the 256-byte header is left as it
    was."""
    say(f"gemm workspace reuse d={d}")
    cfg = bsq.Config(d=d, hidden=d)
    decs = decoders(cfg, seed=d + 3)
    d_out, d_in = 1000, 2048
    W, _ = synth.weight(d_out, d_in, seed=31, k_outliers=cfg.k(d_in), device=gpu)
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer = bsq.bsq_encode(cfg, codec, W)
    Ms = [16, 256, 5, 100, 16, 64, 256]
    need = max(bsq.bsq_workspace_bytes(cfg, bsq.OP_GEMM, 1, d_out, d_in, M) for M in Ms)
    raw = torch.zeros(need + 256, dtype=torch.uint8, device=gpu)
    ws = raw[(-raw.data_ptr()) % 256:][:need]
    A, Bm = synth.lora(d_out, d_in, 16, seed=4, device=gpu)
    for i, M in enumerate(Ms):
        X = synth.activation(d_in, seed=40 + i, device=gpu, batch=M)
        Y = bsq.bsq_gemm(cfg, codec, layer, X, lora=(A, Bm), y_dtype=torch.float32, ws=ws)
        Y_fresh = bsq.bsq_gemm(cfg, codec, layer, X, lora=(A, Bm), y_dtype=torch.float32)
        torch.cuda.synchronize()
        assert torch.equal(Y, Y_fresh), f"M={M}: shared-workspace result differs"
        assert int(torch.count_nonzero(ws[:256])) == 0, f"M={M}: header written"


@pytest.mark.parametrize("d", [8, 16])
def test_grouped_gemv_three_categories(d, gpu):
    """q/k/v-like group: one x, three matrices of different heights, three codecs."""
    say(f"grouped qkv-like 320/96/96 x 1024 d={d}")
    d_in = 1024
    outs = [320, 96, 96]
    cfg = bsq.Config(d=d, hidden=d)
    oc = ocfg(cfg)
    x = synth.activation(d_in, seed=1)
    codecs, layers, encs, decs_all, loras = [], [], [], [], []
    for i, d_out in enumerate(outs):
        decs = decoders(cfg, seed=100 + i)
        W, _ = synth.weight(d_out, d_in, seed=200 + i, k_outliers=cfg.k(d_in))
        codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
        codecs.append(codec)
        layers.append(bsq.bsq_encode(cfg, codec, W.to(gpu)))
        encs.append(oracle.encode(oc, decs, oracle.to_f32(W)))
        decs_all.append(decs)
        loras.append(synth.lora(d_out, d_in, 16, seed=300 + i))
    ys = bsq.bsq_gemv(cfg, codecs, layers, x.to(gpu), loras=[(a.to(gpu), b.to(gpu)) for a, b in loras],
                      y_dtype=torch.float32)
    torch.cuda.synchronize()
    for i in range(3):
        assert_layer_equal(layers[i], encs[i], cfg)
        lref = (oracle.to_f32(loras[i][0]), oracle.to_f32(loras[i][1]))
        tabs = oracle.decoder_table(oc, decs_all[i])
        w_hat = oracle.decode(oc, decs_all[i], encs[i], tables=tabs)
        y_ref = oracle.dense_product(w_hat, oracle.to_f32(x), lref)
        check_product(ys[i].cpu().numpy(), y_ref, "gemv", cfg, encs[i], tabs, w_hat, oracle.to_f32(x), lref,
                      f"group member {i}", torch.float32)


# ---------------------------------------------------------------- edge cases
def _encode_both(cfg, W_cpu, gpu, seed=3):
    decs = decoders(cfg, seed)
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer = bsq.bsq_encode(cfg, codec, W_cpu.to(gpu))
    torch.cuda.synchronize()
    enc = oracle.encode(ocfg(cfg), decs, oracle.to_f32(W_cpu))
    return decs, codec, layer, enc


@pytest.mark.parametrize("d", [8, 16])
def test_edge_values(d, gpu):
    """All-zero rows, constant blocks, -0.0, fp32 subnormals, huge values that
    saturate the fp16 gain, tiny values that underflow it, tied columns."""
    say(f"edge values d={d}")
    cfg = bsq.Config(d=d, hidden=d, protect_num=1, protect_den=16)
    r = np.random.default_rng(1)
    W = r.normal(0, 0.02, (48, 16 * d)).astype(np.float32)
    W[0] = 0.0
    W[1] = -0.0
    W[2] = 0.5
    W[3, : d] = -0.0
    W[4] = np.float32(1e-41) * np.sign(r.normal(size=16 * d))          # subnormal
    W[5] = np.float32(3e38) * np.sign(r.normal(size=16 * d))           # near fp32 max
    W[6] = np.float32(1e6)                                             # gain saturates at 65504
    W[7] = np.float32(1e-9) * r.normal(size=16 * d)                    # gain underflows fp16
    W[:, 5] = W[:, 9]                                                  # tied columns
    W[:, 17] = 0.0
    Wt = torch.from_numpy(W)
    decs, codec, layer, enc = _encode_both(cfg, Wt, gpu)
    assert_layer_equal(layer, enc, cfg)
    w32 = bsq.bsq_decode(cfg, codec, layer, dtype=torch.float32)
    torch.cuda.synchronize()
    ref = oracle.decode(ocfg(cfg), decs, enc)
    np.testing.assert_array_equal(w32.cpu().numpy().view(np.uint32), ref.view(np.uint32))


def test_all_zero_and_constant_matrices(gpu):
    say("all-zero and constant matrices")
    cfg = bsq.Config(d=8, hidden=8)
    for W in (torch.zeros(64, 512), torch.full((64, 512), 0.25)):
        decs, codec, layer, enc = _encode_both(cfg, W.to(torch.bfloat16), gpu)
        assert_layer_equal(layer, enc, cfg)
        np.testing.assert_array_equal(enc.idx, np.arange(cfg.k(512)))     # ties -> lowest columns


def test_empty_matrix_and_empty_batch(gpu):
    say("d_out = 0 and M = 0")
    cfg = bsq.Config(d=8, hidden=8)
    decs, codec, layer, enc = _encode_both(cfg, torch.zeros(0, 512, dtype=torch.bfloat16), gpu)
    np.testing.assert_array_equal(layer.idx.cpu().numpy(), enc.idx)
    np.testing.assert_array_equal(layer.scale.cpu().numpy(), enc.scale)
    y = bsq.bsq_gemv(cfg, codec, layer, synth.activation(512, 1).to(gpu))
    Y = bsq.bsq_gemm(cfg, codec, layer, torch.zeros(0, 512, dtype=torch.bfloat16, device=gpu))
    torch.cuda.synchronize()
    assert y.numel() == 0 and Y.shape == (0, 0)
    W, _ = synth.weight(32, 512, 2, k_outliers=6)
    codec2 = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer2 = bsq.bsq_encode(cfg, codec2, W.to(gpu))
    Y = bsq.bsq_gemm(cfg, codec2, layer2, torch.zeros(0, 512, dtype=torch.bfloat16, device=gpu))
    torch.cuda.synchronize()
    assert Y.shape == (0, 32)


@pytest.mark.parametrize("bad", [float("nan"), float("inf"), float("-inf")])
def test_nonfinite_input_sets_error_word(bad, gpu):
    say(f"non-finite input {bad}")
    cfg = bsq.Config(d=8, hidden=8)
    W = torch.randn(16, 256) * 0.02
    W[3, 77] = bad
    codec = bsq.bsq_codec_prepare(cfg, decoders(cfg), device=gpu)
    with pytest.raises(bsq.BsqError) as e:
        bsq.bsq_encode(cfg, codec, W.to(torch.bfloat16).to(gpu))
    assert e.value.status == bsq.BSQ_ERR_NONFINITE


# ---------------------------------------------------------------- full sizes
FULL = [
    ("qwen3-8b-q-4096x4096-d8", 4096, 4096, 8),
    ("qwen3-8b-q-4096x4096-d16", 4096, 4096, 16),
    ("qwen3-8b-down-4096x12288-d8", 4096, 12288, 8),
    ("qwen3-8b-gate-12288x4096-d16", 12288, 4096, 16),
    ("qwen3-32b-q-8192x5120-d8", 8192, 5120, 8),
    ("qwen3-32b-k-1024x5120-d16", 1024, 5120, 16),
    ("qwen3-32b-o-5120x8192-d8", 5120, 8192, 8),
    ("qwen3-32b-o-5120x8192-d16", 5120, 8192, 16),
    ("qwen3-32b-down-5120x25600-d8", 5120, 25600, 8),
    ("qwen3-32b-gate-25600x5120-d16", 25600, 5120, 16),
]


@pytest.mark.parametrize("case", FULL, ids=[c[0] for c in FULL])
def test_full_size_encode_and_gemv(case, gpu):
    """A whole projection at its real shape: every code, gain, index and int8
    value bit-exact; GEMV (with LoRA) within tolerance on every output."""
    name, d_out, d_in, d = case
    say(f"case {name}")
    cfg = bsq.Config(d=d, hidden=d)
    oc = ocfg(cfg)
    decs = decoders(cfg, seed=d)
    W, cols = synth.weight(d_out, d_in, seed=d_out + d_in, k_outliers=cfg.k(d_in), device=gpu)
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer = bsq.bsq_encode(cfg, codec, W)
    x = synth.activation(d_in, seed=4, device=gpu)
    A, Bm = synth.lora(d_out, d_in, 16, seed=5, device=gpu)
    y = bsq.bsq_gemv(cfg, codec, layer, x, loras=(A, Bm), y_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    Wf = oracle.to_f32(W)
    tabs = oracle.decoder_table(oc, decs)
    enc = oracle.encode(oc, decs, Wf, nthreads=0, tables=tabs)
    np.testing.assert_array_equal(enc.idx, np.asarray(cols))
    assert_layer_equal(layer, enc, cfg)
    lref = (oracle.to_f32(A), oracle.to_f32(Bm))
    w_hat = oracle.decode(oc, decs, enc, tables=tabs)
    xf = oracle.to_f32(x)
    y_ref = oracle.dense_product(w_hat, xf, lref)
    check_product(y.float().cpu().numpy(), y_ref, "gemv", cfg, enc, tabs, w_hat, xf, lref, name, torch.bfloat16)


@pytest.mark.parametrize("M", [16, 64, 256])
@pytest.mark.parametrize("d", [8, 16])
def test_full_size_gemm(d, M, gpu):
    """Qwen3-8B o_proj shape at the batched sizes of the workload, with the
    rank-16 LoRA (token tiles of 16, 64 and 128; at M = 16 and 64 the K steps
    are split over several blocks, whose partials a second launch adds)."""
    say(f"qwen3-8b o_proj 4096x4096 gemm M={M} d={d}")
    cfg = bsq.Config(d=d, hidden=d)
    oc = ocfg(cfg)
    decs = decoders(cfg, seed=d)
    W, _ = synth.weight(4096, 4096, seed=77, k_outliers=cfg.k(4096), device=gpu)
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer = bsq.bsq_encode(cfg, codec, W)
    X = synth.activation(4096, seed=8, device=gpu, batch=M)
    A, Bm = synth.lora(4096, 4096, 16, seed=9, device=gpu)
    Y = bsq.bsq_gemm(cfg, codec, layer, X, lora=(A, Bm), y_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    tabs = oracle.decoder_table(oc, decs)
    enc = oracle.encode(oc, decs, oracle.to_f32(W), tables=tabs)
    assert_layer_equal(layer, enc, cfg)
    lref = (oracle.to_f32(A), oracle.to_f32(Bm))
    w_hat = oracle.decode(oc, decs, enc, tables=tabs)
    Xf = oracle.to_f32(X)
    Y_ref = oracle.dense_product(w_hat, Xf, lref)
    check_product(Y.float().cpu().numpy(), Y_ref, "gemm", cfg, enc, tabs, w_hat, Xf, lref, f"gemm M={M}",
                  torch.bfloat16)


@pytest.mark.parametrize("d_out,d_in,M", [(2304, 4608, 64), (512, 1024, 300)], ids=["2304x4608-M64", "512x1024-M300"])
def test_gemm_wide_and_long_shapes(d_out, d_in, M, gpu):
    """The d = 8 shapes no other case selects: 64-token tiles of 128-row
    blocks (more than 4096 inputs, at most 64 tokens, two blocks per compute
    unit) and 128-token tiles of 64-row blocks (at most 2048 rows, more than
    256 tokens), with rank-16 LoRA and 1% protected columns."""
    say(f"gemm {d_out}x{d_in} M={M} d=8")
    cfg = bsq.Config(d=8, hidden=8)
    oc = ocfg(cfg)
    decs = decoders(cfg, seed=12)
    W, _ = synth.weight(d_out, d_in, seed=78, k_outliers=cfg.k(d_in), device=gpu)
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer = bsq.bsq_encode(cfg, codec, W)
    X = synth.activation(d_in, seed=10, device=gpu, batch=M)
    A, Bm = synth.lora(d_out, d_in, 16, seed=11, device=gpu)
    Y = bsq.bsq_gemm(cfg, codec, layer, X, lora=(A, Bm), y_dtype=torch.float32)
    torch.cuda.synchronize()
    tabs = oracle.decoder_table(oc, decs)
    enc = oracle.encode(oc, decs, oracle.to_f32(W), tables=tabs)
    assert_layer_equal(layer, enc, cfg)
    lref = (oracle.to_f32(A), oracle.to_f32(Bm))
    w_hat = oracle.decode(oc, decs, enc, tables=tabs)
    Xf = oracle.to_f32(X)
    Y_ref = oracle.dense_product(w_hat, Xf, lref)
    check_product(Y.cpu().numpy(), Y_ref, "gemm", cfg, enc, tabs, w_hat, Xf, lref, f"gemm {d_out}x{d_in} M={M}",
                  torch.float32)


@pytest.mark.parametrize("n_mats,d_out,d_in", [(8, 1024, 4096), (64, 1024, 5120)],
                         ids=["8x1024x4096", "64x1024x5120"])
def test_category_batched_stack_encode(n_mats, d_out, d_in, gpu):
    """Layers of one category in one encode (the k_proj shapes of the
    Qwen3-8B stack and, at its full depth, of the 64-layer Qwen3-32B stack):
    every matrix of the stack bit-exact against the oracle's own encoding."""
    say(f"stack of {n_mats} x {d_out}x{d_in}, d=8")
    cfg = bsq.Config(d=8, hidden=8)
    oc = ocfg(cfg)
    decs = decoders(cfg, seed=3)
    W, cols = synth.weight(d_out, d_in, seed=5, k_outliers=cfg.k(d_in), device=gpu, n_mats=n_mats)
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    layer = bsq.bsq_encode(cfg, codec, W)
    torch.cuda.synchronize()
    tabs = oracle.decoder_table(oc, decs)
    for m in range(n_mats):
        enc = oracle.encode(oc, decs, oracle.to_f32(W[m]), tables=tabs)
        np.testing.assert_array_equal(enc.idx, np.asarray(cols[m]))
        assert_layer_equal(layer, enc, cfg, m)


BLOCK_GROUPS = [(blk, d, grp) for blk in ("qwen3-8b", "qwen3-32b") for d in (8, 16)
                for grp in ("qkv", "o", "gateup", "down")]


@pytest.mark.parametrize("blk,d,grp", BLOCK_GROUPS, ids=[f"{b}-d{d}-{g}" for b, d, g in BLOCK_GROUPS])
def test_full_block_grouped_gemv(blk, d, grp, gpu):
    """One decode token through a transformer block's grouped GEMV at full size
    and in the launch configuration of the layer stacks: the group's members
    (q/k/v sharing x, o, gate/up sharing x, down) in one call, one codec per
    projection category, rank-16 LoRA on every member. Every member's
    encoding bit-exact and every output against the oracle."""
    cfg = bsq.Config(d=d, hidden=d)
    oc = ocfg(cfg)
    projs = synth.qwen3_8b_block() if blk == "qwen3-8b" else synth.qwen3_32b_block()
    ps = [p for p in projs if p.group == grp]
    say(f"block {blk} group {grp} d={d}: " + ", ".join(f"{p.name} {p.d_out}x{p.d_in}" for p in ps))
    x = synth.activation(ps[0].d_in, seed=90 + len(grp), device=gpu)
    xf = oracle.to_f32(x)
    codecs, layers, encs, decs_l, loras, Ws = [], [], [], [], [], []
    for p in ps:
        pi = projs.index(p)
        decs = decoders(cfg, seed=100 + pi)
        W, cols = synth.weight(p.d_out, p.d_in, seed=200 + pi, k_outliers=cfg.k(p.d_in), device=gpu)
        codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
        codecs.append(codec)
        layers.append(bsq.bsq_encode(cfg, codec, W))
        Ws.append(W)
        decs_l.append(decs)
        loras.append(synth.lora(p.d_out, p.d_in, 16, seed=300 + pi, device=gpu))
    ys = bsq.bsq_gemv(cfg, codecs, layers, x, loras=loras, y_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    for i, p in enumerate(ps):
        tabs = oracle.decoder_table(oc, decs_l[i])
        enc = oracle.encode(oc, decs_l[i], oracle.to_f32(Ws[i]), tables=tabs)
        assert_layer_equal(layers[i], enc, cfg)
        lref = (oracle.to_f32(loras[i][0]), oracle.to_f32(loras[i][1]))
        w_hat = oracle.decode(oc, decs_l[i], enc, tables=tabs)
        y_ref = oracle.dense_product(w_hat, xf, lref)
        check_product(ys[i].float().cpu().numpy(), y_ref, "gemv", cfg, enc, tabs, w_hat, xf, lref,
                      f"{blk} {p.name} d={d}", torch.bfloat16)
        del w_hat, enc


# ---------------------------------------------------------------- term presence
TERM_CASES = [
    ("d8-table-300x1024", 300, 1024, dict(d=8, hidden=8), torch.bfloat16),
    ("d16-symmetric-200x1024", 200, 1024, dict(d=16, hidden=16), torch.bfloat16),
    ("d16-linear-130x768", 130, 768, dict(d=16, kind=bsq.DEC_LINEAR), torch.bfloat16),
    ("d8-fp32x-256x512", 256, 512, dict(d=8, hidden=8), torch.float32),
    ("d8-4096x4096", 4096, 4096, dict(d=8, hidden=8), torch.bfloat16),
    ("d8-e4m3-300x1024", 300, 1024, dict(d=8, hidden=8, protect_format=bsq.PROT_E4M3), torch.bfloat16),
    ("d16-e5m2-200x1024", 200, 1024, dict(d=16, hidden=16, protect_format=bsq.PROT_E5M2), torch.bfloat16),
    ("d8-res1-e5m2-fp32x-256x512", 256, 512, dict(d=8, hidden=8, kind=bsq.DEC_MLP_RES1,
                                                   protect_format=bsq.PROT_E5M2), torch.float32),
]


def _terms_ref(enc, w_hat, X, lref, fmt=oracle.FMT_INT8):
    """For activations X ([d_in] or [M, d_in]): the oracle's LoRA term
    B (A x), the protected term sum_p value(q8[:, p]) scale_p x_idx_p (stored
    bytes read in format fmt) and the root sum of squares of its parts, and
    the sum of |terms| of the whole product, per output (fp64, the shape of
    the product)."""
    X64 = np.atleast_2d(np.asarray(X, dtype=np.float64))
    A64, B64 = (np.asarray(v, dtype=np.float64) for v in lref)
    q8 = oracle.payload_values(enc.q8, fmt).astype(np.float64)
    lora = (X64 @ A64.T) @ B64.T
    sx = enc.scale.astype(np.float64)[None, :] * X64[:, enc.idx]
    q8t = sx @ q8.T
    q8sq = np.sqrt((sx ** 2) @ (q8 ** 2).T)
    Xa = np.abs(X64)
    total = Xa @ np.abs(w_hat.astype(np.float64)).T + (Xa @ np.abs(A64).T) @ np.abs(B64).T
    out = (lora, q8t, q8sq, total)
    return tuple(v[0] for v in out) if np.ndim(X) == 1 else out


@pytest.mark.parametrize("case", TERM_CASES, ids=[c[0] for c in TERM_CASES])
def test_gemv_lora_and_protected_terms(case, gpu):
    """The LoRA term and the int8 protected term of bsq_gemv, each on its own:
    y(x, with LoRA) - y(x) against the oracle's B (A x), and y(x) - y(x with
    the protected inputs zeroed) against sum_p q8 scale_p x_idx_p, per output,
    to within fp32 rounding (both terms are computed in fp32 from exact
    products on every GEMV path)."""
    name, d_out, d_in, kw, dtype = case
    say(f"term presence {name}")
    cfg, decs, codec, layer, W, encs, tabs = _make(name, d_out, d_in, kw, dtype, 1, False, gpu)
    enc = encs[0]
    x = synth.activation(d_in, seed=15, dtype=dtype)
    A, Bm = synth.lora(d_out, d_in, 16, seed=16)
    xd = x.to(gpu)
    y_l = bsq.bsq_gemv(cfg, codec, layer, xd, loras=(A.to(gpu), Bm.to(gpu)), y_dtype=torch.float32)
    y_0 = bsq.bsq_gemv(cfg, codec, layer, xd, y_dtype=torch.float32)
    xm = x.clone()
    xm[torch.as_tensor(enc.idx, dtype=torch.long)] = 0
    y_m = bsq.bsq_gemv(cfg, codec, layer, xm.to(gpu), y_dtype=torch.float32)
    torch.cuda.synchronize()
    xf = oracle.to_f32(x)
    w_hat = oracle.decode(ocfg(cfg), decs, enc, tables=tabs)
    lora, q8t, _, total = _terms_ref(enc, w_hat, xf, (oracle.to_f32(A), oracle.to_f32(Bm)),
                                     OFMT[cfg.protect_format])
    y_l, y_0, y_m = (v.cpu().numpy() for v in (y_l, y_0, y_m))
    assert term_bar(y_l, y_0, lora, total, 16, "LoRA term") > 100
    assert term_bar(y_0, y_m, q8t, total, len(enc.idx), "protected term") > 100


@pytest.mark.parametrize("d,M,fmt", [(8, 16, bsq.PROT_INT8), (8, 64, bsq.PROT_INT8), (8, 256, bsq.PROT_INT8),
                                     (16, 16, bsq.PROT_INT8), (16, 256, bsq.PROT_INT8), (8, 64, bsq.PROT_E4M3),
                                     (16, 16, bsq.PROT_E5M2)])
def test_gemm_lora_and_protected_terms(d, M, fmt, gpu):
    """As for the GEMV, on the fused GEMM: the LoRA term to within fp32
    rounding (it goes through the MFMA with T split exactly into three bf16
    parts, every partial product exact); the protected term goes through the
    MFMA as bf16(q8 scale), so its bar adds the sub-Gaussian bound of those
    roundings."""
    say(f"gemm term presence d={d} M={M} format={fmt}")
    cfg, decs, codec, layer, W, encs, tabs = _make("gemm-terms", 320, 2048, dict(d=d, hidden=d, protect_format=fmt),
                                                   torch.bfloat16, 1, False, gpu)
    enc = encs[0]
    X = synth.activation(2048, seed=17, dtype=torch.bfloat16, batch=M)
    A, Bm = synth.lora(320, 2048, 16, seed=18)
    Xd = X.to(gpu)
    Y_l = bsq.bsq_gemm(cfg, codec, layer, Xd, lora=(A.to(gpu), Bm.to(gpu)), y_dtype=torch.float32)
    Y_0 = bsq.bsq_gemm(cfg, codec, layer, Xd, y_dtype=torch.float32)
    Xm = X.clone()
    Xm[:, torch.as_tensor(enc.idx, dtype=torch.long)] = 0
    Y_m = bsq.bsq_gemm(cfg, codec, layer, Xm.to(gpu), y_dtype=torch.float32)
    torch.cuda.synchronize()
    Xf = oracle.to_f32(X)
    w_hat = oracle.decode(ocfg(cfg), decs, enc, tables=tabs)
    Y_l, Y_0, Y_m = (v.cpu().numpy() for v in (Y_l, Y_0, Y_m))
    lora, q8t, q8sq, total = _terms_ref(enc, w_hat, Xf, (oracle.to_f32(A), oracle.to_f32(Bm)), OFMT[fmt])
    assert term_bar(Y_l, Y_0, lora, total, 16, "LoRA term") > 100
    assert term_bar(Y_0, Y_m, q8t, total, len(enc.idx), "protected term", rounded=q8sq) > 10
