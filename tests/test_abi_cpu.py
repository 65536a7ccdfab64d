"""The C ABI without a GPU: the library loads, exports every entry point that
include/bsq.h declares, sizes its buffers consistently with the oracle's
storage accounting (eq. real_size), and rejects invalid arguments on the host
before launching anything (fake, never-dereferenced device pointers)."""
import ctypes as ct
import os
import re

import pytest

import oracle
import paper_2607_08643_amd as bsq
from paper_2607_08643_amd import _binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x7F0000000000  # 256-aligned, never dereferenced: every call below fails validation first


def header_functions():
    with open(os.path.join(ROOT, "include", "bsq.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^[a-z0-9_ ]*?\*?\s*(bsq_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_symbol():
    L = bsq.lib()
    names = header_functions()
    assert len(names) >= 11
    for name in names:
        assert hasattr(L, name), name
    assert set(names) == set(B.EXPORTS)
    assert bsq.bsq_version() == 8
    for s in range(0, 9):
        assert bsq.status_str(s) != "unknown status"
    assert bsq.status_str(99) == "unknown status"


@pytest.mark.parametrize("kw,status", [
    (dict(d=12), bsq.BSQ_ERR_UNSUPPORTED),
    (dict(d=0), bsq.BSQ_ERR_ARG),
    (dict(d=17), bsq.BSQ_ERR_ARG),
    (dict(stages=0), bsq.BSQ_ERR_ARG),
    (dict(stages=5), bsq.BSQ_ERR_ARG),
    (dict(kind=4), bsq.BSQ_ERR_ARG),
    (dict(hidden=0), bsq.BSQ_ERR_ARG),
    (dict(kind=bsq.DEC_MLP_RES1, hidden=0), bsq.BSQ_ERR_ARG),
    (dict(kind=bsq.DEC_MLP_RES1, hidden=65), bsq.BSQ_ERR_ARG),
    (dict(protect_format=3), bsq.BSQ_ERR_ARG),
    (dict(protect_format=-1), bsq.BSQ_ERR_ARG),
    (dict(hidden=65), bsq.BSQ_ERR_ARG),
    (dict(protect_num=2, protect_den=1), bsq.BSQ_ERR_ARG),
    (dict(protect_num=-1), bsq.BSQ_ERR_ARG),
    (dict(protect_den=0), bsq.BSQ_ERR_ARG),
    (dict(), bsq.BSQ_OK),
    (dict(d=16, hidden=16), bsq.BSQ_OK),
    (dict(kind=bsq.DEC_IDENTITY, hidden=0), bsq.BSQ_OK),
    (dict(kind=bsq.DEC_MLP_RES1), bsq.BSQ_OK),
    (dict(d=16, kind=bsq.DEC_MLP_RES1, hidden=5), bsq.BSQ_OK),
    (dict(protect_format=bsq.PROT_E4M3), bsq.BSQ_OK),
    (dict(protect_format=bsq.PROT_E5M2, protect_axis=1), bsq.BSQ_OK),
])
def test_config_validation(kw, status):
    assert bsq.bsq_config_check(bsq.Config(**kw)) == status


def test_code_bits_other_than_chunk_length_need_the_linear_encoder():
    """b (codebook_bits) may differ from d (codebook_dim) only with the
    linear encoder (Section III-C's E_phi maps R^d to R^b); b and d are 8 or
    16, and the identity decoder needs b = d."""
    Lib = bsq.lib()
    c = bsq.Config().c()
    c.b = 16
    assert Lib.bsq_config_check(ct.byref(c)) == bsq.BSQ_ERR_ARG
    c.encoder = bsq.ENC_LINEAR
    assert Lib.bsq_config_check(ct.byref(c)) == bsq.BSQ_OK
    c.b = 12
    assert Lib.bsq_config_check(ct.byref(c)) == bsq.BSQ_ERR_UNSUPPORTED
    c.b = 8
    assert Lib.bsq_config_check(ct.byref(c)) == bsq.BSQ_OK            # a linear encoder at b = d
    ok = bsq.Config(d=16, codebook_bits=8, encoder=bsq.ENC_LINEAR)
    assert bsq.bsq_config_check(ok) == bsq.BSQ_OK
    assert bsq.bsq_config_check(bsq.Config(d=16, codebook_bits=8, encoder=bsq.ENC_LINEAR,
                                           kind=bsq.DEC_IDENTITY, hidden=0)) == bsq.BSQ_ERR_ARG
    c.encoder = 2
    assert Lib.bsq_config_check(ct.byref(c)) == bsq.BSQ_ERR_ARG


@pytest.mark.parametrize("d", [8, 16])
@pytest.mark.parametrize("shape", [(4096, 4096), (1024, 4096), (4096, 12288), (25600, 5120), (333, 296), (0, 256)])
@pytest.mark.parametrize("rank", [0, 16])
@pytest.mark.parametrize("axis", [0, 1], ids=["cols", "rows"])
@pytest.mark.parametrize("kind", [bsq.DEC_MLP, bsq.DEC_MLP_RES1], ids=["res0", "res1"])
def test_sizes_match_oracle_accounting(d, shape, rank, axis, kind):
    d_out, d_in = shape
    if d_in % d:
        pytest.skip("not chunkable")
    fmt = bsq.PROT_E4M3 if kind == bsq.DEC_MLP_RES1 else bsq.PROT_INT8   # the format does not change a size
    cfg = bsq.Config(d=d, hidden=d, kind=kind, protect_axis=axis, protect_format=fmt)
    got = bsq.bsq_layer_sizes(cfg, d_out, d_in, rank)
    ref = oracle.sizes(oracle.Config(d=d, b=d, stages=2, kind=kind, hidden=d, protect_axis=axis,
                                     protect_format=fmt), d_out, d_in, rank)
    for key in ("S_code", "S_dec", "S_8bit", "S_LoRA", "S_meta", "S_tot", "bpw_nominal"):
        assert got[key] == pytest.approx(ref[key], rel=0, abs=1e-9), key
    if d_out:
        assert got["bpw_real"] == pytest.approx(ref["bpw_real"], rel=1e-12)
    assert got["pitch"] == oracle.pitch(d_in, d) and got["k"] == ref["k"]
    rows = (d_out + 63) // 64 * 64   # tiled planes pad the rows to 64
    assert got["code_plane_bytes"] == rows * got["pitch"] * (1 if d == 8 else 2)
    assert got["gain_plane_bytes"] == rows * got["pitch"] * 2
    if axis == 1:
        # protected rows: [k][roundup(d_in, 16)] int8 payload and no bitmap
        assert got["k"] == cfg.k(d_out) and got["bits_bytes"] == 0
        assert got["q8_bytes"] == got["k"] * ((d_in + 15) // 16 * 16)
        return
    # one bit per padded input column when there are protected columns
    assert got["bits_bytes"] == (got["pitch"] * d // 8 if got["k"] else 0)


def test_shape_validation():
    cfg = bsq.Config()
    with pytest.raises(bsq.BsqError) as e:
        bsq.bsq_layer_sizes(cfg, 16, 100)  # 100 is not a multiple of 8
    assert e.value.status == bsq.BSQ_ERR_SHAPE
    with pytest.raises(bsq.BsqError) as e:
        bsq.bsq_layer_sizes(cfg, 16, 0)
    assert e.value.status == bsq.BSQ_ERR_SHAPE
    with pytest.raises(bsq.BsqError) as e:
        bsq.bsq_layer_sizes(cfg, -1, 64)
    assert e.value.status == bsq.BSQ_ERR_SHAPE
    with pytest.raises(bsq.BsqError) as e:
        bsq.bsq_layer_sizes(cfg, 16, 64, lora_rank=17)
    assert e.value.status == bsq.BSQ_ERR_ARG


def _fake_layer(cfg, d_out, d_in, n_mats=1, misalign=False):
    L = B.bsq_layer()
    for s in range(cfg.stages):
        L.codes[s] = FAKE + 0x1000 * s + (1 if misalign else 0)
        L.gains[s] = FAKE + 0x100000 + 0x1000 * s
    L.prot_idx, L.prot_q8, L.prot_scale = FAKE + 0x200000, FAKE + 0x300000, FAKE + 0x400000
    L.prot_bits = FAKE + 0x500000
    L.d_out, L.d_in, L.pitch, L.k, L.n_mats = d_out, d_in, cfg.pitch(d_in), cfg.k(d_in), n_mats
    return L


def _encode(cfg, L, *, W=FAKE, dtype=bsq.BSQ_BF16, n_mats=1, d_out=64, d_in=256, ws_bytes=1 << 30, err=FAKE,
            ws=FAKE, codec=FAKE):
    c = cfg.c()
    return bsq.lib().bsq_encode(ct.byref(c), codec and ct.c_void_p(codec), W and ct.c_void_p(W), dtype, n_mats,
                                d_out, d_in, None, ct.byref(L) if L is not None else None,
                                err and ct.c_void_p(err), ws and ct.c_void_p(ws), ws_bytes, None)


def test_encode_rejects_before_launch():
    cfg = bsq.Config()
    L = _fake_layer(cfg, 64, 256)
    assert _encode(cfg, L, W=0) == bsq.BSQ_ERR_ARG
    assert _encode(cfg, None) == bsq.BSQ_ERR_ARG
    assert _encode(cfg, L, err=0) == bsq.BSQ_ERR_ARG
    assert _encode(cfg, L, dtype=7) == bsq.BSQ_ERR_DTYPE
    assert _encode(cfg, L, d_in=250) == bsq.BSQ_ERR_SHAPE
    assert _encode(cfg, L, d_out=65) == bsq.BSQ_ERR_ARG          # layer shape mismatch
    assert _encode(cfg, L, n_mats=2) == bsq.BSQ_ERR_ARG
    assert _encode(cfg, L, W=FAKE + 8) == bsq.BSQ_ERR_ALIGN
    assert _encode(cfg, L, ws=FAKE + 64) == bsq.BSQ_ERR_ALIGN
    assert _encode(cfg, _fake_layer(cfg, 64, 256, misalign=True)) == bsq.BSQ_ERR_ALIGN
    assert _encode(cfg, L, ws_bytes=16) == bsq.BSQ_ERR_BUFFER_TOO_SMALL
    bad = _fake_layer(cfg, 64, 256)
    bad.pitch = 33
    assert _encode(cfg, bad) == bsq.BSQ_ERR_ARG
    bad = _fake_layer(cfg, 64, 256)
    bad.prot_idx = 0
    assert _encode(cfg, bad) == bsq.BSQ_ERR_ARG
    bad = _fake_layer(cfg, 64, 256)
    bad.k = 1
    assert _encode(cfg, bad) == bsq.BSQ_ERR_ARG
    bad = _fake_layer(cfg, 64, 256)
    bad.prot_bits = 0                                          # the encoder writes the bitmap
    assert _encode(cfg, bad) == bsq.BSQ_ERR_ARG
    bad = _fake_layer(cfg, 64, 256)
    bad.prot_bits = FAKE + 0x500004
    assert _encode(cfg, bad) == bsq.BSQ_ERR_ALIGN
    bad = _fake_layer(cfg, 64, 256)
    bad.prot_q8 = FAKE + 0x300008                              # rows are read with 16-byte loads
    assert _encode(cfg, bad) == bsq.BSQ_ERR_ALIGN


def test_decode_gemv_gemm_reject_before_launch():
    cfg = bsq.Config()
    c = cfg.c()
    Lib = bsq.lib()
    L = _fake_layer(cfg, 64, 256)
    assert Lib.bsq_decode(ct.byref(c), ct.c_void_p(FAKE), ct.byref(L), ct.c_void_p(FAKE), 5, None) == bsq.BSQ_ERR_DTYPE
    assert Lib.bsq_decode(ct.byref(c), None, ct.byref(L), ct.c_void_p(FAKE), 0, None) == bsq.BSQ_ERR_ARG
    assert Lib.bsq_decode(ct.byref(c), ct.c_void_p(FAKE), ct.byref(L), ct.c_void_p(FAKE + 4), 0, None) == bsq.BSQ_ERR_ALIGN
    # sequential stage decode: stage in range, accumulate 0/1, fp32 output aligned
    def dstage(stage=0, acc=0, out=FAKE):
        return Lib.bsq_decode_stage(ct.byref(c), ct.c_void_p(FAKE), ct.byref(L), stage, acc,
                                    out and ct.c_void_p(out), None)
    assert dstage(stage=-1) == bsq.BSQ_ERR_ARG
    assert dstage(stage=cfg.stages) == bsq.BSQ_ERR_ARG
    assert dstage(acc=2) == bsq.BSQ_ERR_ARG
    assert dstage(out=0) == bsq.BSQ_ERR_ARG
    assert dstage(out=FAKE + 8) == bsq.BSQ_ERR_ALIGN
    codecs = (ct.c_void_p * 1)(FAKE)
    layers = (B.bsq_layer * 1)(L)
    ys = (ct.c_void_p * 1)(FAKE)

    def gemv(n=1, x=FAKE, xd=1, yd=1, ws=FAKE, ws_bytes=1 << 30, loras=None, lay=layers, err=None, run=False):
        f = Lib.bsq_gemv_run if run else Lib.bsq_gemv
        return f(ct.byref(c), n, codecs, lay, loras, x and ct.c_void_p(x), xd, ys, yd,
                 ws and ct.c_void_p(ws), ws_bytes, err and ct.c_void_p(err), None)
    assert gemv(n=0) == bsq.BSQ_ERR_ARG
    assert gemv(n=9) == bsq.BSQ_ERR_ARG
    assert gemv(x=0) == bsq.BSQ_ERR_ARG
    assert gemv(xd=3) == bsq.BSQ_ERR_DTYPE
    assert gemv(yd=3) == bsq.BSQ_ERR_DTYPE
    assert gemv(ws_bytes=8) == bsq.BSQ_ERR_BUFFER_TOO_SMALL
    assert gemv(ws=FAKE + 16) == bsq.BSQ_ERR_ALIGN
    assert gemv(loras=(B.bsq_lora * 1)(B.bsq_lora(FAKE, FAKE, 17))) == bsq.BSQ_ERR_ARG
    assert gemv(loras=(B.bsq_lora * 1)(B.bsq_lora(0, FAKE, 4))) == bsq.BSQ_ERR_ARG
    stacked = (B.bsq_layer * 1)(_fake_layer(cfg, 64, 256, n_mats=2))
    assert gemv(lay=stacked) == bsq.BSQ_ERR_ARG
    nobits = _fake_layer(cfg, 64, 256)
    nobits.prot_bits = 0                                       # the product masks with the bitmap
    assert gemv(lay=(B.bsq_layer * 1)(nobits)) == bsq.BSQ_ERR_ARG
    # the optional device error word must be 4-byte aligned (both entry points)
    assert gemv(err=FAKE + 2) == bsq.BSQ_ERR_ALIGN
    assert gemv(err=FAKE + 2, run=True) == bsq.BSQ_ERR_ALIGN
    assert gemv(x=0, run=True) == bsq.BSQ_ERR_ARG

    def gemm(M=16, ldx=256, ldy=64, xd=1, X=FAKE, ws_bytes=1 << 30, lora=None, err=None):
        lo = B.bsq_lora(0, 0, 0) if lora is None else lora
        return Lib.bsq_gemm(ct.byref(c), ct.c_void_p(FAKE), ct.byref(L), ct.byref(lo), X and ct.c_void_p(X), xd, M,
                            ldx, ct.c_void_p(FAKE), 1, ldy, ct.c_void_p(FAKE), ws_bytes, err and ct.c_void_p(err),
                            None)
    assert gemm(xd=0) == bsq.BSQ_ERR_DTYPE               # X must be bf16
    assert gemm(M=-1) == bsq.BSQ_ERR_SHAPE
    assert gemm(ldx=128) == bsq.BSQ_ERR_SHAPE
    assert gemm(ldx=260) == bsq.BSQ_ERR_SHAPE            # not a multiple of 8
    assert gemm(ldy=32) == bsq.BSQ_ERR_SHAPE
    assert gemm(X=FAKE + 2) == bsq.BSQ_ERR_ALIGN
    assert gemm(ws_bytes=4) == bsq.BSQ_ERR_BUFFER_TOO_SMALL
    assert gemm(lora=B.bsq_lora(FAKE, FAKE, 0x7fffffff)) == bsq.BSQ_ERR_ARG
    assert gemm(err=FAKE + 1) == bsq.BSQ_ERR_ALIGN


def test_gemv_noalloc_rejects_before_launch():
    """bsq_gemv_noalloc validates on the host before it touches the device:
    a group whose workspace exceeds the library's scratch array is refused
    with BSQ_ERR_BUFFER_TOO_SMALL, bad arguments as bsq_gemv refuses them."""
    cfg = bsq.Config()
    c = cfg.c()
    Lib = bsq.lib()
    assert B.GEMV_NOALLOC_SCRATCH_BYTES == 8 << 20

    def call(L, n=1, clear=0, x=FAKE, err=None):
        return Lib.bsq_gemv_noalloc(ct.byref(c), n, (ct.c_void_p * 1)(FAKE), (B.bsq_layer * 1)(L), None,
                                    x and ct.c_void_p(x), 1, (ct.c_void_p * 1)(FAKE), 1, clear,
                                    err and ct.c_void_p(err), None)
    # 32768 rows x 65536 inputs at d = 8: 512 row groups x 127 slices of
    # flagged partial sums (33 MB), far more than the array holds
    assert bsq.bsq_workspace_bytes(cfg, bsq.OP_GEMV, 1, 32768, 65536) > 3 * B.GEMV_NOALLOC_SCRATCH_BYTES
    assert call(_fake_layer(cfg, 32768, 65536)) == bsq.BSQ_ERR_BUFFER_TOO_SMALL
    L = _fake_layer(cfg, 64, 256)
    assert call(L, clear=2) == bsq.BSQ_ERR_ARG
    assert call(L, n=0) == bsq.BSQ_ERR_ARG
    assert call(L, x=0) == bsq.BSQ_ERR_ARG
    assert call(L, x=FAKE + 2) == bsq.BSQ_ERR_ALIGN
    assert call(L, err=FAKE + 1) == bsq.BSQ_ERR_ALIGN


def test_wait_limit_is_settable_and_restorable():
    """bsq_debug_set_wait_limit returns the previous bound; a negative value
    restores the default (host state only, no launch)."""
    default = bsq.bsq_debug_set_wait_limit(-1)
    assert default > 1000
    assert bsq.bsq_debug_set_wait_limit(0) == default
    assert bsq.bsq_debug_set_wait_limit(7) == 0
    assert bsq.bsq_debug_set_wait_limit(-5) == 7
    assert bsq.bsq_debug_set_wait_limit(-1) == default


def test_product_workspaces_hold_a_header():
    """GEMV and GEMM workspaces start with a 256-byte header for the poison
    word, so they exceed their slot and scratch areas by at least that."""
    cfg = bsq.Config()
    assert bsq.bsq_workspace_bytes(cfg, bsq.OP_GEMM, 1, 64, 256, 1) >= 256 + 16 * 16 * 4
    assert bsq.bsq_workspace_bytes(cfg, bsq.OP_GEMV, 1, 64, 256) >= 256 + 8 * 16 * 4


def test_codec_prepare_rejects_before_launch():
    cfg = bsq.Config()
    c = cfg.c()
    Lib = bsq.lib()
    need = bsq.bsq_codec_bytes(cfg)
    assert need == 2 * 256 * 8 * 8
    # d = 16 symmetric decoder: the four tables, then per stage the byte-split
    # pre-activation halves (fp16 [2][256][h]) and fp32 copies of W2 and b2
    split = 2 * 256 * 16 * 2 + 16 * 16 * 4 + 16 * 4
    assert bsq.bsq_codec_bytes(bsq.Config(d=16, hidden=16)) == 2 * 65536 * 16 * 8 + 2 * split
    assert bsq.bsq_codec_bytes(bsq.Config(d=16, kind=bsq.DEC_LINEAR)) == 2 * 65536 * 16 * 8
    decs = (B.bsq_decoder * 4)(*[B.bsq_decoder(FAKE, FAKE, FAKE, FAKE)] * 4)
    assert Lib.bsq_codec_prepare(ct.byref(c), decs, ct.c_void_p(FAKE), need - 1, None) == bsq.BSQ_ERR_BUFFER_TOO_SMALL
    assert Lib.bsq_codec_prepare(ct.byref(c), decs, ct.c_void_p(FAKE + 128), need, None) == bsq.BSQ_ERR_ALIGN
    assert Lib.bsq_codec_prepare(ct.byref(c), None, ct.c_void_p(FAKE), need, None) == bsq.BSQ_ERR_ARG
    nob2 = (B.bsq_decoder * 4)(*[B.bsq_decoder(FAKE, FAKE, FAKE, 0)] * 4)
    assert Lib.bsq_codec_prepare(ct.byref(c), nob2, ct.c_void_p(FAKE), need, None) == bsq.BSQ_ERR_ARG
    # the residual-block decoder needs R and c as well; it has no split tables at d = 16
    r1 = bsq.Config(kind=bsq.DEC_MLP_RES1)
    c1 = r1.c()
    assert bsq.bsq_codec_bytes(r1) == need
    assert bsq.bsq_codec_bytes(bsq.Config(d=16, hidden=16, kind=bsq.DEC_MLP_RES1)) == 2 * 65536 * 16 * 8
    noR = (B.bsq_decoder * 4)(*[B.bsq_decoder(FAKE, FAKE, FAKE, FAKE, 0, FAKE)] * 4)
    noc = (B.bsq_decoder * 4)(*[B.bsq_decoder(FAKE, FAKE, FAKE, FAKE, FAKE, 0)] * 4)
    for dd in (noR, noc):
        assert Lib.bsq_codec_prepare(ct.byref(c1), dd, ct.c_void_p(FAKE), need, None) == bsq.BSQ_ERR_ARG


def test_workspace_sizes_are_positive_and_grow():
    cfg = bsq.Config()
    e1 = bsq.bsq_workspace_bytes(cfg, bsq.OP_ENCODE, 1, 4096, 4096)
    e8 = bsq.bsq_workspace_bytes(cfg, bsq.OP_ENCODE, 8, 4096, 4096)
    assert 0 < e1 < e8
    g1 = bsq.bsq_workspace_bytes(cfg, bsq.OP_GEMV, 1, 4096, 4096)
    g3 = bsq.bsq_workspace_bytes(cfg, bsq.OP_GEMV, 3, 4096, 4096)
    assert 0 < g1 <= g3 and g3 >= 3 * 16 * 4
    assert bsq.bsq_workspace_bytes(cfg, bsq.OP_GEMM, 1, 4096, 4096, 256) >= 256 * 16 * 4
    with pytest.raises(bsq.BsqError):
        bsq.bsq_workspace_bytes(cfg, bsq.OP_GEMV, 9, 4096, 4096)
    with pytest.raises(bsq.BsqError):
        bsq.bsq_workspace_bytes(cfg, 7, 1, 4096, 4096)


def test_product_path_has_no_cpu_fallback():
    """The binding imports neither the oracle nor any CPU implementation."""
    import inspect
    src = inspect.getsource(B)
    assert "import oracle" not in src and "from oracle" not in src
    with open(os.path.join(ROOT, "paper_2607_08643_amd", "__init__.py")) as f:
        assert "oracle" not in f.read()


def test_row_axis_and_select_reject_before_launch():
    """Protected rows (protect_axis = 1), bsq_encode_with_set and
    bsq_coupled_select validate on the host and return before any launch."""
    c = bsq.Config(protect_axis=2).c()
    assert bsq.lib().bsq_config_check(ct.byref(c)) == bsq.BSQ_ERR_ARG
    cfg = bsq.Config(protect_axis=1)
    L = _fake_layer(cfg, 300, 256)
    L.k = cfg.k(300)                                           # k counts rows on this axis
    L.prot_bits = 0                                            # no bitmap for protected rows
    assert L.k == 3
    ws_rows = bsq.bsq_workspace_bytes(cfg, bsq.OP_ENCODE, 1, 300, 256)
    ws_cols = bsq.bsq_workspace_bytes(bsq.Config(), bsq.OP_ENCODE, 1, 300, 256)
    assert ws_rows != ws_cols                                  # scores over rows, not columns
    bad = _fake_layer(cfg, 300, 256)
    bad.k = cfg.k(600)                                         # not ceil(rho * d_out)
    assert _encode(cfg, bad, d_out=300) == bsq.BSQ_ERR_ARG
    L.prot_q8 = FAKE + 0x300008
    assert _encode(cfg, L, d_out=300) == bsq.BSQ_ERR_ALIGN
    L.prot_q8 = 0
    assert _encode(cfg, L, d_out=300) == bsq.BSQ_ERR_ARG
    L.prot_q8 = FAKE + 0x300000
    cc = cfg.c()
    lib = bsq.lib()
    # a protected set is required when k > 0
    assert lib.bsq_encode_with_set(ct.byref(cc), ct.c_void_p(FAKE), ct.c_void_p(FAKE), bsq.BSQ_BF16, 1, 300, 256,
                                   None, ct.byref(L), ct.c_void_p(FAKE), ct.c_void_p(FAKE), 1 << 30,
                                   None) == bsq.BSQ_ERR_ARG
    assert lib.bsq_encode_with_set(ct.byref(cc), ct.c_void_p(FAKE), ct.c_void_p(FAKE), bsq.BSQ_BF16, 1, 300, 256,
                                   ct.c_void_p(FAKE + 2), ct.byref(L), ct.c_void_p(FAKE), ct.c_void_p(FAKE),
                                   1 << 30, None) == bsq.BSQ_ERR_ALIGN

    def sel(d_model=256, d_ffn=1000, dtype=bsq.BSQ_BF16, ws_bytes=1 << 30, Wg=FAKE, idx=FAKE, ws=FAKE):
        return lib.bsq_coupled_select(ct.byref(cc), Wg and ct.c_void_p(Wg), ct.c_void_p(FAKE), ct.c_void_p(FAKE),
                                      dtype, d_model, d_ffn, None, None, None, idx and ct.c_void_p(idx), None,
                                      ct.c_void_p(FAKE), ws and ct.c_void_p(ws), ws_bytes, None)
    assert sel(Wg=0) == bsq.BSQ_ERR_ARG
    assert sel(idx=0) == bsq.BSQ_ERR_ARG
    assert sel(ws=0) == bsq.BSQ_ERR_ARG
    assert sel(dtype=9) == bsq.BSQ_ERR_DTYPE
    assert sel(d_ffn=0) == bsq.BSQ_ERR_SHAPE
    assert sel(d_ffn=(1 << 18) + 1) == bsq.BSQ_ERR_UNSUPPORTED
    assert sel(Wg=FAKE + 4) == bsq.BSQ_ERR_ALIGN
    assert sel(ws_bytes=64) == bsq.BSQ_ERR_BUFFER_TOO_SMALL
    assert bsq.bsq_workspace_bytes(cfg, bsq.OP_SELECT, 1, 25600, 5120) > 25600 * 8 * 4


@pytest.mark.parametrize("d,b", [(8, 16), (16, 8), (8, 8), (16, 16)])
@pytest.mark.parametrize("axis", [0, 1], ids=["cols", "rows"])
def test_sizes_with_a_linear_encoder_match_oracle(d, b, axis):
    """b bits per chunk and stage, b / 8 bytes per chunk in the code planes,
    and the encoder's b d parameters in S_dec, as the oracle counts them."""
    cfg = bsq.Config(d=d, codebook_bits=b, hidden=b, encoder=bsq.ENC_LINEAR, protect_axis=axis)
    got = bsq.bsq_layer_sizes(cfg, 4096, 4096, 16)
    ref = oracle.sizes(oracle.Config(d=d, b=b, stages=2, kind=oracle.KIND_MLP, hidden=b, protect_axis=axis,
                                     encoder=oracle.ENC_LINEAR), 4096, 4096, 16)
    for key in ("S_code", "S_dec", "S_8bit", "S_LoRA", "S_meta", "S_tot", "bpw_nominal", "bpw_real"):
        assert got[key] == pytest.approx(ref[key], rel=1e-12), key
    assert got["code_plane_bytes"] == 4096 * got["pitch"] * (b // 8)


def test_codec_with_a_linear_encoder_needs_E():
    Lib = bsq.lib()
    cfg = bsq.Config(d=8, codebook_bits=16, hidden=16, encoder=bsq.ENC_LINEAR)
    c = cfg.c()
    need = bsq.bsq_codec_bytes(cfg)
    # three tables of 2^16 x 8 entries per stage (fp32, bf16, fp16), then the two E copies
    assert need == 2 * 65536 * 8 * 8 + 2 * 16 * 8 * 4
    noE = (B.bsq_decoder * 4)(*[B.bsq_decoder(FAKE, FAKE, FAKE, FAKE, 0, 0, 0)] * 4)
    assert Lib.bsq_codec_prepare(ct.byref(c), noE, ct.c_void_p(FAKE), need, None) == bsq.BSQ_ERR_ARG
    assert Lib.bsq_codec_prepare(ct.byref(c), noE, ct.c_void_p(FAKE), need - 1, None) == bsq.BSQ_ERR_BUFFER_TOO_SMALL


def test_training_entry_points_validate_before_launch():
    """Codec training takes the linear encoder and the plain symmetric
    decoder; parameter count b d + h b + h + d h + d; every bad argument is
    refused on the host."""
    Lib = bsq.lib()
    cfg = bsq.Config(d=8, hidden=8, encoder=bsq.ENC_LINEAR)
    assert bsq.bsq_train_param_count(cfg) == 64 + 64 + 8 + 64 + 8
    assert bsq.bsq_train_param_count(bsq.Config(d=8, codebook_bits=16, hidden=12, encoder=bsq.ENC_LINEAR)) == \
        16 * 8 + 12 * 16 + 12 + 8 * 12 + 8
    for bad in (bsq.Config(d=8, hidden=8), bsq.Config(d=8, hidden=8, encoder=bsq.ENC_LINEAR, kind=bsq.DEC_MLP_RES1),
                bsq.Config(d=8, encoder=bsq.ENC_LINEAR, kind=bsq.DEC_LINEAR)):
        with pytest.raises(bsq.BsqError) as e:
            bsq.bsq_train_param_count(bad)
        assert e.value.status == bsq.BSQ_ERR_UNSUPPORTED
    ws = bsq.bsq_train_workspace_bytes(cfg, 4096)
    assert ws > 4096 * (2 * 8 + 2 * 8 + 2 * 8) * 4
    c = cfg.c()
    hp = bsq.TrainHyper().c()
    F = ct.c_void_p(FAKE)
    ok = dict(chunks=F, x=bsq.BSQ_F32, nt=4096, idx=None, n=4096, th=F, g=F, l=F, err=None, ws=F, wsb=ws)

    def call(**kw):
        a = {**ok, **kw}
        return Lib.bsq_train_grad(ct.byref(c), ct.byref(a.get("hp", hp)), a["chunks"], a["x"], a["nt"], a["idx"],
                                  a["n"], a["th"], a["g"], a["l"], a["err"], a["ws"], a["wsb"], None)
    assert call(n=0) == bsq.BSQ_ERR_SHAPE
    assert call(n=4097) == bsq.BSQ_ERR_SHAPE          # more than the chunks, with no index list
    assert call(wsb=ws - 1) == bsq.BSQ_ERR_BUFFER_TOO_SMALL
    assert call(x=7) == bsq.BSQ_ERR_DTYPE
    assert call(th=None) == bsq.BSQ_ERR_ARG
    assert call(ws=ct.c_void_p(FAKE + 64)) == bsq.BSQ_ERR_ALIGN
    assert call(idx=ct.c_void_p(FAKE + 4)) == bsq.BSQ_ERR_ALIGN
    nan_hp = bsq.TrainHyper(lr=float("nan")).c()
    assert call(hp=nan_hp) == bsq.BSQ_ERR_ARG
    assert call(hp=bsq.TrainHyper(beta2=1.0).c()) == bsq.BSQ_ERR_ARG
    assert Lib.bsq_train_adam(ct.byref(c), ct.byref(hp), 0, F, F, F, F, None) == bsq.BSQ_ERR_ARG
    assert Lib.bsq_train_adam(ct.byref(c), ct.byref(hp), 1, F, None, F, F, None) == bsq.BSQ_ERR_ARG
