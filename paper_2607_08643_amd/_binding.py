"""ctypes binding of libbsq.so (include/bsq.h). Argument marshalling only:
torch provides device memory and the current stream; every step of the codec
and of the products runs in the library's HIP kernels.

The functions carry the C names. Where the C call writes into caller buffers,
the Python function allocates them with torch unless `out=` / `ws=` are given
(pre-allocated buffers are what a HIP-graph capture needs).
"""
from __future__ import annotations

import ctypes as ct
import math
import os
from dataclasses import dataclass, field

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbsq.so")

MAX_STAGES = 4
PITCH_ALIGN = 16
MAX_LORA_RANK = 16
MAX_GROUP = 8
GEMV_NOALLOC_SCRATCH_BYTES = 8 << 20

BSQ_OK, BSQ_ERR_ARG, BSQ_ERR_SHAPE, BSQ_ERR_DTYPE, BSQ_ERR_ALIGN = 0, 1, 2, 3, 4
BSQ_ERR_BUFFER_TOO_SMALL, BSQ_ERR_NONFINITE, BSQ_ERR_DEVICE, BSQ_ERR_UNSUPPORTED = 5, 6, 7, 8
BSQ_F32, BSQ_BF16 = 0, 1
DEC_IDENTITY, DEC_LINEAR, DEC_MLP, DEC_MLP_RES1 = 0, 1, 2, 3
PROT_INT8, PROT_E4M3, PROT_E5M2 = 0, 1, 2
ENC_IDENTITY, ENC_LINEAR = 0, 1
OP_ENCODE, OP_GEMV, OP_GEMM, OP_SELECT = 0, 1, 2, 3
DEVERR_NONFINITE, DEVERR_BAD_SET, DEVERR_TIMEOUT, DEVERR_POISONED = 1, 2, 4, 8


class BsqError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_str(status)} (status {status})")
        self.status = status


# ---------------------------------------------------------------- C structs
class bsq_config(ct.Structure):
    _fields_ = [("d", ct.c_int32), ("b", ct.c_int32), ("stages", ct.c_int32), ("dec_kind", ct.c_int32),
                ("hidden", ct.c_int32), ("protect_num", ct.c_int32), ("protect_den", ct.c_int32),
                ("protect_axis", ct.c_int32), ("protect_format", ct.c_int32), ("encoder", ct.c_int32)]


class bsq_decoder(ct.Structure):
    _fields_ = [("W1", ct.c_void_p), ("b1", ct.c_void_p), ("W2", ct.c_void_p), ("b2", ct.c_void_p),
                ("R", ct.c_void_p), ("c", ct.c_void_p), ("E", ct.c_void_p)]


class bsq_layer(ct.Structure):
    _fields_ = [("codes", ct.c_void_p * MAX_STAGES), ("gains", ct.c_void_p * MAX_STAGES),
                ("prot_idx", ct.c_void_p), ("prot_q8", ct.c_void_p), ("prot_scale", ct.c_void_p),
                ("prot_bits", ct.c_void_p),
                ("d_out", ct.c_int64), ("d_in", ct.c_int64), ("pitch", ct.c_int64), ("k", ct.c_int64),
                ("n_mats", ct.c_int64)]


class bsq_lora(ct.Structure):
    _fields_ = [("A", ct.c_void_p), ("B", ct.c_void_p), ("rank", ct.c_int32)]


class bsq_sizes(ct.Structure):
    _fields_ = [("pitch", ct.c_int64), ("k", ct.c_int64), ("chunks", ct.c_int64),
                ("code_plane_bytes", ct.c_int64), ("gain_plane_bytes", ct.c_int64),
                ("idx_bytes", ct.c_int64), ("q8_bytes", ct.c_int64), ("scale_bytes", ct.c_int64),
                ("bits_bytes", ct.c_int64),
                ("S_code", ct.c_double), ("S_dec", ct.c_double), ("S_8bit", ct.c_double),
                ("S_LoRA", ct.c_double), ("S_meta", ct.c_double), ("S_tot", ct.c_double),
                ("bpw_nominal", ct.c_double), ("bpw_real", ct.c_double)]


EXPORTS = ("bsq_version", "bsq_status_str", "bsq_config_check", "bsq_layer_sizes", "bsq_workspace_bytes",
           "bsq_codec_bytes", "bsq_codec_prepare", "bsq_encode", "bsq_decode", "bsq_gemv", "bsq_gemv_prepare",
           "bsq_gemv_run", "bsq_gemm", "bsq_encode_with_set", "bsq_coupled_select",
           "bsq_debug_set_wait_limit", "bsq_decode_stage", "bsq_gemv_noalloc", "bsq_train_param_count",
           "bsq_train_workspace_bytes", "bsq_train_grad", "bsq_train_adam")

# struct layouts above follow this version of include/bsq.h
ABI_VERSION = 8

_lib = None


def lib():
    """Load libbsq.so; raise if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; "
                          f"g.build()'` (the HIP library is the only implementation)")
    L = ct.CDLL(LIB_PATH)
    P, I32, I64, SZ = ct.c_void_p, ct.c_int32, ct.c_int64, ct.c_size_t
    L.bsq_version.restype = I32
    L.bsq_status_str.argtypes = [I32]
    L.bsq_status_str.restype = ct.c_char_p
    L.bsq_config_check.argtypes = [P]
    L.bsq_layer_sizes.argtypes = [P, I64, I64, I32, P]
    L.bsq_workspace_bytes.argtypes = [P, I32, I64, I64, I64, I64, ct.POINTER(SZ)]
    L.bsq_codec_bytes.argtypes = [P, ct.POINTER(SZ)]
    L.bsq_codec_prepare.argtypes = [P, P, P, SZ, P]
    L.bsq_encode.argtypes = [P, P, P, I32, I64, I64, I64, P, P, P, P, SZ, P]
    L.bsq_decode.argtypes = [P, P, P, P, I32, P]
    L.bsq_gemv.argtypes = [P, I32, P, P, P, P, I32, P, I32, P, SZ, P, P]
    L.bsq_gemv_prepare.argtypes = [P, I32, P, P, P, P, I32, P, SZ, P]
    L.bsq_gemv_run.argtypes = [P, I32, P, P, P, P, I32, P, I32, P, SZ, P, P]
    L.bsq_gemm.argtypes = [P, P, P, P, P, I32, I64, I64, P, I32, I64, P, SZ, P, P]
    L.bsq_debug_set_wait_limit.argtypes = [I32]
    L.bsq_decode_stage.argtypes = [P, P, P, I32, I32, P, P]
    L.bsq_gemv_noalloc.argtypes = [P, I32, P, P, P, P, I32, P, I32, I32, P, P]
    L.bsq_encode_with_set.argtypes = [P, P, P, I32, I64, I64, I64, P, P, P, P, SZ, P]
    L.bsq_coupled_select.argtypes = [P, P, P, P, I32, I64, I64, P, P, P, P, P, P, P, SZ, P]
    L.bsq_train_param_count.argtypes = [P, ct.POINTER(I64)]
    L.bsq_train_workspace_bytes.argtypes = [P, I64, ct.POINTER(SZ)]
    L.bsq_train_grad.argtypes = [P, P, P, I32, I64, P, I64, P, P, P, P, P, SZ, P]
    L.bsq_train_adam.argtypes = [P, P, I32, P, P, P, P, P]
    for f in EXPORTS[2:]:
        getattr(L, f).restype = I32
    if L.bsq_version() != ABI_VERSION:
        raise ImportError(f"{LIB_PATH} implements ABI version {L.bsq_version()}, these bindings expect "
                          f"{ABI_VERSION}: rebuild the library")
    _lib = L
    return L


def status_str(status: int) -> str:
    return lib().bsq_status_str(int(status)).decode()


def _check(status: int, what: str):
    if status != BSQ_OK:
        raise BsqError(status, what)


def _ptr(t):
    if t is None:
        return None
    return ct.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ct.c_void_p(stream.cuda_stream)


def _dtype_code(dt) -> int:
    if dt == torch.float32:
        return BSQ_F32
    if dt == torch.bfloat16:
        return BSQ_BF16
    raise TypeError(f"unsupported dtype {dt}")


# ---------------------------------------------------------------- config
@dataclass(frozen=True)
class Config:
    d: int = 8
    stages: int = 2
    kind: int = DEC_MLP
    hidden: int = 8
    protect_num: int = 1
    protect_den: int = 100
    protect_axis: int = 0   # 0: protected input columns, 1: protected output rows
    protect_format: int = PROT_INT8   # payload of the protected slices: int8, FP8-E4M3 or FP8-E5M2
    encoder: int = ENC_IDENTITY       # ENC_LINEAR: each stage codec carries E [b, d]
    codebook_bits: int = 0            # b; 0 means b = d

    @property
    def b(self) -> int:
        return self.codebook_bits or self.d

    def c(self) -> bsq_config:
        return bsq_config(self.d, self.b, self.stages, self.kind, self.hidden, self.protect_num,
                          self.protect_den, self.protect_axis, self.protect_format, self.encoder)

    def k(self, n: int) -> int:
        """ceil(rho * n): protected channels among n."""
        if self.protect_num == 0:
            return 0
        return (n * self.protect_num + self.protect_den - 1) // self.protect_den

    def k_for(self, d_out: int, d_in: int) -> int:
        """Protected slices of a d_out x d_in matrix on this config's axis."""
        return self.k(d_out if self.protect_axis == 1 else d_in)

    def pitch(self, d_in: int) -> int:
        C = d_in // self.d
        return (C + PITCH_ALIGN - 1) // PITCH_ALIGN * PITCH_ALIGN


def bsq_version() -> int:
    return lib().bsq_version()


def bsq_config_check(cfg: Config) -> int:
    c = cfg.c()
    return lib().bsq_config_check(ct.byref(c))


def bsq_layer_sizes(cfg: Config, d_out: int, d_in: int, lora_rank: int = 0) -> dict:
    c, s = cfg.c(), bsq_sizes()
    _check(lib().bsq_layer_sizes(ct.byref(c), d_out, d_in, lora_rank, ct.byref(s)), "bsq_layer_sizes")
    return {name: getattr(s, name) for name, _ in bsq_sizes._fields_}


def bsq_workspace_bytes(cfg: Config, op: int, n_mats: int, d_out: int, d_in: int, M: int = 0) -> int:
    c, out = cfg.c(), ct.c_size_t(0)
    _check(lib().bsq_workspace_bytes(ct.byref(c), op, n_mats, d_out, d_in, M, ct.byref(out)),
           "bsq_workspace_bytes")
    return out.value


def bsq_codec_bytes(cfg: Config) -> int:
    c, out = cfg.c(), ct.c_size_t(0)
    _check(lib().bsq_codec_bytes(ct.byref(c), ct.byref(out)), "bsq_codec_bytes")
    return out.value


# ---------------------------------------------------------------- codec
@dataclass
class Codec:
    """Prepared decoder tables of one category (device buffer) plus the
    device copies of the decoder parameters they were built from."""
    cfg: Config
    buf: torch.Tensor
    params: list = field(default_factory=list)

    def ptr(self):
        return self.buf.data_ptr()


def _empty_aligned(nbytes: int, device, align: int = 256, zero: bool = False) -> torch.Tensor:
    """A uint8 device buffer whose data pointer is `align`-byte aligned."""
    t = (torch.zeros if zero else torch.empty)(nbytes + align, dtype=torch.uint8, device=device)
    off = (-t.data_ptr()) % align
    return t[off:off + nbytes]


def bsq_codec_prepare(cfg: Config, decoders, device="cuda", stream=None) -> Codec:
    """decoders: per stage an object with W1/b1/W2/b2 and, for the residual-block
    decoder, R/c (numpy or torch, fp32; None or absent where unused)."""
    dev = torch.device(device)
    params = []
    arr = (bsq_decoder * MAX_STAGES)()
    for s in range(cfg.stages):
        dec = decoders[s] if decoders is not None else None
        ts = []
        for name in ("W1", "b1", "W2", "b2", "R", "c", "E"):
            v = getattr(dec, name, None) if dec is not None else None
            if v is None:
                ts.append(None)
                continue
            t = torch.as_tensor(v, dtype=torch.float32).contiguous().to(dev)
            ts.append(t)
        params.append(ts)
        arr[s] = bsq_decoder(*[None if t is None else t.data_ptr() for t in ts])
    buf = _empty_aligned(bsq_codec_bytes(cfg), dev)
    c = cfg.c()
    _check(lib().bsq_codec_prepare(ct.byref(c), arr, _ptr(buf), buf.numel(), _stream(stream)),
           "bsq_codec_prepare")
    return Codec(cfg, buf, params)


# ---------------------------------------------------------------- layers
@dataclass
class Layer:
    """Encoded matrix (or stack of n_mats): torch tensors holding the planes."""
    cfg: Config
    codes: list
    gains: list
    idx: torch.Tensor | None
    q8: torch.Tensor | None
    scale: torch.Tensor | None
    d_out: int
    d_in: int
    n_mats: int = 1
    bits: torch.Tensor | None = None  # protected-column bitmap, int32 [.., pitch * d / 32]

    @property
    def pitch(self) -> int:
        return self.cfg.pitch(self.d_in)

    @property
    def k(self) -> int:
        return self.cfg.k_for(self.d_out, self.d_in)

    def c(self) -> bsq_layer:
        L = bsq_layer()
        for s in range(self.cfg.stages):
            L.codes[s] = self.codes[s].data_ptr()
            L.gains[s] = self.gains[s].data_ptr()
        if self.k > 0:
            L.prot_idx = self.idx.data_ptr()
            L.prot_q8 = self.q8.data_ptr()
            L.prot_scale = self.scale.data_ptr()
            if self.bits is not None:
                L.prot_bits = self.bits.data_ptr()
        L.d_out, L.d_in, L.pitch, L.k, L.n_mats = self.d_out, self.d_in, self.pitch, self.k, self.n_mats
        return L

    @property
    def row_groups(self) -> int:
        return (self.d_out + 63) // 64

    def rowmajor(self, plane):
        """A tiled plane [.., RG, pitch/16, 64, 16] as row-major [.., d_out, pitch]
        (a view change for comparisons and host tools; no arithmetic)."""
        lead = plane.shape[:-4]
        t = plane.transpose(-3, -2).reshape(*lead, self.row_groups * 64, self.pitch)
        return t[..., :self.d_out, :]

    def mat(self, m: int) -> "Layer":
        """Matrix m of a stack, as a single-matrix layer (views, no copy)."""
        if self.n_mats == 1:
            return self
        k = self.k
        return Layer(self.cfg, [c[m] for c in self.codes], [g[m] for g in self.gains],
                     None if k == 0 else self.idx[m], None if k == 0 else self.q8[m],
                     None if k == 0 else self.scale[m], self.d_out, self.d_in, 1,
                     None if (k == 0 or self.bits is None) else self.bits[m])

    def nbytes_streamed(self) -> int:
        """Bytes a product reads from this layer: the code and gain planes of
        the d_out real rows, the protected payload, scales, indices and bitmap."""
        per_row = self.pitch * (self.codes[0].element_size() + 2) * self.cfg.stages
        n = per_row * self.d_out
        if self.k and self.cfg.protect_axis == 1:
            n += self.q8.numel() + self.scale.numel() * 4 + self.idx.numel() * 4
        elif self.k:
            n += self.d_out * self.k + self.scale.numel() * 4 + self.idx.numel() * 4
            if self.bits is not None:
                n += self.bits.numel() * 4
        return n


def layer_empty(cfg: Config, d_out: int, d_in: int, n_mats: int = 1, device="cuda") -> Layer:
    """Planes in the tiled layout [n_mats][ceil(d_out/64)][pitch/16][64][16];
    the protected payload (one byte per element) as [n_mats][d_out][roundup(k, 16)] (protected rows:
    [n_mats][k][roundup(d_in, 16)], and no bitmap)."""
    P, k = cfg.pitch(d_in), cfg.k_for(d_out, d_in)
    ct_ = torch.uint8 if cfg.b <= 8 else torch.int16
    tiles = ((d_out + 63) // 64, P // 16, 64, 16)
    shape = ((n_mats,) + tiles) if n_mats > 1 else tiles
    codes = [torch.empty(shape, dtype=ct_, device=device) for _ in range(cfg.stages)]
    gains = [torch.empty(shape, dtype=torch.float16, device=device) for _ in range(cfg.stages)]
    idx = q8 = scale = bits = None
    if k > 0:
        lead = (n_mats,) if n_mats > 1 else ()
        idx = torch.empty(lead + (k,), dtype=torch.int32, device=device)
        scale = torch.empty(lead + (k,), dtype=torch.float32, device=device)
        if cfg.protect_axis == 1:
            q8 = torch.empty(lead + (k, (d_in + 15) // 16 * 16), dtype=torch.int8, device=device)
        else:
            q8 = torch.empty(lead + (d_out, (k + 15) // 16 * 16), dtype=torch.int8, device=device)
            bits = torch.empty(lead + (P * cfg.d // 32,), dtype=torch.int32, device=device)
    return Layer(cfg, codes, gains, idx, q8, scale, d_out, d_in, n_mats, bits)


def bsq_encode(cfg: Config, codec: Codec, W: torch.Tensor, g: torch.Tensor | None = None,
               out: Layer | None = None, ws: torch.Tensor | None = None, err: torch.Tensor | None = None,
               check: bool = True, stream=None) -> Layer:
    """Encode W [d_out, d_in] or a stack [n_mats, d_out, d_in] (bf16 or fp32, on the GPU)."""
    if W.dim() == 2:
        n_mats, (d_out, d_in) = 1, W.shape
    elif W.dim() == 3:
        n_mats, d_out, d_in = W.shape
    else:
        raise ValueError("W must be 2-D or 3-D")
    W = W.contiguous()
    dev = W.device
    out = out or layer_empty(cfg, d_out, d_in, n_mats, dev)
    need = bsq_workspace_bytes(cfg, OP_ENCODE, n_mats, d_out, d_in)
    ws = ws if ws is not None else _empty_aligned(need, dev)
    own_err = err is None
    err = err if err is not None else torch.zeros(1, dtype=torch.int32, device=dev)
    c, L = cfg.c(), out.c()
    gp = None if g is None else _ptr(g.contiguous().to(torch.float32))
    _check(lib().bsq_encode(ct.byref(c), ct.c_void_p(codec.ptr()), _ptr(W), _dtype_code(W.dtype), n_mats, d_out,
                            d_in, gp, ct.byref(L), _ptr(err), _ptr(ws), ws.numel(), _stream(stream)),
           "bsq_encode")
    if check and own_err:
        if int(err.item()) & 1:
            raise BsqError(BSQ_ERR_NONFINITE, "bsq_encode")
    return out


def bsq_encode_with_set(cfg: Config, codec: Codec, W: torch.Tensor, idx: torch.Tensor, out: Layer | None = None,
                        ws: torch.Tensor | None = None, err: torch.Tensor | None = None, check: bool = True,
                        stream=None) -> Layer:
    """Encode W with a given protected set idx (int32 [k] or [n_mats, k], ascending)
    on cfg.protect_axis: columns (axis 0) or rows (axis 1)."""
    if W.dim() == 2:
        n_mats, (d_out, d_in) = 1, W.shape
    elif W.dim() == 3:
        n_mats, d_out, d_in = W.shape
    else:
        raise ValueError("W must be 2-D or 3-D")
    W = W.contiguous()
    dev = W.device
    out = out or layer_empty(cfg, d_out, d_in, n_mats, dev)
    need = bsq_workspace_bytes(cfg, OP_ENCODE, n_mats, d_out, d_in)
    ws = ws if ws is not None else _empty_aligned(need, dev)
    own_err = err is None
    err = err if err is not None else torch.zeros(1, dtype=torch.int32, device=dev)
    idx = idx.to(device=dev, dtype=torch.int32).contiguous()
    if idx.numel() != n_mats * out.k:
        raise ValueError(f"idx holds {idx.numel()} entries, the layout needs {n_mats} x {out.k}")
    c, L = cfg.c(), out.c()
    _check(lib().bsq_encode_with_set(ct.byref(c), ct.c_void_p(codec.ptr()), _ptr(W), _dtype_code(W.dtype), n_mats,
                                     d_out, d_in, _ptr(idx) if idx.numel() else None, ct.byref(L), _ptr(err),
                                     _ptr(ws), ws.numel(), _stream(stream)), "bsq_encode_with_set")
    if check and own_err:
        e = int(err.item())
        if e & 1:
            raise BsqError(BSQ_ERR_NONFINITE, "bsq_encode_with_set")
        if e & 2:
            raise BsqError(BSQ_ERR_ARG, "bsq_encode_with_set (protected set not ascending or out of range)")
    return out


def bsq_coupled_select(cfg: Config, W_gate: torch.Tensor, W_up: torch.Tensor, W_down: torch.Tensor,
                       g_gate=None, g_up=None, g_down=None, with_scores: bool = False, check: bool = True,
                       stream=None):
    """Coupled MLP intermediate-channel set (eq. mlp_coupled_protection): int32
    [ceil(rho d_ffn)] ascending, and with_scores the fp64 scores [d_ffn]."""
    d_ffn, d_model = W_gate.shape
    if tuple(W_up.shape) != (d_ffn, d_model) or tuple(W_down.shape) != (d_model, d_ffn):
        raise ValueError("W_gate, W_up must be [d_ffn, d_model] and W_down [d_model, d_ffn]")
    if not (W_gate.dtype == W_up.dtype == W_down.dtype):
        raise TypeError("the three matrices must share one dtype")
    dev = W_gate.device
    Wg, Wu, Wd = (t.contiguous() for t in (W_gate, W_up, W_down))
    k = cfg.k(d_ffn)
    idx = torch.empty(max(k, 1), dtype=torch.int32, device=dev)
    scores = torch.empty(d_ffn, dtype=torch.float64, device=dev) if with_scores else None
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ws = _empty_aligned(bsq_workspace_bytes(cfg, OP_SELECT, 1, d_ffn, d_model), dev)
    gs = [None if g is None else g.to(device=dev, dtype=torch.float32).contiguous() for g in (g_gate, g_up, g_down)]
    c = cfg.c()
    _check(lib().bsq_coupled_select(ct.byref(c), _ptr(Wg), _ptr(Wu), _ptr(Wd), _dtype_code(Wg.dtype), d_model,
                                    d_ffn, *[_ptr(g) for g in gs], _ptr(idx), _ptr(scores), _ptr(err), _ptr(ws),
                                    ws.numel(), _stream(stream)), "bsq_coupled_select")
    if check and int(err.item()) & 1:
        raise BsqError(BSQ_ERR_NONFINITE, "bsq_coupled_select")
    idx = idx[:k]
    return (idx, scores) if with_scores else idx


def bsq_decode(cfg: Config, codec: Codec, layer: Layer, dtype=torch.float32, out: torch.Tensor | None = None,
               stream=None) -> torch.Tensor:
    dev = layer.codes[0].device
    shape = (layer.n_mats, layer.d_out, layer.d_in) if layer.n_mats > 1 else (layer.d_out, layer.d_in)
    out = out if out is not None else torch.empty(shape, dtype=dtype, device=dev)
    c, L = cfg.c(), layer.c()
    _check(lib().bsq_decode(ct.byref(c), ct.c_void_p(codec.ptr()), ct.byref(L), _ptr(out), _dtype_code(out.dtype),
                            _stream(stream)), "bsq_decode")
    return out


def bsq_decode_stage(cfg: Config, codec: Codec, layer: Layer, stage: int, accumulate: bool, out: torch.Tensor,
                     stream=None) -> torch.Tensor:
    """One residual stage of a sequential decode into the fp32 `out`
    (bsq_decode_stage); stages 0 .. S-1, accumulating from stage 1, give the
    bits of bsq_decode."""
    c, L = cfg.c(), layer.c()
    _check(lib().bsq_decode_stage(ct.byref(c), ct.c_void_p(codec.ptr()), ct.byref(L), int(stage), int(accumulate),
                                  _ptr(out), _stream(stream)), "bsq_decode_stage")
    return out


def _lora_struct(lora) -> bsq_lora:
    if lora is None:
        return bsq_lora(None, None, 0)
    A, B = lora
    return bsq_lora(A.data_ptr(), B.data_ptr(), int(A.shape[0]))


class GemvPlan:
    """Marshalled arguments of one grouped bsq_gemv call, reusable across
    calls (and inside a HIP-graph capture) with the same buffers."""

    def __init__(self, cfg: Config, codecs, layers, x: torch.Tensor, loras=None, y_dtype=torch.bfloat16,
                 out=None, ws=None, err=None):
        n = len(layers)
        if not (1 <= n <= MAX_GROUP) or len(codecs) != n:
            raise ValueError("group size must be 1..8 with one codec per layer")
        dev = x.device
        self.cfg, self.n, self.x = cfg, n, x
        self.layers, self.codecs, self.loras = layers, codecs, loras
        self.out = out if out is not None else [torch.empty(L.d_out, dtype=y_dtype, device=dev) for L in layers]
        need = bsq_workspace_bytes(cfg, OP_GEMV, n, max(L.d_out for L in layers), layers[0].d_in)
        # zero-filled once: the kernels leave their flagged slots at zero
        self.ws = ws if ws is not None else _empty_aligned(need, dev, zero=True)
        self.err = err  # device int32 error word (TIMEOUT / POISONED bits), or None
        self._c = cfg.c()
        self._codecs = (ct.c_void_p * n)(*[cd.ptr() for cd in codecs])
        self._layers = (bsq_layer * n)(*[L.c() for L in layers])
        self._loras = None if loras is None else (bsq_lora * n)(*[_lora_struct(l) for l in loras])
        self._y = (ct.c_void_p * n)(*[t.data_ptr() for t in self.out])
        self._xd = _dtype_code(x.dtype)
        self._yd = _dtype_code(self.out[0].dtype)

    def __call__(self, stream=None):
        _check(lib().bsq_gemv(ct.byref(self._c), self.n, self._codecs, self._layers, self._loras, _ptr(self.x),
                              self._xd, self._y, self._yd, _ptr(self.ws), self.ws.numel(), _ptr(self.err),
                              _stream(stream)), "bsq_gemv")
        return self.out

    def prepare(self, stream=None):
        """bsq_gemv_prepare: the LoRA vectors A x and, for the d = 16 symmetric
        decoder, the folded activations (no launch when neither applies)."""
        _check(lib().bsq_gemv_prepare(ct.byref(self._c), self.n, self._codecs, self._layers, self._loras,
                                      _ptr(self.x), self._xd, _ptr(self.ws), self.ws.numel(), _stream(stream)),
               "bsq_gemv_prepare")

    def run(self, stream=None):
        """bsq_gemv_run: the streaming product over the prepared workspace."""
        _check(lib().bsq_gemv_run(ct.byref(self._c), self.n, self._codecs, self._layers, self._loras,
                                  _ptr(self.x), self._xd, self._y, self._yd, _ptr(self.ws), self.ws.numel(),
                                  _ptr(self.err), _stream(stream)), "bsq_gemv_run")
        return self.out


def bsq_gemv(cfg: Config, codecs, layers, x: torch.Tensor, loras=None, y_dtype=torch.bfloat16, out=None,
             ws=None, stream=None, err=None):
    """Grouped fused decode-GEMV: returns [W_hat_g x + B_g A_g x for each layer g]."""
    if isinstance(layers, Layer):
        layers, codecs = [layers], [codecs]
        loras = None if loras is None else [loras]
        single = True
    else:
        single = False
    plan = GemvPlan(cfg, codecs, layers, x.contiguous(), loras, y_dtype, out, ws, err)
    ys = plan(stream)
    return ys[0] if single else ys


def bsq_gemv_noalloc(cfg: Config, codecs, layers, x: torch.Tensor, loras=None, y_dtype=torch.bfloat16, out=None,
                     clear_scratch=False, err=None, stream=None):
    """bsq_gemv on the library's own scratch array (bsq_gemv_noalloc): no
    workspace argument, nothing allocated by the call (outputs are allocated
    here unless `out` is given)."""
    single = isinstance(layers, Layer)
    if single:
        layers, codecs = [layers], [codecs]
        loras = None if loras is None else [loras]
    n = len(layers)
    dev = x.device
    outs = out if out is not None else [torch.empty(L.d_out, dtype=y_dtype, device=dev) for L in layers]
    c = cfg.c()
    cds = (ct.c_void_p * n)(*[cd.ptr() for cd in codecs])
    lys = (bsq_layer * n)(*[L.c() for L in layers])
    los = None if loras is None else (bsq_lora * n)(*[_lora_struct(l) for l in loras])
    ys = (ct.c_void_p * n)(*[t.data_ptr() for t in outs])
    _check(lib().bsq_gemv_noalloc(ct.byref(c), n, cds, lys, los, _ptr(x), _dtype_code(x.dtype), ys,
                                  _dtype_code(outs[0].dtype), int(bool(clear_scratch)), _ptr(err), _stream(stream)),
           "bsq_gemv_noalloc")
    return outs[0] if single else outs


def bsq_gemm(cfg: Config, codec: Codec, layer: Layer, X: torch.Tensor, lora=None, y_dtype=torch.bfloat16,
             out=None, ws=None, stream=None, err=None) -> torch.Tensor:
    """Fused decode-GEMM: Y = X W_hat^T + (X A^T) B^T for X [M, d_in] bf16."""
    M, d_in = X.shape
    dev = X.device
    out = out if out is not None else torch.empty((M, layer.d_out), dtype=y_dtype, device=dev)
    need = bsq_workspace_bytes(cfg, OP_GEMM, 1, layer.d_out, d_in, M)
    ws = ws if ws is not None else _empty_aligned(need, dev, zero=True)
    c, L = cfg.c(), layer.c()
    lo = _lora_struct(lora)
    _check(lib().bsq_gemm(ct.byref(c), ct.c_void_p(codec.ptr()), ct.byref(L), ct.byref(lo), _ptr(X),
                          _dtype_code(X.dtype), M, X.stride(0), _ptr(out), _dtype_code(out.dtype), out.stride(0),
                          _ptr(ws), ws.numel(), _ptr(err), _stream(stream)), "bsq_gemm")
    return out


def bsq_debug_set_wait_limit(polls: int) -> int:
    """Testing aid (bsq_debug_set_wait_limit): polls before a product's
    finishing workgroup gives up waiting; 0 forces every such wait to give
    up, a negative value restores the default. Returns the previous value."""
    return int(lib().bsq_debug_set_wait_limit(int(polls)))


# ---------------------------------------------------------------- codec training
class bsq_train_hparams(ct.Structure):
    _fields_ = [(n, ct.c_float) for n in ("lambda_c", "lambda_e", "gamma", "tau", "lr", "beta1", "beta2", "eps")]


@dataclass(frozen=True)
class TrainHyper:
    """Codec-training hyperparameters (bsq_train_hparams)."""
    lambda_c: float = 0.25
    lambda_e: float = 0.1
    gamma: float = 1.0
    tau: float = 1.0
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8

    def c(self) -> bsq_train_hparams:
        return bsq_train_hparams(self.lambda_c, self.lambda_e, self.gamma, self.tau, self.lr, self.beta1,
                                 self.beta2, self.eps)


def bsq_train_param_count(cfg: Config) -> int:
    out = ct.c_int64()
    c = cfg.c()
    _check(lib().bsq_train_param_count(ct.byref(c), ct.byref(out)), "bsq_train_param_count")
    return out.value


def bsq_train_workspace_bytes(cfg: Config, n: int) -> int:
    out = ct.c_size_t()
    c = cfg.c()
    _check(lib().bsq_train_workspace_bytes(ct.byref(c), n, ct.byref(out)), "bsq_train_workspace_bytes")
    return out.value


def bsq_train_grad(cfg: Config, hp: TrainHyper, chunks, theta, idx=None, n=None, grad=None, loss=None, err=None,
                   ws=None, stream=None):
    """Loss [4] (L, L_rec, L_com, L_ent) and gradient [P] of one mini-batch.
    chunks: a device tensor (fp32 or bf16) whose elements are the category's
    chunks back to back (any shape with numel a multiple of d); idx: device
    int64 chunk indices or None for the first n chunks."""
    dev = chunks.device
    x_dtype = BSQ_BF16 if chunks.dtype == torch.bfloat16 else BSQ_F32
    n_total = chunks.numel() // cfg.d
    if n is None:
        n = idx.numel() if idx is not None else n_total
    P = bsq_train_param_count(cfg)
    grad = torch.empty(P, dtype=torch.float32, device=dev) if grad is None else grad
    loss = torch.empty(4, dtype=torch.float32, device=dev) if loss is None else loss
    if ws is None:
        ws = _empty_aligned(bsq_train_workspace_bytes(cfg, n), dev)
    c, h = cfg.c(), hp.c()
    _check(lib().bsq_train_grad(ct.byref(c), ct.byref(h), _ptr(chunks), x_dtype, n_total, _ptr(idx), n, _ptr(theta),
                                _ptr(grad), _ptr(loss), _ptr(err), _ptr(ws), ws.numel(), _stream(stream)),
           "bsq_train_grad")
    return loss, grad


def bsq_train_adam(cfg: Config, hp: TrainHyper, step: int, theta, grad, m, v, stream=None):
    c, h = cfg.c(), hp.c()
    _check(lib().bsq_train_adam(ct.byref(c), ct.byref(h), step, _ptr(theta), _ptr(grad), _ptr(m), _ptr(v),
                                _stream(stream)), "bsq_train_adam")
