"""CPU oracle for the BSQ weight codec (BiSCo-LLM, Section III) and its
matrix-vector / matrix-matrix products.

TEST INFRASTRUCTURE ONLY: only tests/, __graft_entry__.smoke() and the
benchmark's cpu_baseline leg may import this package. It shares no code with
the HIP library (paper_2607_08643_amd) and never imports it.

The encoder, decoder assembly and fused product route live in plain C
(bsq_oracle.c, fp32 canonical order, fmaf chains, no contraction); this module
adds the fp64 dense product route (decode, then an fp64 matmul), the storage
accounting of eq. real_size, and numpy marshalling.

Parity pins (tests/test_oracle_pins.py): unit-norm codes, nearest-vertex sign
rule by brute force, pack/unpack round trip, residual non-increase, closed form
of the identity decoder, least-squares gains against numpy lstsq, MLP special
cases that reduce to known maps, Q8 bounds, TopK on planted outliers, binary16
rounding against numpy, the paper's rate arithmetic, and agreement of the two
product routes. Output-row and coupled MLP protection
(tests/test_oracle_protection_axes.py): the coupled score on rows and columns
with exact integer norms, ties, reductions to the single-matrix selections,
row keys and row Q8 as the column versions of the transpose, and bit-identity
of the coded rows with the unprotected encoding. Trained-codec quality (PPL,
accuracy) is parity unpinned: the paper publishes no decoder weights.
"""
from __future__ import annotations

import ctypes as ct
import math
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "bsq_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

KIND_IDENTITY, KIND_LINEAR, KIND_MLP, KIND_MLP_RES1 = 0, 1, 2, 3
FMT_INT8, FMT_E4M3, FMT_E5M2 = 0, 1, 2   # protected payload formats
ENC_IDENTITY, ENC_LINEAR = 0, 1          # encoder E: z = r (b = d), or z = E r with E [b][d]
ORC_OK, ORC_ERR_ARG, ORC_ERR_NONFINITE = 0, 1, 6
PITCH_ALIGN = 16  # rows of the code/gain planes are padded to 16 chunks


class OracleError(RuntimeError):
    pass


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (no contraction, no fast-math)."""
    if not force and os.path.exists(LIB):
        return LIB
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
           "-fno-fast-math", "-fopenmp", "-Wall", "-Werror", SRC, "-o", LIB + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ct.CDLL(LIB)
        P, I64, I32 = ct.c_void_p, ct.c_int64, ct.c_int
        L.orc_f32_to_f16.argtypes = [ct.c_float]
        L.orc_f32_to_f16.restype = ct.c_uint16
        L.orc_f16_to_f32.argtypes = [ct.c_uint16]
        L.orc_f16_to_f32.restype = ct.c_float
        L.orc_gain_to_f16.argtypes = [ct.c_float]
        L.orc_gain_to_f16.restype = ct.c_uint16
        L.orc_code_scale.argtypes = [I32]
        L.orc_code_scale.restype = ct.c_float
        L.orc_decoder_eval.argtypes = [I32, I32, I32, I32, P, P, P, P, P, P, ct.c_uint32, P]
        L.orc_decoder_table.argtypes = [I32, I32, I32, I32, P, P, P, P, P, P, P]
        L.orc_payload_max.argtypes = [I32]
        L.orc_payload_max.restype = ct.c_float
        L.orc_payload_value.argtypes = [ct.c_uint8, I32]
        L.orc_payload_value.restype = ct.c_float
        L.orc_payload_quant.argtypes = [ct.c_float, I32]
        L.orc_payload_quant.restype = ct.c_uint8
        L.orc_column_keys.argtypes = [P, I64, I64, P, P]
        L.orc_protect_select.argtypes = [P, I64, I64, P, I64, P, P]
        L.orc_q8.argtypes = [P, I64, I64, P, I64, I32, P, P]
        L.orc_encode.argtypes = [I32, I32, I32, P, P, P, I64, I64, P, I64, I64, I32, P, P, P, P, P, I32]
        L.orc_decode.argtypes = [I32, I32, I32, P, I64, I64, I64, P, P, P, P, P, I64, I32, P, I32]
        L.orc_gemv_fused.argtypes = [I32, I32, I32, P, I64, I64, I64, P, P, P, P, P, I64, I32,
                                     P, I32, P, P, P, I32]
        L.orc_topk.argtypes = [P, I64, I64, P]
        L.orc_row_keys.argtypes = [P, I64, I64, P, P]
        L.orc_coupled_select.argtypes = [P, P, P, I64, I64, P, P, P, I64, P, P]
        L.orc_q8_rows.argtypes = [P, I64, I64, P, I64, I32, P, P]
        L.orc_encode_set.argtypes = [I32, I32, I32, P, P, P, I64, I64, I32, P, I64, I64, I32, P, P, P, P, I32]
        L.orc_max_threads.restype = I32
        L.orc_train_decisions.argtypes = [I32, I32, I32, P, P, P, P, I64, P, P]
        for f in ("orc_decoder_eval", "orc_decoder_table", "orc_protect_select",
                  "orc_encode", "orc_decode", "orc_gemv_fused", "orc_topk", "orc_coupled_select",
                  "orc_encode_set"):
            getattr(L, f).restype = I32
        _lib = L
    return _lib


def _p(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ct.c_void_p)


def _ptr_array(arrs):
    return (ct.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])


def _encoders(cfg, decs):
    """With cfg.encoder == ENC_LINEAR: per stage the encoder E [b][d] (fp32,
    the attribute E of the stage codec object) and the pointer array the C
    oracle takes; with the identity encoder (b = d): None."""
    if cfg.encoder == ENC_IDENTITY:
        if cfg.b != cfg.d:
            raise OracleError("b != d needs the linear encoder")
        return None, None
    es = [None if getattr(dec, "E", None) is None else _f32(dec.E) for dec in decs[:cfg.stages]]
    if any(e is None or e.shape != (cfg.b, cfg.d) for e in es):
        raise OracleError("every stage needs an encoder E of shape [b][d]")
    return es, _ptr_array(es)


def _check(rc: int, what: str):
    if rc == ORC_ERR_NONFINITE:
        raise OracleError(f"{what}: non-finite input")
    if rc != ORC_OK:
        raise OracleError(f"{what}: error {rc}")


# --------------------------------------------------------------------------
@dataclass(frozen=True)
class Config:
    d: int = 8
    b: int = 8
    stages: int = 2
    kind: int = KIND_MLP
    hidden: int = 8
    protect_num: int = 1
    protect_den: int = 100
    protect_axis: int = 0   # 0: input columns, 1: output rows
    protect_format: int = FMT_INT8  # payload of the protected slices
    encoder: int = ENC_IDENTITY     # ENC_LINEAR: each stage codec carries E [b][d]

    def k(self, d_in: int) -> int:
        """k = ceil(rho * n), rho = num/den, in integer arithmetic, for n
        channels on the protected axis."""
        if self.protect_num == 0:
            return 0
        return (d_in * self.protect_num + self.protect_den - 1) // self.protect_den

    def k_for(self, d_out: int, d_in: int) -> int:
        """Protected slices of a d_out x d_in matrix on this config's axis."""
        return self.k(d_out if self.protect_axis == 1 else d_in)


def pitch(d_in: int, d: int) -> int:
    C = d_in // d
    return (C + PITCH_ALIGN - 1) // PITCH_ALIGN * PITCH_ALIGN


@dataclass
class Encoded:
    codes: list          # per stage: uint8/uint16 [d_out, pitch]
    gains: list          # per stage: uint16 (fp16 bits) [d_out, pitch]
    idx: np.ndarray      # int32 [k]
    q8: np.ndarray       # payload bytes (int8 view) [d_out, k] (axis 0) or [k, d_in] (axis 1)
    scale: np.ndarray    # fp32 [k]
    pitch: int = 0
    d_out: int = 0
    d_in: int = 0
    axis: int = 0        # 0: protected input columns, 1: protected output rows


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def _dec_params(dec):
    """W1, b1, W2, b2, R, c of one stage decoder as fp32 arrays (None where
    the decoder object has no such tensor; R and c only for the res1 kind)."""
    vals = (dec.W1, dec.b1, dec.W2, dec.b2, getattr(dec, "R", None), getattr(dec, "c", None))
    return tuple(None if v is None else _f32(v) for v in vals)


def decoder_eval(cfg: Config, dec, code: int) -> np.ndarray:
    y = np.zeros(cfg.d, dtype=np.float32)
    W1, b1, W2, b2, R, c = _dec_params(dec)
    rc = lib().orc_decoder_eval(cfg.kind, cfg.d, cfg.b, cfg.hidden, _p(W1), _p(b1), _p(W2),
                                _p(b2), _p(R), _p(c), code, _p(y))
    _check(rc, "decoder_eval")
    return y


def decoder_table(cfg: Config, decs) -> list:
    out = []
    for dec in decs[:cfg.stages]:
        t = np.zeros((1 << cfg.b, cfg.d), dtype=np.float32)
        W1, b1, W2, b2, R, c = _dec_params(dec)
        rc = lib().orc_decoder_table(cfg.kind, cfg.d, cfg.b, cfg.hidden, _p(W1), _p(b1),
                                     _p(W2), _p(b2), _p(R), _p(c), _p(t))
        _check(rc, "decoder_table")
        out.append(t)
    return out


def column_keys(w: np.ndarray, g=None) -> np.ndarray:
    w = _f32(w)
    d_out, d_in = w.shape
    key = np.zeros(d_in, dtype=np.float64)
    g = None if g is None else _f32(g)
    lib().orc_column_keys(_p(w), d_out, d_in, _p(g), _p(key))
    return key


def protect_select(w: np.ndarray, k: int, g=None) -> np.ndarray:
    w = _f32(w)
    d_out, d_in = w.shape
    idx = np.zeros(max(k, 1), dtype=np.int32)
    g = None if g is None else _f32(g)
    _check(lib().orc_protect_select(_p(w), d_out, d_in, _p(g), k, _p(idx), None), "protect_select")
    return idx[:k].copy()


def topk(key: np.ndarray, k: int) -> np.ndarray:
    key = np.ascontiguousarray(key, dtype=np.float64)
    idx = np.zeros(max(k, 1), dtype=np.int32)
    _check(lib().orc_topk(_p(key), len(key), k, _p(idx)), "topk")
    return idx[:k].copy()


def row_keys(w: np.ndarray, g=None) -> np.ndarray:
    w = _f32(w)
    d_out, d_in = w.shape
    key = np.zeros(d_out, dtype=np.float64)
    g = None if g is None else _f32(g)
    lib().orc_row_keys(_p(w), d_out, d_in, _p(g), _p(key))
    return key


def coupled_select(w_gate, w_up, w_down, k: int, g_gate=None, g_up=None, g_down=None):
    """Coupled MLP intermediate-channel set (eq. mlp_coupled_protection):
    (idx ascending [k], score fp64 [d_ffn])."""
    wg, wu, wd = _f32(w_gate), _f32(w_up), _f32(w_down)
    d_ffn, d_model = wg.shape
    if wu.shape != (d_ffn, d_model) or wd.shape != (d_model, d_ffn):
        raise OracleError("coupled_select: shapes")
    idx = np.zeros(max(k, 1), dtype=np.int32)
    score = np.zeros(max(d_ffn, 1), dtype=np.float64)
    gs = [None if v is None else _f32(v) for v in (g_gate, g_up, g_down)]
    _check(lib().orc_coupled_select(_p(wg), _p(wu), _p(wd), d_model, d_ffn, _p(gs[0]), _p(gs[1]),
                                    _p(gs[2]), k, _p(idx), _p(score)), "coupled_select")
    return idx[:k].copy(), score[:d_ffn].copy()


def payload_max(fmt: int = FMT_INT8) -> float:
    return float(lib().orc_payload_max(fmt))


def payload_value(q: int, fmt: int = FMT_INT8) -> float:
    """The value of one stored protected byte (0..255) in format fmt."""
    return float(lib().orc_payload_value(int(q) & 0xFF, fmt))


def payload_quant(v: float, fmt: int = FMT_INT8) -> int:
    """The stored byte (0..255) of the scaled value v in format fmt."""
    return int(lib().orc_payload_quant(float(v), fmt))


def payload_values(q: np.ndarray, fmt: int = FMT_INT8) -> np.ndarray:
    """fp32 values of an array of stored bytes (any integer dtype of 8 bits)."""
    table = np.array([payload_value(v, fmt) for v in range(256)], dtype=np.float32)
    return table[np.asarray(q).view(np.uint8)]


def q8_rows(w: np.ndarray, idx: np.ndarray, fmt: int = FMT_INT8):
    w = _f32(w)
    d_out, d_in = w.shape
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    k = len(idx)
    q = np.zeros((max(k, 1), d_in), dtype=np.int8)
    s = np.zeros(max(k, 1), dtype=np.float32)
    lib().orc_q8_rows(_p(w), d_out, d_in, _p(idx), k, fmt, _p(q), _p(s))
    return q[:k].copy(), s[:k].copy()


def q8(w: np.ndarray, idx: np.ndarray, fmt: int = FMT_INT8):
    w = _f32(w)
    d_out, d_in = w.shape
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    k = len(idx)
    q = np.zeros((d_out, max(k, 1)), dtype=np.int8)
    s = np.zeros(max(k, 1), dtype=np.float32)
    lib().orc_q8(_p(w), d_out, d_in, _p(idx), k, fmt, _p(q), _p(s))
    return q[:, :k].copy(), s[:k].copy()


def encode(cfg: Config, decs, w: np.ndarray, g=None, nthreads: int = 0,
           tables=None) -> Encoded:
    """Encode one fp32 matrix w [d_out, d_in] (bf16 inputs: convert exactly first).
    With protect_axis = 1 the protected slices are the output rows of largest
    energy (row_keys, g per output row), encoded by encode_set."""
    w = _f32(w)
    d_out, d_in = w.shape
    if d_in % cfg.d:
        raise OracleError("d_in must be a multiple of d")
    if cfg.protect_axis == 1:
        idx = topk(row_keys(w, g), cfg.k(d_out))
        return encode_set(cfg, decs, w, idx, nthreads=nthreads, tables=tables)
    P = pitch(d_in, cfg.d)
    k = cfg.k(d_in)
    tables = tables or decoder_table(cfg, decs)
    es, enc_arr = _encoders(cfg, decs)
    ctype = np.uint8 if cfg.b <= 8 else np.uint16
    codes = [np.zeros((d_out, P), dtype=ctype) for _ in range(cfg.stages)]
    gains = [np.zeros((d_out, P), dtype=np.uint16) for _ in range(cfg.stages)]
    idx = np.zeros(max(k, 1), dtype=np.int32)
    q = np.zeros((d_out, max(k, 1)), dtype=np.int8)
    s = np.zeros(max(k, 1), dtype=np.float32)
    g = None if g is None else _f32(g)
    rc = lib().orc_encode(cfg.d, cfg.b, cfg.stages, _ptr_array(tables), enc_arr, _p(w), d_out, d_in, _p(g), k, P,
                          cfg.protect_format, _ptr_array(codes), _ptr_array(gains), _p(idx), _p(q), _p(s), nthreads)
    _check(rc, "encode")
    return Encoded(codes, gains, idx[:k].copy(), np.ascontiguousarray(q[:, :k]), s[:k].copy(),
                   P, d_out, d_in)


def encode_set(cfg: Config, decs, w: np.ndarray, idx, nthreads: int = 0, tables=None) -> Encoded:
    """Encode with a given protected set on cfg.protect_axis (orc_encode_set)."""
    w = _f32(w)
    d_out, d_in = w.shape
    if d_in % cfg.d:
        raise OracleError("d_in must be a multiple of d")
    axis = cfg.protect_axis
    P = pitch(d_in, cfg.d)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    k = len(idx)
    tables = tables or decoder_table(cfg, decs)
    es, enc_arr = _encoders(cfg, decs)
    ctype = np.uint8 if cfg.b <= 8 else np.uint16
    codes = [np.zeros((d_out, P), dtype=ctype) for _ in range(cfg.stages)]
    gains = [np.zeros((d_out, P), dtype=np.uint16) for _ in range(cfg.stages)]
    qshape = (max(k, 1), d_in) if axis == 1 else (d_out, max(k, 1))
    q = np.zeros(qshape, dtype=np.int8)
    s = np.zeros(max(k, 1), dtype=np.float32)
    idx_arg = idx if k else np.zeros(1, np.int32)
    rc = lib().orc_encode_set(cfg.d, cfg.b, cfg.stages, _ptr_array(tables), enc_arr, _p(w), d_out, d_in, axis,
                              _p(idx_arg), k, P, cfg.protect_format, _ptr_array(codes), _ptr_array(gains), _p(q), _p(s),
                              nthreads)
    _check(rc, "encode_set")
    q = q[:k] if axis == 1 else q[:, :k]
    return Encoded(codes, gains, idx.copy(), np.ascontiguousarray(q), s[:k].copy(), P, d_out, d_in, axis)


def decode(cfg: Config, decs, enc: Encoded, nthreads: int = 0, tables=None) -> np.ndarray:
    """W_hat (eq. parallel_stage_decode, eq. protected_8bit_scatter). Row
    protection: the stage sum of the coded rows, then each protected row is
    q8[p, :] * scale_p (fp32 products)."""
    tables = tables or decoder_table(cfg, decs)
    w_hat = np.zeros((enc.d_out, enc.d_in), dtype=np.float32)
    if enc.axis == 1:
        rc = lib().orc_decode(cfg.d, cfg.b, cfg.stages, _ptr_array(tables), enc.d_out, enc.d_in, enc.pitch,
                              _ptr_array(enc.codes), _ptr_array(enc.gains), None, None, None, 0,
                              cfg.protect_format, _p(w_hat), nthreads)
        _check(rc, "decode")
        for p, i in enumerate(enc.idx):
            w_hat[i, :] = payload_values(enc.q8[p], cfg.protect_format) * np.float32(enc.scale[p])
        return w_hat
    k = len(enc.idx)
    idx = enc.idx if k else np.zeros(1, np.int32)
    q = enc.q8 if k else np.zeros((enc.d_out, 1), np.int8)
    s = enc.scale if k else np.zeros(1, np.float32)
    rc = lib().orc_decode(cfg.d, cfg.b, cfg.stages, _ptr_array(tables), enc.d_out, enc.d_in, enc.pitch,
                          _ptr_array(enc.codes), _ptr_array(enc.gains), _p(idx),
                          _p(np.ascontiguousarray(q)), _p(s), k, cfg.protect_format, _p(w_hat), nthreads)
    _check(rc, "decode")
    return w_hat


def gemv_fused(cfg: Config, decs, enc: Encoded, x, lora=None, nthreads: int = 0,
               tables=None) -> np.ndarray:
    """Fused route in fp64 (never forms W_hat). Row protection: the coded
    rows by the C route with no protected column, then each protected row as
    scale_p * <q8[p, :], x> + B (A x)."""
    tables = tables or decoder_table(cfg, decs)
    x64 = np.ascontiguousarray(x, dtype=np.float64)
    if enc.axis == 1:
        plain = Encoded(enc.codes, enc.gains, np.zeros(0, np.int32), np.zeros((enc.d_out, 0), np.int8),
                        np.zeros(0, np.float32), enc.pitch, enc.d_out, enc.d_in, 0)
        y = gemv_fused(cfg, decs, plain, x64, lora, nthreads, tables)
        for p, i in enumerate(enc.idx):
            acc = float(enc.scale[p]) * float(np.dot(payload_values(enc.q8[p], cfg.protect_format)
                                                     .astype(np.float64), x64))
            if lora is not None:
                A64 = np.asarray(lora[0], dtype=np.float64)
                B64 = np.asarray(lora[1], dtype=np.float64)
                acc += float(B64[i] @ (A64 @ x64))
            y[i] = acc
        return y
    y = np.zeros(enc.d_out, dtype=np.float64)
    k = len(enc.idx)
    idx = enc.idx if k else np.zeros(1, np.int32)
    q = enc.q8 if k else np.zeros((enc.d_out, 1), np.int8)
    s = enc.scale if k else np.zeros(1, np.float32)
    rank, A64, B64 = 0, None, None
    if lora is not None:
        A64 = np.ascontiguousarray(lora[0], dtype=np.float64)
        B64 = np.ascontiguousarray(lora[1], dtype=np.float64)
        rank = A64.shape[0]
    rc = lib().orc_gemv_fused(cfg.d, cfg.b, cfg.stages, _ptr_array(tables), enc.d_out, enc.d_in,
                              enc.pitch, _ptr_array(enc.codes), _ptr_array(enc.gains), _p(idx),
                              _p(np.ascontiguousarray(q)), _p(s), k, cfg.protect_format, _p(x64), rank, _p(A64),
                              _p(B64), _p(y), nthreads)
    _check(rc, "gemv_fused")
    return y


def dense_product(w_hat: np.ndarray, X, lora=None) -> np.ndarray:
    """Y = X W_hat^T + (X A^T) B^T in fp64 (a matmul is the library step)."""
    X64 = np.asarray(X, dtype=np.float64)
    Y = X64 @ w_hat.astype(np.float64).T
    if lora is not None:
        A64 = np.asarray(lora[0], dtype=np.float64)
        B64 = np.asarray(lora[1], dtype=np.float64)
        Y = Y + (X64 @ A64.T) @ B64.T
    return Y


def gemv(cfg: Config, decs, enc: Encoded, x, lora=None, nthreads: int = 0) -> np.ndarray:
    """Dense route: y = W_hat x + B (A x), fp64, from the oracle's decode."""
    return dense_product(decode(cfg, decs, enc, nthreads), x, lora)


def gemm(cfg: Config, decs, enc: Encoded, X, lora=None, nthreads: int = 0) -> np.ndarray:
    return dense_product(decode(cfg, decs, enc, nthreads), X, lora)


# --------------------------------------------------------------------------
# Storage accounting, eq. real_size: S_tot = S_code + S_dec + S_8bit + S_LoRA + S_meta
# --------------------------------------------------------------------------
def decoder_param_count(cfg: Config) -> int:
    """Parameters of one stage decoder (fp32 each); a learned linear encoder
    adds b * d per stage (counted by sizes())."""
    if cfg.kind == KIND_MLP:
        return cfg.hidden * cfg.b + cfg.hidden + cfg.d * cfg.hidden + cfg.d
    if cfg.kind == KIND_MLP_RES1:
        return cfg.hidden * cfg.b + cfg.hidden + cfg.hidden * cfg.hidden + cfg.hidden + cfg.d * cfg.hidden + cfg.d
    if cfg.kind == KIND_LINEAR:
        return cfg.d * cfg.b + cfg.d
    return 0


def sizes(cfg: Config, d_out: int, d_in: int, lora_rank: int = 0) -> dict:
    """Byte counts for one matrix (decoder parameters counted per stage, fp32;
    a model counts them once per category, since every layer of a category
    shares its decoders)."""
    C = d_in // cfg.d
    k = cfg.k_for(d_out, d_in)
    # row protection: the protected rows carry no BSQ codes or gains (their
    # all-zero rows in the planes are layout, not payload), and each holds
    # d_in int8 values
    coded_rows = d_out - k if cfg.protect_axis == 1 else d_out
    s_code = cfg.stages * coded_rows * C * cfg.b / 8
    s_dec = cfg.stages * (decoder_param_count(cfg) + (cfg.b * cfg.d if cfg.encoder == ENC_LINEAR else 0)) * 4
    s_8bit = k * d_in if cfg.protect_axis == 1 else d_out * k
    s_lora = 2 * lora_rank * (d_in + d_out)
    s_meta = cfg.stages * coded_rows * C * 2 + 4 * k + 4 * k
    tot = s_code + s_dec + s_8bit + s_lora + s_meta
    return dict(S_code=s_code, S_dec=s_dec, S_8bit=s_8bit, S_LoRA=s_lora, S_meta=s_meta,
                S_tot=tot, chunks=d_out * C, k=k,
                bpw_nominal=cfg.stages * cfg.b / cfg.d,
                bpw_real=(8 * tot / (d_out * d_in)) if d_out * d_in else 0.0)


# --------------------------------------------------------------------------
# Conversions used by callers that hand bf16 tensors to the oracle.
# --------------------------------------------------------------------------
def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 -> fp32 is exact: the bf16 bits are the top half of the fp32 bits."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def f16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float32)


def to_f32(t) -> np.ndarray:
    """A torch tensor (any device, fp32/bf16/fp16) or array -> fp32 numpy, exactly."""
    try:
        import torch
        if isinstance(t, torch.Tensor):
            t = t.detach().cpu()
            if t.dtype == torch.bfloat16:
                return bf16_bits_to_f32(t.view(torch.int16).numpy().view(np.uint16))
            return t.to(torch.float32).numpy()
    except ImportError:
        pass
    return np.asarray(t, dtype=np.float32)


def code_scale(b: int) -> float:
    """fp32(1 / sqrt(b)), the magnitude of a spherical code entry."""
    return float(lib().orc_code_scale(b))


def train_decisions(b: int, h: int, E, W1, b1, x):
    """fp32 decisions of a training forward pass over chunks x [n, d]: the
    codes of z = E x and the ReLU masks [n, h] of the decoder's hidden layer
    (orc_train_decisions)."""
    x = _f32(x)
    n, d = x.shape
    E, W1, b1 = _f32(E), _f32(W1), _f32(b1)
    codes = np.zeros(max(n, 1), dtype=np.uint32)
    masks = np.zeros((max(n, 1), h), dtype=np.uint8)
    lib().orc_train_decisions(d, b, h, _p(E), _p(W1), _p(b1), _p(x), n, _p(codes), _p(masks))
    return codes[:n].copy(), masks[:n].copy()


def max_threads() -> int:
    return lib().orc_max_threads()
