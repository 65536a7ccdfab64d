"""Per-output error bars of the fused products against the oracle.

The oracle's product is exact up to fp64 rounding of the decoded fp32 values
(y = W_hat x + B (A x), summed in fp64). The GPU computes the same sum with
fp32 accumulation, and on its bf16 paths rounds some operands once:

  * bf16 GEMV (d = 8 table path, d = 16 bf16-table path): every stage term
    g_s D_s(code_s)_j x_j uses the decoder entry rounded to bf16, a relative
    error of at most u = 2^-8 per term. The int8 protected term and the LoRA
    term are computed in fp32 from exact products.
    (The d = 16 symmetric-decoder path evaluates its decoder in fp16, 2^-11
    per rounding, and is held to the same bar.)
  * fused GEMM: each weight is decoded from fp16 table entries (2^-11 per
    stage term) and rounded once to bf16 (u of the weight) as an MFMA operand;
    the protected input columns enter the same MFMA as bf16(q8 * scale).
  * fp32 activations: fp32 arithmetic throughout.

Rounding to nearest leaves an error uniform on half an ulp of each rounded
value, at most u |t| for a term t. A variable uniform on [-a, a] is
sub-Gaussian with variance proxy a^2 / 3, so for independent roundings the
sum's error exceeds sqrt(2 ln(2 / lam)) * u / sqrt(3) * sqrt(sum_t t^2) with
probability at most lam (lam = 1e-9 per output: a factor 3.78 u). On top,
fp32 accumulation contributes at most n 2^-24 times the sum of |terms| for n
terms in the worst case (recursive summation); the bf16 bars add the much
smaller 2^-20 times that sum for re-association, the fp32 bar the full n 2^-24.

Each output must satisfy |y - y_ref| <= max(rel |y_ref|, floor); the
fraction of outputs decided by the floor and the worst err/tol are printed.
"""
import sys

import numpy as np

import oracle

U_BF16 = 2.0 ** -8
U_F16 = 2.0 ** -11
SUBGAUSS = float(np.sqrt(2.0 * np.log(2.0 / 1e-9)) / np.sqrt(3.0))   # 3.78
F32_EPS = 2.0 ** -24


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def stage_terms(d, enc, tabs, rows):
    """The per-stage decoded weights g_s D_s(code_s) of the given rows, fp64
    [S][len(rows)][d_in], zero where the protected path replaces them."""
    C = enc.d_in // d
    out = []
    for s, tab in enumerate(tabs):
        codes = enc.codes[s][rows, :C].astype(np.int64)
        g = oracle.f16_bits_to_f32(enc.gains[s][rows, :C]).astype(np.float64)
        T = (g[:, :, None] * tab[codes].astype(np.float64)).reshape(len(rows), enc.d_in)
        if enc.axis == 0 and len(enc.idx):
            T[:, enc.idx] = 0.0
        out.append(T)
    return out


def product_floor(kind, d, enc, tabs, w_hat, X, lora=None, block=2048):
    """Absolute error floor per output ([d_out] for a vector x, [M, d_out]
    for X) of the product y = W_hat x + B (A x) on the GPU path `kind`
    ("gemv" bf16, "gemm" bf16 MFMA, or "fp32"); see the module docstring."""
    X64 = np.atleast_2d(np.asarray(X, dtype=np.float64))
    M, d_in = X64.shape
    d_out = enc.d_out
    X2, Xa = X64 ** 2, np.abs(X64)
    var = np.zeros((M, d_out))       # sum of (u_t t)^2 over the rounded terms
    absum = np.zeros((M, d_out))     # sum of |terms|
    n_terms = len(tabs) * d_in + d_in
    prot_cols = (enc.axis == 0 and len(enc.idx) > 0)
    for r0 in range(0, d_out, block):
        rows = np.arange(r0, min(d_out, r0 + block))
        Ts = stage_terms(d, enc, tabs, rows)
        S2 = sum(T ** 2 for T in Ts)
        S1 = sum(np.abs(T) for T in Ts)
        W = w_hat[rows].astype(np.float64)
        Wp = np.zeros_like(W)
        if prot_cols:
            Wp[:, enc.idx] = W[:, enc.idx]
        elif enc.axis == 1:
            sel = np.isin(rows, enc.idx)
            Wp[sel] = W[sel]
        absum[:, rows] = Xa @ (S1 + np.abs(Wp)).T
        if kind == "gemv":
            var[:, rows] = U_BF16 ** 2 * (X2 @ S2.T)
        elif kind == "gemm":
            # bf16 weight operand: BSQ weights and (column axis) protected columns
            Wb = W if enc.axis == 0 else np.where(np.isin(rows, enc.idx)[:, None], 0.0, W)
            var[:, rows] = U_BF16 ** 2 * (X2 @ (Wb ** 2).T) + U_F16 ** 2 * (X2 @ S2.T)
    if lora is not None:
        A64 = np.asarray(lora[0], dtype=np.float64)
        B64 = np.asarray(lora[1], dtype=np.float64)
        absum += (Xa @ np.abs(A64).T) @ np.abs(B64).T
        n_terms += A64.shape[0]
    if kind == "fp32":
        floor = n_terms * F32_EPS * absum
    else:
        floor = SUBGAUSS * np.sqrt(var) + 2.0 ** -20 * absum
    return floor[0] if np.ndim(X) == 1 else floor


def check_close(y, y_ref, rel, what, floor, out_bf16=False):
    """|y - y_ref| <= max(rel |y_ref|, floor) for every output; a bf16 output
    adds its own rounding (u |y_ref|) to the floor."""
    y = np.asarray(y, dtype=np.float64)
    if not y_ref.size:
        return
    floor = np.broadcast_to(np.asarray(floor, dtype=np.float64), y_ref.shape)
    if out_bf16:
        floor = floor + U_BF16 * np.abs(y_ref)
    tol = np.maximum(rel * np.abs(y_ref), floor)
    err = np.abs(y - y_ref)
    bad = ~(err <= tol)
    on_floor = float(np.mean(floor > rel * np.abs(y_ref)))
    worst = float(np.max(err / np.maximum(tol, 1e-300)))
    say(f"  {what}: max err/tol {worst:.2e}, {on_floor:.2%} of outputs on the floor")
    assert not bad.any(), f"{what}: {int(bad.sum())} outputs outside tolerance (worst err/tol {worst:.3e})"


def term_bar(y_with, y_without, term_ref, total_abs, n_terms, what, rel=1e-4, rounded=None):
    """Presence check of one term of the product (LoRA, or the int8 protected
    columns): the GPU's difference of two calls that differ only in that term,
    against the oracle's value of the term, per output. The bar is rel |term|
    plus the fp32 rounding that can separate the two calls: the term's own
    chain of n_terms fp32 additions on top of a partial sum, and the rounding
    of both outputs, each bounded by 2^-24 times total_abs (the sum of |terms|
    of the whole product, which bounds every partial sum); plus, where the GPU
    rounds the term's operands to bf16, the sub-Gaussian bound on `rounded`
    (sqrt of the sum of the squared rounded parts)."""
    y1 = np.asarray(y_with, dtype=np.float64)
    y0 = np.asarray(y_without, dtype=np.float64)
    diff = y1 - y0
    tol = rel * np.abs(term_ref) + (n_terms + 4) * F32_EPS * np.asarray(total_abs, dtype=np.float64)
    if rounded is not None:
        tol = tol + SUBGAUSS * U_BF16 * rounded
    err = np.abs(diff - term_ref)
    worst = float(np.max(err / np.maximum(tol, 1e-300)))
    mag = float(np.median(np.abs(term_ref)) / np.maximum(np.median(tol), 1e-300))
    say(f"  {what}: max err/tol {worst:.2e}; median |term| / tol {mag:.1f}")
    assert np.all(err <= tol), f"{what}: {int((err > tol).sum())} outputs off (worst err/tol {worst:.3e})"
    return mag
