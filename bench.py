#!/usr/bin/env python3
"""Benchmark of the BSQ codec hot path on one MI355X.

Headline (`value`, `ms_per_step`): one decode token through the whole
Qwen3-32B-shaped 64-layer stack (hidden 5120, intermediate 25600; q
8192x5120, k/v 1024x5120, o 5120x8192, gate/up 25600x5120, down 5120x25600),
bf16 weights N(0, 0.02) with 1% outlier input columns x10, d = 8, two BSQ
stages with the symmetric decoder, 1% int8-protected input columns, batch-1
bf16 activations. A step is one token: per layer the four grouped fused GEMVs
(q/k/v, o, gate/up, down), 256 launches, replayed from one HIP graph. `value`
is the compressed bytes the token must move (code and gain planes, int8
payload, scales, indices, bitmap, x, y) over the token's time. The stack
(23.7 GB at d = 8) is far larger than the 256 MB last-level cache.

Same run, extra keys:
  * stacks: the 64-layer stack at d = 16; the 36-layer Qwen3-8B-shaped stack
    with rank-16 LoRA on every projection at d = 8 and 16 (encode G chunks/s
    of every stack, one launch per projection category);
  * qwen3_8b_block: one Qwen3-8B-shaped block (q/o 4096x4096, k/v 1024x4096,
    gate/up 12288x4096, down 4096x12288), 8 independently encoded copies
    rotated, d = 8 and 16: step time, GB/s, decode GB/s;
  * gemm: the fused GEMM over all seven Qwen3-8B projections with rank-16
    LoRA, M = 16, 64, 256 tokens, d = 8 and 16 (TFLOP/s, % of bf16 MFMA peak);
  * comparator: the paper's own inference path on the gate projection
    (bsq_decode to bf16, then the library product; the library product on
    stored W_hat, 8 decoded copies rotated so that the cache cannot hold them)
    beside the fused kernels, and sequential (one launch per stage) against
    stage-parallel residual decoding;
  * tiny: the 256x256 fp32 layer's GPU latencies (encode, decode, GEMV);
  * roofline: the dominant kernel of the headline (the gate/up GEMV launch),
    algorithmic bytes per launch over its mean launch time from HIP events on
    its own stream; `traffic` from the committed rocprofv3 counter summary;
  * cpu_baseline: the oracle (plain C, fp64 products, OpenMP rows) on the
    host cores: its fused GEMV on the q projection of the block, its encode
    and decode of that projection and of the tiny layer.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fused BSQ decode-GEMV compressed-weight GB/s (% HBM peak) at batch 1; encode Mchunks/s"
HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemv_c5_gateup_d8_traffic.txt")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20, help="timed decode tokens of the headline stack")
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--d", type=int, default=8, help="chunk length of the headline")
    p.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    p.add_argument("--headline-only", action="store_true", help="only the headline stack and its roofline")
    p.add_argument("--profile", choices=["c5", "gemm"], default=None,
                   help="rocprofv3 runs: only the headline stack's encode, its gate/up GEMV launches and a bf16 "
                        "decode of 8 gate matrices (c5), or the batched GEMMs (gemm), plus the 256 MiB "
                        "calibration copy")
    return p.parse_args()


def source_hash() -> str:
    h = hashlib.sha256()
    for f in ("gemv.hip", "bsq_internal.h"):
        with open(os.path.join(ROOT, "paper_2607_08643_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def read_traffic():
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3
    counter summary, if it was taken on the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            kv = dict(line.split("=", 1) for line in f.read().split("\n") if "=" in line and not line.startswith("#"))
        if kv.get("source_hash", "").strip() != source_hash():
            return None
        return float(kv["hbm_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def algorithmic_bytes(layers, d_in, d_out_total, lora_rank=0):
    """Compressed stream + activation + output bytes of one grouped GEMV; with
    adapters, their A [r][d_in] and B [d_out][r] in bf16."""
    b = sum(L.nbytes_streamed() for L in layers) + 2 * d_in + 2 * d_out_total
    if lora_rank:
        b += sum(2 * lora_rank * (L.d_in + L.d_out) for L in layers)
    return b


class Stack:
    """n_layers layers of one block shape, each projection category encoded
    as one stack (one encode launch per category, timed), one codec per
    category, optional rank-r LoRA per projection and layer, one activation
    per projection group. plans[li][g] is the grouped GEMV of group g in
    layer li."""

    def __init__(self, bsq, synth, torch, projs, n_layers, d, lora_rank, dev, seed, kind=None, fmt=0, b=None):
        """b: code bits per chunk other than d, with a (seeded, untrained)
        linear encoder per stage."""
        self.torch, self.bsq = torch, bsq
        self.d, self.n_layers, self.lora_rank = d, n_layers, lora_rank
        kind = bsq.DEC_MLP if kind is None else kind
        b = b or d
        self.cfg = bsq.Config(d=d, stages=2, kind=kind, hidden=b, protect_num=1, protect_den=100, protect_format=fmt,
                              codebook_bits=b, encoder=bsq.ENC_LINEAR if b != d else bsq.ENC_IDENTITY)
        self.projs = projs
        self.codecs, self.layers, self.loras = {}, {}, {}
        self.encode_s, self.chunks = 0.0, 0
        for ci, p in enumerate(projs):
            decs = synth.decoder_params(kind, d, b, b, 2, seed=synth.BASE_SEED, category=ci, encoder=(b != d))
            self.codecs[p.name] = bsq.bsq_codec_prepare(self.cfg, decs, device=dev)
            W, _ = synth.weight(p.d_out, p.d_in, seed=seed + 100 * ci + d, k_outliers=self.cfg.k(p.d_in),
                                device=dev, n_mats=n_layers)
            if n_layers == 1:
                W = W.unsqueeze(0)
            out = bsq.layer_empty(self.cfg, p.d_out, p.d_in, n_layers, dev)
            ws = torch.empty(bsq.bsq_workspace_bytes(self.cfg, bsq.OP_ENCODE, n_layers, p.d_out, p.d_in) + 256,
                             dtype=torch.uint8, device=dev)
            ws = ws[(-ws.data_ptr()) % 256:]
            err = torch.zeros(1, dtype=torch.int32, device=dev)
            bsq.bsq_encode(self.cfg, self.codecs[p.name], W, out=out, ws=ws, err=err, check=False)   # warm
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            bsq.bsq_encode(self.cfg, self.codecs[p.name], W, out=out, ws=ws, err=err, check=False)
            e1.record()
            torch.cuda.synchronize()
            if int(err.item()):
                raise RuntimeError("non-finite synthetic weights")
            self.encode_s += e0.elapsed_time(e1) / 1e3
            self.chunks += n_layers * p.d_out * p.d_in // d
            self.layers[p.name] = out
            del W, ws
            if lora_rank:
                self.loras[p.name] = [synth.lora(p.d_out, p.d_in, lora_rank, seed=seed + 9000 + 100 * ci + li,
                                                 device=dev) for li in range(n_layers)]
        self.groups = {}
        for p in projs:
            self.groups.setdefault(p.group, []).append(p)
        self.xs = {g: synth.activation(ps[0].d_in, seed=seed + 300 + i, device=dev)
                   for i, (g, ps) in enumerate(self.groups.items())}
        self.plans, self.group_bytes = [], {}
        for li in range(n_layers):
            row = {}
            for g, ps in self.groups.items():
                Ls = [self.layers[p.name].mat(li) for p in ps]
                lr = [self.loras[p.name][li] for p in ps] if lora_rank else None
                row[g] = bsq.GemvPlan(self.cfg, [self.codecs[p.name] for p in ps], Ls, self.xs[g], loras=lr,
                                      y_dtype=torch.bfloat16)
                if li == 0:
                    self.group_bytes[g] = algorithmic_bytes(Ls, ps[0].d_in, sum(p.d_out for p in ps), lora_rank)
            self.plans.append(row)
        self.token_bytes = n_layers * sum(self.group_bytes.values())
        torch.cuda.synchronize()

    def encode_gchunks(self):
        return self.chunks / self.encode_s / 1e9

    def graph(self, fns, stream):
        torch = self.torch
        with torch.cuda.stream(stream):
            for f in fns:
                f()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                for f in fns:
                    f()
        torch.cuda.synchronize()
        return g

    def token_graph(self, stream):
        return self.graph([pl for row in self.plans for pl in row.values()], stream)

    def time_tokens(self, stream, warmup, steps):
        """Mean ms per decode token over `steps` graph replays after `warmup`."""
        torch = self.torch
        g = self.token_graph(stream)
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            t0.record(stream)
            for _ in range(steps):
                g.replay()
            t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / steps

    def group_launch_us(self, group, stream, reps=10):
        """The streaming kernel of one group alone (bsq_gemv_run), its launches
        for every layer back to back in one graph on `stream`, HIP events on
        that stream: median, p10 and p90 over the replays of the mean time per
        launch."""
        import numpy as np
        torch = self.torch
        with torch.cuda.stream(stream):
            for row in self.plans:
                row[group].prepare(stream)
        g = self.graph([(lambda pl=row[group]: pl.run()) for row in self.plans], stream)
        ts = []
        with torch.cuda.stream(stream):
            g.replay()
            torch.cuda.synchronize()
            for _ in range(reps):
                a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a0.record(stream)
                g.replay()
                a1.record(stream)
                torch.cuda.synchronize()
                ts.append(a0.elapsed_time(a1) * 1e3 / len(self.plans))
        return float(np.median(ts)), float(np.percentile(ts, 10)), float(np.percentile(ts, 90))

    def release(self):
        self.plans = self.layers = self.codecs = self.loras = None
        self.torch.cuda.synchronize()
        self.torch.cuda.empty_cache()


def stack_figures(st, ms, tag):
    gbs = st.token_bytes / (ms / 1e3) / 1e9
    log(f"[bench] {tag}: encode {st.encode_gchunks():.2f} G chunks/s; decode token {ms:.3f} ms, {gbs:.0f} GB/s "
        f"({gbs / HBM_PEAK_GBS:.1%} of 8 TB/s)")
    return {"d": st.d, "layers": st.n_layers, "lora_rank": st.lora_rank,
            "encode_gchunks_per_s": round(st.encode_gchunks(), 2), "encode_chunks": st.chunks,
            "gemv_ms_per_token": round(ms, 4), "gemv_bytes_per_token": st.token_bytes,
            "gemv_gbs": round(gbs, 1), "gemv_pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
            "launches_per_token": st.n_layers * len(st.groups)}


def graph_us(torch, fns, reps=4):
    """Mean time per call of fns (callables issued in order), captured in one
    HIP graph on a side stream and replayed."""
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        for f in fns:
            f()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for f in fns:
                f()
        g.replay()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        for _ in range(reps):
            g.replay()
        b.record(s)
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e3 / (reps * len(fns))


def gemm_figures(blk, bsq, synth, torch, dev):
    """The fused GEMM over all seven projections of the block, each with its
    rank-16 LoRA, at M = 16, 64, 256 tokens; every (projection, copy) call in
    one graph per M. TFLOP/s counts the algorithmic 2 M d_out d_in of the
    products plus the LoRA's 2 M r (d_in + d_out)."""
    out = {}
    R = blk.n_layers
    loras = {p.name: synth.lora(p.d_out, p.d_in, 16, seed=4000 + i, device=dev) for i, p in enumerate(blk.projs)}
    for M in (16, 64, 256):
        fns, flops = [], 0.0
        wss, Ys, Xs = [], [], {}
        for p in blk.projs:
            if p.d_in not in Xs:
                Xs[p.d_in] = synth.activation(p.d_in, seed=M + p.d_in, device=dev, batch=M)
            Y = torch.empty((M, p.d_out), dtype=torch.bfloat16, device=dev)
            ws = torch.zeros(bsq.bsq_workspace_bytes(blk.cfg, bsq.OP_GEMM, 1, p.d_out, p.d_in, M) + 256,
                             dtype=torch.uint8, device=dev)
            ws = ws[(-ws.data_ptr()) % 256:]
            wss.append(ws)
            Ys.append(Y)
            for r in range(R):
                fns.append(lambda p=p, r=r, Y=Y, ws=ws: bsq.bsq_gemm(
                    blk.cfg, blk.codecs[p.name], blk.layers[p.name].mat(r), Xs[p.d_in], lora=loras[p.name],
                    out=Y, ws=ws))
                flops += 2.0 * M * p.d_out * p.d_in + 2.0 * M * 16 * (p.d_in + p.d_out)
        us = graph_us(torch, fns, reps=3) * len(fns)
        tf = flops / (us / 1e6) / 1e12
        out[str(M)] = {"tflops": round(tf, 1), "pct_bf16_mfma_peak": round(100 * tf / BF16_MFMA_PEAK_TFLOPS, 2),
                       "us_per_block": round(us / R, 1)}
        log(f"[bench] d={blk.d}: gemm over 7 projections + LoRA, M={M}: {tf:.1f} TFLOP/s, "
            f"{us / R:.1f} us per block")
        del wss, Ys, Xs
    return out


def comparator(blk, bsq, synth, torch, dev):
    """The paper's own inference path as an unfused comparator on the gate
    projection: bsq_decode to bf16 W_hat then the library product
    (torch.matmul, i.e. hipBLASLt), per call; the library product alone on a
    stored W_hat (decoded once per copy, 2 B per weight; the 8 copies rotate,
    0.8 GB, beyond the last-level cache); the fused bsq_gemv (M = 1) and
    bsq_gemm (M >= 16). And residual decoding one stage per launch
    (bsq_decode_stage, fp32 W_hat accumulated) against the stage-parallel
    bsq_decode, same fp32 output."""
    name = "gate"
    R = blk.n_layers
    Ls = [blk.layers[name].mat(r) for r in range(R)]
    codec = blk.codecs[name]
    d_out, d_in = Ls[0].d_out, Ls[0].d_in
    W_hat = torch.empty((d_out, d_in), dtype=torch.bfloat16, device=dev)
    stored = []
    for L in Ls:
        w = torch.empty((d_out, d_in), dtype=torch.bfloat16, device=dev)
        bsq.bsq_decode(blk.cfg, codec, L, out=w)
        stored.append(w)
    out = {}
    for M in (1, 16, 64, 256):
        X = synth.activation(d_in, seed=900 + M, device=dev, batch=M) if M > 1 else \
            synth.activation(d_in, seed=901, device=dev)
        Y = torch.empty((M, d_out) if M > 1 else (d_out,), dtype=torch.bfloat16, device=dev)
        Xm = X if M > 1 else X.view(1, d_in)
        Yv = Y.view(Xm.shape[0], d_out)
        if M == 1:
            plans = [bsq.GemvPlan(blk.cfg, [codec], [L], X) for L in Ls]
            fused = graph_us(torch, [(lambda pl=pl: pl()) for pl in plans])
        else:
            ws = torch.zeros(bsq.bsq_workspace_bytes(blk.cfg, bsq.OP_GEMM, 1, d_out, d_in, M) + 256,
                             dtype=torch.uint8, device=dev)
            ws = ws[(-ws.data_ptr()) % 256:]
            fused = graph_us(torch, [(lambda L=L: bsq.bsq_gemm(blk.cfg, codec, L, X, out=Y, ws=ws)) for L in Ls])
            del ws
        unfused = graph_us(torch, [(lambda L=L: (bsq.bsq_decode(blk.cfg, codec, L, out=W_hat),
                                                 torch.matmul(Xm, W_hat.t(), out=Yv))) for L in Ls])
        library = graph_us(torch, [(lambda w=w: torch.matmul(Xm, w.t(), out=Yv)) for w in stored])
        out[str(M)] = {"fused_us": round(fused, 1), "decode_then_library_us": round(unfused, 1),
                       "library_on_stored_w_hat_us": round(library, 1)}
        log(f"[bench] d={blk.d} comparator M={M}: fused {fused:.1f} us, decode+library {unfused:.1f} us, "
            f"library on stored W_hat (8 copies rotated) {library:.1f} us")
    del stored
    # sequential against stage-parallel residual decoding, fp32 W_hat
    W32 = torch.empty((d_out, d_in), dtype=torch.float32, device=dev)
    S = blk.cfg.stages
    par = graph_us(torch, [(lambda L=L: bsq.bsq_decode(blk.cfg, codec, L, out=W32)) for L in Ls])
    seq = graph_us(torch, [(lambda L=L: [bsq.bsq_decode_stage(blk.cfg, codec, L, s, s > 0, W32) for s in range(S)])
                           for L in Ls])
    bytes_par = Ls[0].nbytes_streamed() + 4 * d_out * d_in
    log(f"[bench] d={blk.d} residual decode, fp32 W_hat: stage-parallel {par:.1f} us, sequential {seq:.1f} us "
        f"({S} launches)")
    del W32, W_hat
    return {"projection": f"gate {d_out}x{d_in}, d={blk.d}", "library": "torch.matmul (hipBLASLt), bf16",
            "per_M": out,
            "residual_decode_fp32": {"stage_parallel_us": round(par, 1), "sequential_us": round(seq, 1),
                                     "stages": S, "stage_parallel_gbs": round(bytes_par / par / 1e3, 1)}}


def variants(bsq, synth, torch, dev, s):
    """The codec-component ablation's variants (Section IV-D) on the
    Qwen3-8B-shaped block, 8 encoded copies rotated: the symmetric decoder
    with one residual block, the FP8-E4M3 / FP8-E5M2 protected payloads, and
    code lengths b other than d with a linear encoder (b/d = 2 and 1/2 bits
    per weight and stage, Section III-D); encode rate and batch-1 GEMV step
    per block."""
    out = {}
    for d, kind, fmt, b, tag in ((8, bsq.DEC_MLP_RES1, bsq.PROT_INT8, 8, "res1"),
                                 (8, bsq.DEC_MLP, bsq.PROT_E4M3, 8, "e4m3"),
                                 (8, bsq.DEC_MLP, bsq.PROT_E5M2, 8, "e5m2"),
                                 (16, bsq.DEC_MLP_RES1, bsq.PROT_INT8, 16, "res1"),
                                 (16, bsq.DEC_MLP, bsq.PROT_E4M3, 16, "e4m3"),
                                 (8, bsq.DEC_MLP, bsq.PROT_INT8, 16, "b16_linear_encoder"),
                                 (16, bsq.DEC_MLP, bsq.PROT_INT8, 8, "b8_linear_encoder")):
        blk = Stack(bsq, synth, torch, synth.qwen3_8b_block(), 8, d, 0, dev, seed=1000, kind=kind, fmt=fmt, b=b)
        step_ms = blk.time_tokens(s, 8, 64) / blk.n_layers
        step_bytes = blk.token_bytes // blk.n_layers
        gbs = step_bytes / (step_ms / 1e3) / 1e9
        out[f"d{d}_{tag}"] = {"ms_per_step": round(step_ms, 5), "gbs": round(gbs, 1),
                              "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
                              "encode_mchunks_per_s": round(1e3 * blk.encode_gchunks(), 1)}
        log(f"[bench] variant d={d} {tag}: block step {step_ms * 1e3:.1f} us, {gbs:.0f} GB/s, "
            f"encode {blk.encode_gchunks():.2f} G chunks/s")
        blk.release()
    return out


def training(bsq, synth, torch, dev, d=8, b=8, batch=1 << 16, steps=40):
    """Codec training (Section III-C; category-batched, Section III-G): one
    step = loss and straight-through gradient of a mini-batch of chunks drawn
    from the 36-layer Qwen3-8B-shaped q_proj category (bf16, 75.5 M chunks at
    d = 8) plus one Adam step; indices drawn before the timed region."""
    import numpy as np
    h = b
    cfg = bsq.Config(d=d, codebook_bits=b, hidden=h, encoder=bsq.ENC_LINEAR, stages=1)
    hp = bsq.TrainHyper(lr=2e-3)
    W, _ = synth.weight(4096, 4096, seed=77, dtype=torch.bfloat16, device=dev, n_mats=36)
    n_total = W.numel() // d
    dec = synth.decoder_params(synth.DEC_MLP, d, b, h, 1, seed=78, encoder=True)[0]
    theta = torch.from_numpy(np.concatenate([np.ravel(v) for v in (dec.E, dec.W1, dec.b1, dec.W2, dec.b2)])
                             .astype(np.float32)).to(dev)
    P = theta.numel()
    m, v = torch.zeros(P, device=dev), torch.zeros(P, device=dev)
    grad, loss = torch.empty(P, device=dev), torch.empty(4, device=dev)
    ws = torch.empty(bsq.bsq_train_workspace_bytes(cfg, batch) + 256, dtype=torch.uint8, device=dev)
    ws = ws[(-ws.data_ptr()) % 256:]
    gen = torch.Generator(device=dev).manual_seed(79)
    idx = torch.randint(0, n_total, (steps + 4, batch), generator=gen, device=dev, dtype=torch.int64)
    losses = []

    def step(k):
        bsq.bsq_train_grad(cfg, hp, W, theta, idx=idx[k], grad=grad, loss=loss, ws=ws)
        bsq.bsq_train_adam(cfg, hp, k + 1, theta, grad, m, v)

    for k in range(4):
        step(k)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    first = None
    e0.record()
    for k in range(4, steps + 4):
        step(k)
        if k == 4:
            first = loss.clone()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    out = {"d": d, "b": b, "h": h, "batch_chunks": batch, "category_chunks": n_total, "ms_per_step": round(ms, 4),
           "mchunks_per_s": round(batch / ms / 1e3, 1), "loss_first": round(float(first[0]), 5),
           "loss_last": round(float(loss[0]), 5)}
    log(f"[bench] codec training d={d} b={b}: {ms * 1e3:.1f} us per step of {batch} chunks "
        f"({out['mchunks_per_s']} M chunks/s), loss {out['loss_first']} -> {out['loss_last']}")
    del W
    torch.cuda.empty_cache()
    return out


def tiny_latency(bsq, synth, torch, dev):
    """The 256x256 fp32 layer (d = 8, no protection): GPU time of one encode,
    one fp32 decode and one fp32 GEMV, each by graph replay."""
    cfg = bsq.Config(d=8, stages=2, kind=bsq.DEC_MLP, hidden=8, protect_num=0, protect_den=100)
    decs = synth.decoder_params(synth.DEC_MLP, 8, 8, 8, 2, seed=1)
    codec = bsq.bsq_codec_prepare(cfg, decs, device=dev)
    W, _ = synth.weight(256, 256, seed=2, dtype=torch.float32, device=dev)
    x = synth.activation(256, seed=3, dtype=torch.float32, device=dev)
    out = bsq.layer_empty(cfg, 256, 256, 1, dev)
    ws = torch.empty(bsq.bsq_workspace_bytes(cfg, bsq.OP_ENCODE, 1, 256, 256) + 256, dtype=torch.uint8, device=dev)
    ws = ws[(-ws.data_ptr()) % 256:]
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    enc = graph_us(torch, [lambda: bsq.bsq_encode(cfg, codec, W, out=out, ws=ws, err=err, check=False)] * 8)
    w_hat = torch.empty((256, 256), dtype=torch.float32, device=dev)
    dec = graph_us(torch, [lambda: bsq.bsq_decode(cfg, codec, out, out=w_hat)] * 8)
    plan = bsq.GemvPlan(cfg, [codec], [out], x, y_dtype=torch.float32)
    gemv = graph_us(torch, [lambda: plan()] * 8)
    log(f"[bench] tiny 256x256 fp32: encode {enc:.1f} us, decode {dec:.1f} us, gemv {gemv:.1f} us")
    return {"workload": "256x256 fp32 layer, d=8, 2 stages, symmetric decoder h=8, no protection",
            "encode_us": round(enc, 2), "decode_us": round(dec, 2), "gemv_us": round(gemv, 2)}


def cpu_baseline(blk, bsq, torch):
    """The oracle as it stands (plain C, fp64 products, OpenMP rows) on the
    host cores: its fused GEMV route over the q projection of block copy 0
    (the metric's unit), repeated for about 10 s; then its encode and decode
    of that projection and of the tiny layer, each repeated for about 2 s."""
    import numpy as np

    import oracle
    import synth
    cfg = blk.cfg
    oc = oracle.Config(d=cfg.d, b=cfg.d, stages=cfg.stages, kind=oracle.KIND_MLP, hidden=cfg.hidden,
                       protect_num=cfg.protect_num, protect_den=cfg.protect_den)
    ci = [p.name for p in blk.projs].index("q")
    decs = synth.decoder_params(synth.DEC_MLP, cfg.d, cfg.d, cfg.d, 2, seed=synth.BASE_SEED, category=ci)
    L = blk.layers["q"].mat(0)
    codes = [L.rowmajor(c).contiguous().cpu().numpy() for c in L.codes]
    codes = [c.view(np.uint16) if c.dtype == np.int16 else c for c in codes]
    gains = [L.rowmajor(g).contiguous().cpu().view(torch.int16).numpy().view(np.uint16) for g in L.gains]
    enc = oracle.Encoded(codes, gains, L.idx.cpu().numpy(), np.ascontiguousarray(L.q8.cpu().numpy()[:, :L.k]),
                         L.scale.cpu().numpy(), L.pitch, L.d_out, L.d_in)
    x = np.random.default_rng(0).normal(size=L.d_in).astype(np.float32)
    tabs = oracle.decoder_table(oc, decs)
    nbytes = L.nbytes_streamed() + 2 * L.d_in + 2 * L.d_out
    cores = oracle.max_threads()

    def rate(fn, seconds):
        fn()
        reps, t0 = 0, time.perf_counter()
        while True:
            fn()
            reps += 1
            el = time.perf_counter() - t0
            if el > seconds:
                return reps, el
    reps, el = rate(lambda: oracle.gemv_fused(oc, decs, enc, x, tables=tabs), 10.0)
    gbs = reps * nbytes / el / 1e9
    log(f"[bench] cpu oracle gemv: {gbs:.3f} GB/s on {cores} threads ({reps} reps)")
    r1, e1 = rate(lambda: oracle.gemv_fused(oc, decs, enc, x, tables=tabs, nthreads=1), 3.0)
    W, _ = synth.weight(L.d_out, L.d_in, seed=5, k_outliers=cfg.k(L.d_in))
    Wf = oracle.to_f32(W)
    re, ee = rate(lambda: oracle.encode(oc, decs, Wf, tables=tabs), 2.0)
    rd, ed = rate(lambda: oracle.decode(oc, decs, enc, tables=tabs), 2.0)
    chunks = L.d_out * L.d_in // cfg.d
    # the tiny layer in full
    toc = oracle.Config(d=8, b=8, stages=2, kind=oracle.KIND_MLP, hidden=8, protect_num=0)
    tdecs = synth.decoder_params(synth.DEC_MLP, 8, 8, 8, 2, seed=1)
    tt = oracle.decoder_table(toc, tdecs)
    tW = oracle.to_f32(synth.weight(256, 256, seed=2, dtype=torch.float32)[0])
    tx = oracle.to_f32(synth.activation(256, seed=3, dtype=torch.float32))
    tenc = oracle.encode(toc, tdecs, tW, tables=tt)
    rte, ete = rate(lambda: oracle.encode(toc, tdecs, tW, tables=tt), 1.0)
    rtd, etd = rate(lambda: oracle.decode(toc, tdecs, tenc, tables=tt), 1.0)
    rtg, etg = rate(lambda: oracle.gemv_fused(toc, tdecs, tenc, tx, tables=tt), 1.0)
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    res = {"value": round(gbs, 4), "unit": "GB/s", "cores": cores, "kind": "oracle",
           "sample": f"the oracle's fused fp64 GEMV route over copy 0 of the Qwen3-8B q projection (4096x4096, "
                     f"d={cfg.d}), {reps} repetitions in {el:.1f} s; then its encode and decode of a 4096x4096 "
                     f"projection and of the 256x256 fp32 layer",
           "single_thread_value": round(r1 * nbytes / e1 / 1e9, 4),
           "encode_mchunks_per_s": round(re * chunks / ee / 1e6, 2),
           "decode_gbs": round(rd * (L.nbytes_streamed() + 4 * L.d_out * L.d_in) / ed / 1e9, 3),
           "tiny_encode_us": round(ete / rte * 1e6, 1), "tiny_decode_us": round(etd / rtd * 1e6, 1),
           "tiny_gemv_us": round(etg / rtg * 1e6, 1),
           "cpu_model": model, "affinity_cores": len(os.sched_getaffinity(0))}
    # one codec-training step (loss and gradient, fp64 numpy) on 65536 chunks
    import oracle.train as OT
    tdec = synth.decoder_params(synth.DEC_MLP, 8, 8, 8, 1, seed=9, encoder=True)[0]
    th = OT.pack(tdec.E, tdec.W1, tdec.b1, tdec.W2, tdec.b2)
    Xc = Wf.reshape(-1, 8)[:65536]
    rt, et = rate(lambda: OT.loss_and_grad(th, Xc, 8, 8, 8, OT.Hyper()), 2.0)
    res["train_step_mchunks_per_s"] = round(rt * 65536 / et / 1e6, 3)
    log(f"[bench] cpu oracle: encode {res['encode_mchunks_per_s']} Mchunks/s, decode {res['decode_gbs']} GB/s; "
        f"tiny encode {res['tiny_encode_us']} us, decode {res['tiny_decode_us']} us, gemv {res['tiny_gemv_us']} us")
    return res


def copy_reference(torch, dev):
    """A plain 256 MiB device-to-device copy (also the calibration kernel of
    the byte counters)."""
    src = torch.empty(64 << 20, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(4):
        dst.copy_(src)
    c1.record()
    torch.cuda.synchronize()
    gbs = 2 * src.numel() * 4 / (c0.elapsed_time(c1) / 4 / 1e3) / 1e9
    log(f"[bench] device copy of 256 MiB: {gbs:.0f} GB/s (read + write)")
    return gbs


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): there is no multi-GPU path in this "
              f"library; the row-sharded design is described in DESIGN.md.", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2607_08643_amd as bsq
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    bsq.lib()
    s = torch.cuda.Stream()
    d = args.d
    other_d = 16 if d == 8 else 8

    if args.profile == "gemm":
        blk = Stack(bsq, synth, torch, synth.qwen3_8b_block(), 8, 8, 0, dev, seed=1000)
        gemm_figures(blk, bsq, synth, torch, dev)
        copy_reference(torch, dev)
        return

    # headline: the 64-layer Qwen3-32B-shaped stack, one decode token per step
    log(f"[bench] encoding the 64-layer Qwen3-32B-shaped stack at d={d}")
    c5 = Stack(bsq, synth, torch, synth.qwen3_32b_block(), 64, d, 0, dev, seed=7000)
    if args.profile == "c5":
        c5.group_launch_us("gateup", s, reps=3)
        L0 = c5.layers["gate"].mat(0)
        W_hat = torch.empty((L0.d_out, L0.d_in), dtype=torch.bfloat16, device=dev)
        for r in range(8):
            bsq.bsq_decode(c5.cfg, c5.codecs["gate"], c5.layers["gate"].mat(r), out=W_hat)
        torch.cuda.synchronize()
        del W_hat
        copy_reference(torch, dev)
        return
    ms = c5.time_tokens(s, args.warmup, args.steps)
    head = stack_figures(c5, ms, f"Qwen3-32B 64-layer stack d={d}")
    k_us, k_p10, k_p90 = c5.group_launch_us("gateup", s)
    k_bytes = c5.group_bytes["gateup"]
    k_gbs = k_bytes / k_us / 1e3
    log(f"[bench] d={d}: gate/up GEMV launch {k_us:.2f} us, {k_gbs:.0f} GB/s")
    group_us = {g: round(c5.group_launch_us(g, s, reps=3)[0], 2) for g in c5.groups}
    c5.release()
    del c5
    traffic = read_traffic()
    line = {
        "metric": METRIC,
        "value": round(head["gemv_gbs"], 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"Qwen3-32B-shaped 64-layer stack (q 8192x5120, k/v 1024x5120, o 5120x8192, gate/up "
                        f"25600x5120, down 5120x25600 per layer), bf16 weights N(0,0.02) with 1% outlier input "
                        f"columns x10, d={d}, 2 BSQ stages, symmetric decoder h={d}, 1% int8-protected input "
                        f"columns; one step = one batch-1 decode token through all 256 grouped GEMVs",
            "global_batch": 1,
            "layers": 64,
            "bytes_per_step": head["gemv_bytes_per_token"],
        },
        "pct_hbm_peak": head["gemv_pct_hbm_peak"],
        "encode_mchunks_per_s": round(1e3 * head["encode_gchunks_per_s"], 1),
        "group_launch_us": group_us,
        "roofline": {
            "kernel": f"gemv_lane_kernel<{d}, 2, TPW> (gate/up group launch of bsq_gemv_run, 2 x 25600x5120, d={d})",
            "bound": "hbm",
            "achieved": round(k_gbs, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(k_gbs / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": k_bytes,
            "mean_launch_us": round(k_us, 2),
            "launch_us_p10_p90": [round(k_p10, 2), round(k_p90, 2)],
        },
    }
    if args.headline_only:
        print(json.dumps(line), flush=True)
        return

    stacks = {f"qwen3_32b_64_layers_d{d}": head}
    log(f"[bench] encoding the 64-layer Qwen3-32B-shaped stack at d={other_d}")
    st = Stack(bsq, synth, torch, synth.qwen3_32b_block(), 64, other_d, 0, dev, seed=7000)
    stacks[f"qwen3_32b_64_layers_d{other_d}"] = stack_figures(st, st.time_tokens(s, 2, 5),
                                                              f"Qwen3-32B 64-layer stack d={other_d}")
    st.release()
    for dd in (d, other_d):
        st = Stack(bsq, synth, torch, synth.qwen3_8b_block(), 36, dd, 16, dev, seed=8000)
        stacks[f"qwen3_8b_36_layers_lora16_d{dd}"] = stack_figures(st, st.time_tokens(s, 2, 10),
                                                                   f"Qwen3-8B 36-layer stack + LoRA d={dd}")
        st.release()
    line["stacks"] = stacks

    block, gemm, comp = {}, {}, {}
    for dd in (d, other_d):
        log(f"[bench] Qwen3-8B block at d={dd}, 8 copies rotated")
        blk = Stack(bsq, synth, torch, synth.qwen3_8b_block(), 8, dd, 0, dev, seed=1000)
        step_ms = blk.time_tokens(s, 8, 64) / blk.n_layers
        step_bytes = blk.token_bytes // blk.n_layers
        gbs = step_bytes / (step_ms / 1e3) / 1e9
        L = blk.layers["gate"].mat(0)
        W_hat = torch.empty((L.d_out, L.d_in), dtype=torch.bfloat16, device=dev)
        dec_us = graph_us(torch, [(lambda r=r: bsq.bsq_decode(blk.cfg, blk.codecs["gate"], blk.layers["gate"].mat(r),
                                                              out=W_hat)) for r in range(blk.n_layers)])
        del W_hat
        block[f"d{dd}"] = {"ms_per_step": round(step_ms, 5), "bytes_per_step": step_bytes, "gbs": round(gbs, 1),
                           "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
                           "encode_mchunks_per_s": round(1e3 * blk.encode_gchunks(), 1),
                           "decode_gate_bf16_gbs": round((L.nbytes_streamed() + 2 * L.d_out * L.d_in) / dec_us / 1e3,
                                                         1)}
        log(f"[bench] Qwen3-8B block d={dd}: {step_ms * 1e3:.1f} us/step, {gbs:.0f} GB/s; "
            f"bf16 decode of gate {block[f'd{dd}']['decode_gate_bf16_gbs']} GB/s")
        gemm[f"d{dd}"] = gemm_figures(blk, bsq, synth, torch, dev)
        comp[f"d{dd}"] = comparator(blk, bsq, synth, torch, dev)
        if dd == d and not args.no_cpu:
            line["cpu_baseline"] = cpu_baseline(blk, bsq, torch)
        blk.release()
    line["qwen3_8b_block"] = block
    line["gemm"] = gemm
    line["comparator"] = comp
    line["variants"] = variants(bsq, synth, torch, dev, s)
    line["codec_training"] = {f"d{dd}_b{bb}": training(bsq, synth, torch, dev, dd, bb) for dd, bb in ((8, 8), (8, 16))}
    line["tiny"] = tiny_latency(bsq, synth, torch, dev)
    line["copy_reference_gbs"] = round(copy_reference(torch, dev), 1)
    if "cpu_baseline" not in line:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
