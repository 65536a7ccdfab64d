#!/usr/bin/env python3
"""Benchmark of the BSQ codec hot path on one MI355X.

Workload: the Qwen3-8B-shaped transformer block (q/o 4096x4096, k/v 1024x4096,
gate/up 12288x4096, down 4096x12288), bf16 weights N(0, 0.02) with 1% outlier
input columns x10, d = 8 (and d = 16 as a second line of figures), two BSQ
stages with the MLP decoder, 1% int8-protected input columns, batch-1 bf16
activations. The block is encoded R times from independent weights (8 copies,
1.2 GB of compressed planes at d = 8), so consecutive steps stream different
copies and the 256 MB last-level cache cannot hold the working set.

A step is one decode token through the block: four grouped fused GEMVs
(q/k/v, o, gate/up, down), each an activation prep and a streaming kernel.
Steps are replayed from a HIP graph holding one pass over the copies. `value`
is the compressed bytes the step must move (code planes, gain planes, int8
payload, scales, indices, x, y) divided by the step time. Encode throughput
(Mchunks/s), decode GB/s and the fused GEMM's TFLOP/s at M = 16/64/256 are
measured in the same run on the same weights, as is `comparator`: on the gate
projection, the unfused path (bsq_decode to bf16, then the library product)
and the library product on a stored W_hat, beside the fused kernels.

`roofline` covers the dominant kernel (the streaming GEMV of the gate/up
group): algorithmic bytes per launch / its mean launch time from HIP events
on the launch stream. `cpu_baseline` times the oracle's fused product route on
the host cores over one projection of the same workload.
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
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemv_gateup_d8_traffic.txt")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=400)
    p.add_argument("--warmup", type=int, default=40)
    p.add_argument("--copies", type=int, default=8)
    p.add_argument("--d", type=int, default=8, help="chunk length of the headline line")
    p.add_argument("--no-d16", action="store_true", help="skip the d = 16 figures")
    p.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    p.add_argument("--no-gemm", action="store_true")
    p.add_argument("--profile-gemm-only", action="store_true",
                   help="d = 8 GEMV step and the fused GEMM at M = 16/64/256 only (for counter runs)")
    p.add_argument("--profile-gemv-only", action="store_true",
                   help="only run the GEMV steps (for rocprofv3 counter passes)")
    p.add_argument("--no-stacks", action="store_true",
                   help="skip the 36-layer Qwen3-8B (+LoRA) and 64-layer Qwen3-32B stack figures")
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


class Block:
    """One encoded copy set of the block: 7 projections x R copies."""

    def __init__(self, bsq, synth, torch, d, copies, dev):
        self.d, self.R = d, copies
        self.cfg = bsq.Config(d=d, stages=2, kind=bsq.DEC_MLP, hidden=d, protect_num=1, protect_den=100)
        self.projs = synth.qwen3_8b_block()
        self.codecs, self.layers = {}, {}
        self.encode_s = 0.0
        self.chunks = 0
        for ci, p in enumerate(self.projs):
            decs = synth.decoder_params(synth.DEC_MLP, d, d, d, 2, seed=synth.BASE_SEED, category=ci)
            codec = bsq.bsq_codec_prepare(self.cfg, decs, device=dev)
            k = self.cfg.k(p.d_in)
            W, _ = synth.weight(p.d_out, p.d_in, seed=1000 * ci + d, k_outliers=k, device=dev, n_mats=copies)
            if copies == 1:
                W = W.unsqueeze(0)
            layer = bsq.bsq_encode(self.cfg, codec, W)                # encode once (setup)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            layer2 = bsq.bsq_encode(self.cfg, codec, W, check=False)  # timed re-encode
            e1.record()
            torch.cuda.synchronize()
            self.encode_s += e0.elapsed_time(e1) / 1e3
            self.chunks += copies * p.d_out * p.d_in // d
            if not torch.equal(layer.codes[1], layer2.codes[1]):
                raise RuntimeError("encode is not deterministic")
            del W, layer2
            self.codecs[p.name] = codec
            self.layers[p.name] = layer
        torch.cuda.synchronize()

    def groups(self):
        out = {}
        for p in self.projs:
            out.setdefault(p.group, []).append(p)
        return out


def algorithmic_bytes(layers, d_in, d_out_total):
    """Compressed stream + activation + output bytes of one grouped GEMV."""
    b = 0
    for L in layers:
        b += L.nbytes_streamed()
    return b + 2 * d_in + 2 * d_out_total


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); this build has no multi-GPU "
              f"path: every box here has one GPU and the row-sharded design is described in DESIGN.md.",
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2607_08643_amd as bsq
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    bsq.lib()
    results = {}
    only = args.profile_gemv_only or args.profile_gemm_only
    d_list = [args.d] + ([] if (args.no_d16 or only) else [16 if args.d == 8 else 8])
    head = None
    for d in d_list:
        log(f"[bench] encoding {args.copies} copies of the Qwen3-8B block at d={d}")
        blk = Block(bsq, synth, torch, d, args.copies, dev)
        log(f"[bench] encode {blk.chunks / blk.encode_s / 1e6:.1f} Mchunks/s")
        xs = {g: synth.activation(ps[0].d_in, seed=77 + i, device=dev)
              for i, (g, ps) in enumerate(blk.groups().items())}
        # one plan per (copy, group); a graph per copy holds that copy's four grouped GEMVs
        plans, step_bytes = [], 0
        for r in range(args.copies):
            pr = []
            for g, ps in blk.groups().items():
                layers = [blk.layers[p.name].mat(r) for p in ps]
                codecs = [blk.codecs[p.name] for p in ps]
                pr.append(bsq.GemvPlan(blk.cfg, codecs, layers, xs[g], y_dtype=torch.bfloat16))
                if r == 0:
                    step_bytes += algorithmic_bytes(layers, ps[0].d_in, sum(p.d_out for p in ps))
            plans.append(pr)
        # one graph per copy (one step each) and one graph of a whole pass
        # over the copies (R consecutive steps, so that a replay's launch cost
        # is paid once per R steps, as a decode loop captured once would)
        s = torch.cuda.Stream()
        graphs = []
        with torch.cuda.stream(s):
            for r in range(args.copies):
                for pl in plans[r]:
                    pl()
            torch.cuda.synchronize()
            for r in range(args.copies):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=s):
                    for pl in plans[r]:
                        pl()
                graphs.append(g)
            g_pass = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_pass, stream=s):
                for r in range(args.copies):
                    for pl in plans[r]:
                        pl()
        torch.cuda.synchronize()
        log(f"[bench] d={d}: {step_bytes / 1e6:.1f} MB per step; warmup {args.warmup}, timed {args.steps}")

        def run_steps(k):
            # exactly k steps: whole passes, then single steps
            for _ in range(k // args.copies):
                g_pass.replay()
            for i in range(k % args.copies):
                graphs[i].replay()

        run_steps(args.warmup)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        run_steps(args.steps)
        t1.record()
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / args.steps
        gbs = step_bytes / (ms / 1e3) / 1e9
        log(f"[bench] d={d}: {ms * 1e3:.1f} us/step, {gbs:.0f} GB/s ({gbs / HBM_PEAK_GBS:.1%} of 8 TB/s)")

        # dominant kernel: the streaming GEMV of the gate/up group (bsq_gemv_run
        # only), launches back to back from a graph on stream s, copies rotated;
        # HIP events on s bracket the replays
        gi = list(blk.groups()).index("gateup")
        n_k = 8 * args.copies
        with torch.cuda.stream(s):
            for r in range(args.copies):
                plans[r][gi].prepare()
            torch.cuda.synchronize()
            kg = torch.cuda.CUDAGraph()
            with torch.cuda.graph(kg, stream=s):
                for i in range(n_k):
                    plans[i % args.copies][gi].run()
        torch.cuda.synchronize()
        k_times = []
        with torch.cuda.stream(s):
            kg.replay()
            torch.cuda.synchronize()
            for _ in range(20):
                a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a0.record(s)
                kg.replay()
                a1.record(s)
                torch.cuda.synchronize()
                k_times.append(a0.elapsed_time(a1) / n_k)
        k_ms = float(np.median(k_times))
        k_p10, k_p90 = float(np.percentile(k_times, 10)), float(np.percentile(k_times, 90))
        gu = [blk.layers[p.name].mat(0) for p in blk.groups()["gateup"]]
        k_bytes = algorithmic_bytes(gu, 4096, 2 * 12288)
        k_gbs = k_bytes / (k_ms / 1e3) / 1e9
        log(f"[bench] d={d}: gate/up streaming GEMV {k_ms * 1e3:.1f} us/launch, {k_gbs:.0f} GB/s")
        res = dict(ms_per_step=ms, gbs=gbs, step_bytes=step_bytes, encode_mchunks=blk.chunks / blk.encode_s / 1e6,
                   kernel_us=k_ms * 1e3, kernel_bytes=k_bytes, kernel_gbs=k_gbs,
                   kernel_us_p10=k_p10 * 1e3, kernel_us_p90=k_p90 * 1e3)

        if not args.profile_gemv_only and not args.profile_gemm_only:
            # decode GB/s (reads the planes, writes bf16 W_hat) on the largest projection
            L = blk.layers["gate"].mat(0)
            out = torch.empty((L.d_out, L.d_in), dtype=torch.bfloat16, device=dev)
            bsq.bsq_decode(blk.cfg, blk.codecs["gate"], L, out=out)
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for i in range(10):
                bsq.bsq_decode(blk.cfg, blk.codecs["gate"], blk.layers["gate"].mat(i % args.copies), out=out)
            b.record()
            torch.cuda.synchronize()
            dms = a.elapsed_time(b) / 10
            res["decode_gbs"] = (L.nbytes_streamed() + out.numel() * 2) / (dms / 1e3) / 1e9
            del out
        if not args.profile_gemv_only:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            if not args.no_gemm:
                gem = {}
                for M in (16, 64, 256):
                    X = synth.activation(4096, seed=M, device=dev, batch=M)
                    tot_flops, tot_ms = 0.0, 0.0
                    for pname in ("q", "gate", "up"):
                        Lp = blk.layers[pname].mat(0)
                        Y = torch.empty((M, Lp.d_out), dtype=torch.bfloat16, device=dev)
                        ws = torch.zeros(bsq.bsq_workspace_bytes(blk.cfg, bsq.OP_GEMM, 1, Lp.d_out, 4096, M) + 256,
                                         dtype=torch.uint8, device=dev)
                        ws = ws[(-ws.data_ptr()) % 256:]
                        # 8 calls over the copies captured in one graph and
                        # replayed, so that the figure is the GPU's time and
                        # not the Python call rate
                        gs = torch.cuda.Stream()
                        with torch.cuda.stream(gs):
                            for r in range(2):
                                bsq.bsq_gemm(blk.cfg, blk.codecs[pname], blk.layers[pname].mat(r), X, out=Y, ws=ws)
                            torch.cuda.synchronize()
                            gg = torch.cuda.CUDAGraph()
                            with torch.cuda.graph(gg, stream=gs):
                                for r in range(8):
                                    bsq.bsq_gemm(blk.cfg, blk.codecs[pname], blk.layers[pname].mat(r % args.copies), X,
                                                 out=Y, ws=ws)
                            gg.replay()
                            torch.cuda.synchronize()
                            a.record(gs)
                            for _ in range(4):
                                gg.replay()
                            b.record(gs)
                        torch.cuda.synchronize()
                        del gg
                        tot_ms += a.elapsed_time(b) / 32
                        tot_flops += 2.0 * M * Lp.d_out * Lp.d_in
                    tf = tot_flops / (tot_ms / 1e3) / 1e12
                    gem[str(M)] = dict(tflops=round(tf, 1), pct_bf16_mfma_peak=round(100 * tf / BF16_MFMA_PEAK_TFLOPS, 2))
                    log(f"[bench] d={d}: gemm M={M}: {tf:.1f} TFLOP/s")
                res["gemm"] = gem
                if not args.profile_gemm_only:
                    res["comparator"] = comparator(blk, bsq, synth, torch, dev, args.copies)
        results[d] = res
        if head is None:
            head = (blk, plans)
        else:
            del blk, plans, graphs, g_pass
        torch.cuda.synchronize()

    # same-box copy reference (and the calibration kernel for the byte
    # counters): a plain 256 MiB device-to-device copy
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
    copy_gbs = 2 * src.numel() * 4 / (c0.elapsed_time(c1) / 4 / 1e3) / 1e9
    log(f"[bench] device copy of 256 MiB: {copy_gbs:.0f} GB/s (read + write)")
    del src, dst
    hd = results[args.d]
    cpu = None
    if not args.no_cpu and not only:
        cpu = cpu_baseline(head[0], torch)
    stacks = {}
    if not args.no_stacks and not only:
        del head
        torch.cuda.empty_cache()
        stacks["qwen3_8b_36_layers_lora16"] = stack_bench(bsq, synth, torch, np, synth.qwen3_8b_block(), 36, args.d,
                                                          16, dev, "Qwen3-8B 36-layer stack + LoRA")
        stacks["qwen3_32b_64_layers"] = stack_bench(bsq, synth, torch, np, synth.qwen3_32b_block(), 64, args.d, 0,
                                                    dev, "Qwen3-32B 64-layer stack")
    traffic = read_traffic()
    line = {
        "metric": METRIC,
        "value": round(hd["gbs"], 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(hd["ms_per_step"], 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"Qwen3-8B-shaped block (q/o 4096x4096, k/v 1024x4096, gate/up 12288x4096, down "
                        f"4096x12288), d={args.d}, 2 BSQ stages, MLP decoder h={args.d}, 1% int8-protected input "
                        f"columns, batch-1 bf16 GEMV, {args.copies} independently encoded copies rotated",
            "global_batch": 1,
            "copies": args.copies,
            "bytes_per_step": hd["step_bytes"],
        },
        "pct_hbm_peak": round(100 * hd["gbs"] / HBM_PEAK_GBS, 2),
        "copy_reference_gbs": round(copy_gbs, 1),
        "encode_mchunks_per_s": round(hd["encode_mchunks"], 1),
        "decode_gbs": round(hd.get("decode_gbs", 0.0), 1),
        "gemm": hd.get("gemm"),
        "comparator": hd.get("comparator"),
        "roofline": {
            "kernel": f"gemv_lane_kernel<{args.d}, 2, TPW> (gate/up launch of bsq_gemv_run, d={args.d})",
            "bound": "hbm",
            "achieved": round(hd["kernel_gbs"], 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(hd["kernel_gbs"] / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": hd["kernel_bytes"],
            "mean_launch_us": round(hd["kernel_us"], 2),
            "launch_us_p10_p90": [round(hd["kernel_us_p10"], 2), round(hd["kernel_us_p90"], 2)],
        },
        "cpu_baseline": cpu,
        "stacks": stacks or None,
    }
    other = [d for d in results if d != args.d]
    if other:
        o = results[other[0]]
        line["other_d"] = {"d": other[0], "value_gbs": round(o["gbs"], 1),
                           "pct_hbm_peak": round(100 * o["gbs"] / HBM_PEAK_GBS, 2),
                           "encode_mchunks_per_s": round(o["encode_mchunks"], 1),
                           "kernel_gbs": round(o["kernel_gbs"], 1), "gemm": o.get("gemm"),
                           "decode_gbs": round(o.get("decode_gbs", 0.0), 1)}
    print(json.dumps(line), flush=True)


def stack_bench(bsq, synth, torch, np, projs, n_layers, d, lora_rank, dev, tag):
    """A whole stack of layers: every projection of every layer encoded in one
    launch per category (timed), then one decode token through all layers,
    captured in one HIP graph: per layer the four grouped GEMVs (with their
    LoRA prep when adapters are present). Returns encode G chunks/s and the
    token's compressed-byte rate."""
    cfg = bsq.Config(d=d, stages=2, kind=bsq.DEC_MLP, hidden=d, protect_num=1, protect_den=100)
    codecs, layers, loras = {}, {}, {}
    enc_s, chunks = 0.0, 0
    for ci, p in enumerate(projs):
        decs = synth.decoder_params(synth.DEC_MLP, d, d, d, 2, seed=synth.BASE_SEED, category=ci)
        codecs[p.name] = bsq.bsq_codec_prepare(cfg, decs, device=dev)
        W, _ = synth.weight(p.d_out, p.d_in, seed=7000 + 100 * ci + d, k_outliers=cfg.k(p.d_in), device=dev,
                            n_mats=n_layers)
        if n_layers == 1:
            W = W.unsqueeze(0)
        out = bsq.layer_empty(cfg, p.d_out, p.d_in, n_layers, dev)
        ws = torch.empty(bsq.bsq_workspace_bytes(cfg, bsq.OP_ENCODE, n_layers, p.d_out, p.d_in) + 256,
                         dtype=torch.uint8, device=dev)
        ws = ws[(-ws.data_ptr()) % 256:]
        err = torch.zeros(1, dtype=torch.int32, device=dev)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        bsq.bsq_encode(cfg, codecs[p.name], W, out=out, ws=ws, err=err, check=False)
        e1.record()
        torch.cuda.synchronize()
        if int(err.item()):
            raise RuntimeError(f"{tag}: non-finite weights")
        enc_s += e0.elapsed_time(e1) / 1e3
        chunks += n_layers * p.d_out * p.d_in // d
        layers[p.name] = out
        del W, ws
        if lora_rank:
            loras[p.name] = [synth.lora(p.d_out, p.d_in, lora_rank, seed=9000 + 100 * ci + li, device=dev)
                             for li in range(n_layers)]
    groups = {}
    for p in projs:
        groups.setdefault(p.group, []).append(p)
    xs = {g: synth.activation(ps[0].d_in, seed=300 + i, device=dev) for i, (g, ps) in enumerate(groups.items())}
    plans, nbytes = [], 0
    for li in range(n_layers):
        for g, ps in groups.items():
            Ls = [layers[p.name].mat(li) for p in ps]
            lr = [loras[p.name][li] for p in ps] if lora_rank else None
            plans.append(bsq.GemvPlan(cfg, [codecs[p.name] for p in ps], Ls, xs[g], loras=lr,
                                      y_dtype=torch.bfloat16))
            nbytes += algorithmic_bytes(Ls, ps[0].d_in, sum(p.d_out for p in ps))
            if lora_rank:
                nbytes += sum(2 * lora_rank * (p.d_in + p.d_out) * 2 for p in ps)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        for pl in plans:
            pl()
        torch.cuda.synchronize()
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr, stream=s):
            for pl in plans:
                pl()
        gr.replay()
        torch.cuda.synchronize()
        reps = max(3, int(0.3 / max(1e-6, nbytes / 2.5e12)))
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(s)
        for _ in range(reps):
            gr.replay()
        t1.record(s)
        torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / reps
    gbs = nbytes / (ms / 1e3) / 1e9
    res = {"d": d, "layers": n_layers, "lora_rank": lora_rank, "encode_gchunks_per_s": round(chunks / enc_s / 1e9, 2),
           "encode_chunks": chunks, "gemv_ms_per_token": round(ms, 4), "gemv_bytes_per_token": nbytes,
           "gemv_gbs": round(gbs, 1), "gemv_pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
           "launches_per_token": len(plans) * (2 if lora_rank else 1)}
    log(f"[bench] {tag}: encode {res['encode_gchunks_per_s']} G chunks/s; decode token {ms:.3f} ms, "
        f"{gbs:.0f} GB/s ({gbs / HBM_PEAK_GBS:.1%} of 8 TB/s)")
    del plans, gr, layers, codecs, loras
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def graph_us(torch, fns, reps=4):
    """Mean time per call of fns (a list of callables issued in order),
    captured in one HIP graph on a side stream and replayed."""
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


def comparator(blk, bsq, synth, torch, dev, copies):
    """The paper's own inference path as an unfused comparator on the gate
    projection: bsq_decode to bf16 W_hat, then the library product
    (torch.nn.functional.linear, i.e. hipBLASLt), per call; and the library
    product alone (W_hat decoded once and kept, 2 B per weight). Against the
    fused bsq_gemv (M = 1) and bsq_gemm (M = 16, 64, 256), all timed by graph
    replay over the encoded copies."""
    import torch.nn.functional as F
    name = "gate"
    Ls = [blk.layers[name].mat(r) for r in range(copies)]
    codec = blk.codecs[name]
    d_out, d_in = Ls[0].d_out, Ls[0].d_in
    W_hat = torch.empty((d_out, d_in), dtype=torch.bfloat16, device=dev)
    out = {}
    for M in (1, 16, 64, 256):
        X = synth.activation(d_in, seed=900 + M, device=dev, batch=M) if M > 1 else synth.activation(d_in, seed=901, device=dev)
        Y = torch.empty((M, d_out) if M > 1 else (d_out,), dtype=torch.bfloat16, device=dev)
        Xm = X if M > 1 else X.view(1, d_in)
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
                                                 torch.matmul(Xm, W_hat.t(), out=Y.view(Xm.shape[0], d_out))))
                                   for L in Ls])
        library = graph_us(torch, [(lambda: torch.matmul(Xm, W_hat.t(), out=Y.view(Xm.shape[0], d_out)))] * copies)
        out[str(M)] = {"fused_us": round(fused, 1), "decode_then_library_us": round(unfused, 1),
                       "library_on_stored_w_hat_us": round(library, 1)}
        log(f"[bench] comparator M={M}: fused {fused:.1f} us, decode+library {unfused:.1f} us, "
            f"library on stored W_hat {library:.1f} us")
    del W_hat
    return {"projection": f"gate {d_out}x{d_in}, d={blk.cfg.d}", "library": "torch.matmul (hipBLASLt), bf16",
            "per_M": out}


def cpu_baseline(blk, torch):
    """The oracle's fused GEMV route (plain C, fp64, OpenMP rows) on the host
    cores over copy 0 of the q projection, repeated to about 10 s of CPU time."""
    import numpy as np

    import oracle
    import synth
    L = blk.layers["q"].mat(0)
    cfg = blk.cfg
    oc = oracle.Config(d=cfg.d, b=cfg.d, stages=cfg.stages, kind=oracle.KIND_MLP, hidden=cfg.hidden,
                       protect_num=cfg.protect_num, protect_den=cfg.protect_den)
    ci = [p.name for p in blk.projs].index("q")
    decs = synth.decoder_params(synth.DEC_MLP, cfg.d, cfg.d, cfg.d, 2, seed=synth.BASE_SEED, category=ci)
    codes = [L.rowmajor(c).contiguous().cpu().numpy() for c in L.codes]
    codes = [c.view(np.uint16) if c.dtype == np.int16 else c for c in codes]
    gains = [L.rowmajor(g).contiguous().cpu().view(torch.int16).numpy().view(np.uint16) for g in L.gains]
    enc = oracle.Encoded(codes, gains, L.idx.cpu().numpy(), np.ascontiguousarray(L.q8.cpu().numpy()[:, :L.k]),
                         L.scale.cpu().numpy(),
                         L.pitch, L.d_out, L.d_in)
    x = np.random.default_rng(0).normal(size=L.d_in).astype(np.float32)
    tabs = oracle.decoder_table(oc, decs)
    nbytes = L.nbytes_streamed() + 2 * L.d_in + 2 * L.d_out
    cores = oracle.max_threads()
    oracle.gemv_fused(oc, decs, enc, x, tables=tabs)
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.gemv_fused(oc, decs, enc, x, tables=tabs)
        reps += 1
        el = time.perf_counter() - t0
        if el > 10.0:
            break
    gbs = reps * nbytes / el / 1e9
    log(f"[bench] cpu oracle: {gbs:.3f} GB/s on {cores} threads ({reps} reps)")
    # the same route on one thread (bit-identical: rows are independent)
    reps1, t1 = 0, time.perf_counter()
    while True:
        oracle.gemv_fused(oc, decs, enc, x, tables=tabs, nthreads=1)
        reps1 += 1
        el1 = time.perf_counter() - t1
        if el1 > 3.0:
            break
    gbs1 = reps1 * nbytes / el1 / 1e9
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": cores, "kind": "oracle",
            "sample": f"fused fp64 GEMV route of the oracle over copy 0 of the q projection "
                      f"(4096x4096, d={cfg.d}), {reps} repetitions, {el:.1f} s",
            "single_thread_value": round(gbs1, 4), "cpu_model": model,
            "affinity_cores": len(os.sched_getaffinity(0))}


if __name__ == "__main__":
    main()
