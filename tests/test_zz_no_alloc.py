"""bsq_gemv_noalloc, the GEMV entry point that allocates nothing: its
workspace is the library's own device array (one per GPU), reached through
hipGetSymbolAddress. Through the C ABI it must give exactly what bsq_gemv
gives with a workspace of its own (same kernels, same order of additions),
call after call on the shared array, with a smaller group after a larger one
and with the d = 16 decoder path (which keeps per-chunk records in the array)
next to the d = 8 path.
"""
import pytest
import torch

import paper_2607_08643_amd as bsq
import synth
from parity_bounds import say

pytestmark = pytest.mark.gpu


def _group(d, shapes, d_in, seed, gpu, lora_rank):
    cfg = bsq.Config(d=d, hidden=d)
    codecs, layers, loras = [], [], []
    for i, d_out in enumerate(shapes):
        decs = synth.decoder_params(cfg.kind, d, d, cfg.hidden, cfg.stages, seed=seed + i)
        codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
        W, _ = synth.weight(d_out, d_in, seed=seed + 10 + i, k_outliers=cfg.k(d_in), device=gpu)
        codecs.append(codec)
        layers.append(bsq.bsq_encode(cfg, codec, W))
        loras.append(synth.lora(d_out, d_in, lora_rank, seed=seed + 20 + i, device=gpu) if lora_rank else None)
    x = synth.activation(d_in, seed=seed + 30, device=gpu)
    return cfg, codecs, layers, (loras if lora_rank else None), x


# per d: a larger group with LoRA, then a smaller one without (other d_in)
CALLS = {
    8: [((1500, 1500), 2048, 16), ((300,), 1024, 0)],
    16: [((700, 700), 2048, 16), ((200,), 1024, 0)],
}


@pytest.mark.parametrize("d", [16, 8])
def test_gemv_noalloc_equals_gemv(d, gpu):
    for call, (shapes, d_in, rank) in enumerate(CALLS[d]):
        say(f"noalloc d={d} call {call}: {len(shapes)} x {shapes[0]}x{d_in}, LoRA rank {rank}")
        cfg, codecs, layers, loras, x = _group(d, shapes, d_in, 100 * d + 40 * call, gpu, rank)
        err = torch.zeros(1, dtype=torch.int32, device=gpu)
        got = bsq.bsq_gemv_noalloc(cfg, codecs, layers, x, loras=loras, y_dtype=torch.float32, err=err)
        want = bsq.bsq_gemv(cfg, codecs, layers, x, loras=loras, y_dtype=torch.float32)
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        for g, w in zip(got, want):
            assert not torch.isnan(g).any()
            assert torch.equal(g, w), f"d={d} call {call}: noalloc output differs from bsq_gemv"
        # the same call again on the array the previous call left behind
        again = bsq.bsq_gemv_noalloc(cfg, codecs, layers, x, loras=loras, y_dtype=torch.float32, err=err)
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        for g, w in zip(again, want):
            assert torch.equal(g, w)
