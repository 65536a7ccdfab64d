"""The products' bounded waits, forced from the host.

A finishing workgroup of bsq_gemv waits for the other
workgroups' flagged partial results. The wait is bounded, and with
bsq_debug_set_wait_limit(0) every such wait gives up at once, so the
give-up path runs with every kernel still exiting normally. Expected, per
call on one workspace:
  1. normal call: error word 0, result equal to a fresh workspace's;
  2. forced give-up: BSQ_DEVERR_TIMEOUT (and possibly POISONED, from a
     finishing workgroup that comes after another one gave up), every output
     NaN (each output here is written by a finishing workgroup that waits),
     flagged slots left as they are and the workspace poisoned;
  3. next call at the normal bound: BSQ_DEVERR_POISONED, outputs NaN,
     nothing in the workspace consumed;
  4. after the caller zero-fills the workspace: error word 0 and the result
     of call 1, bit for bit.
"""
import pytest
import torch

import paper_2607_08643_amd as bsq
import synth
from parity_bounds import say

pytestmark = pytest.mark.gpu


def _layer(d, d_out, d_in, gpu, seed=3):
    cfg = bsq.Config(d=d, hidden=d)
    decs = synth.decoder_params(cfg.kind, d, d, cfg.hidden, cfg.stages, seed=seed)
    codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
    W, _ = synth.weight(d_out, d_in, seed=seed + 1, k_outliers=cfg.k(d_in), device=gpu)
    layer = bsq.bsq_encode(cfg, codec, W)
    return cfg, codec, layer


def _four_calls(call, ws, err):
    """The four calls of the module docstring; returns their outputs and
    error words."""
    outs, errs = [], []
    for step in range(4):
        err.zero_()
        if step == 3:
            torch.cuda.synchronize()
            ws.zero_()
        prev = bsq.bsq_debug_set_wait_limit(0 if step == 1 else -1)
        try:
            y = call().clone()
        finally:
            bsq.bsq_debug_set_wait_limit(-1)
        torch.cuda.synchronize()
        outs.append(y)
        errs.append(int(err.item()))
        assert prev >= 0
    return outs, errs


def _check(outs, errs, what):
    say(f"  {what}: error words {errs}")
    assert errs[0] == 0
    # (a finishing workgroup that reads the poison word after another one of
    # the same call set it reports POISONED rather than TIMEOUT)
    assert errs[1] & bsq.DEVERR_TIMEOUT and errs[1] & ~(bsq.DEVERR_TIMEOUT | bsq.DEVERR_POISONED) == 0
    assert errs[2] == bsq.DEVERR_POISONED
    assert errs[3] == 0
    assert not torch.isnan(outs[0]).any()
    assert torch.isnan(outs[1]).all() and torch.isnan(outs[2]).all()
    assert torch.equal(outs[3], outs[0])


@pytest.mark.parametrize("d", [8, 16])
def test_gemv_wait_give_up_poisons_workspace(d, gpu):
    # 4096 inputs and 256 rows: every 64-row group is split over several
    # workgroups (the finishing one waits for the others' partial sums), and
    # the rank-16 LoRA adds the wait for the LoRA vector
    say(f"gemv forced wait give-up d={d}")
    cfg, codec, layer = _layer(d, 256, 4096, gpu)
    x = synth.activation(4096, seed=5, device=gpu)
    A, B = synth.lora(256, 4096, 16, seed=6, device=gpu)
    err = torch.zeros(1, dtype=torch.int32, device=gpu)
    plan = bsq.GemvPlan(cfg, [codec], [layer], x, loras=[(A, B)], y_dtype=torch.float32, err=err)
    outs, errs = _four_calls(lambda: plan()[0], plan.ws, err)
    _check(outs, errs, f"gemv d={d}")
    fresh = bsq.bsq_gemv(cfg, codec, layer, x, loras=(A, B), y_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(fresh, outs[0])


@pytest.mark.parametrize("d,M", [(8, 1), (8, 16), (8, 64), (16, 64), (8, 256)])
def test_gemm_does_not_wait(d, M, gpu):
    """No workgroup of bsq_gemm waits for another (a second launch sums the
    split-K partials): with the wait bound at zero the result and the error
    word are those of a normal call, whatever the workspace header holds."""
    say(f"gemm ignores the wait bound d={d} M={M}")
    cfg, codec, layer = _layer(d, 256, 4096, gpu, seed=7)
    X = synth.activation(4096, seed=8, device=gpu, batch=M)
    A, B = synth.lora(256, 4096, 16, seed=9, device=gpu)
    err = torch.zeros(1, dtype=torch.int32, device=gpu)
    need = bsq.bsq_workspace_bytes(cfg, bsq.OP_GEMM, 1, 256, 4096, M)
    raw = torch.zeros(need + 256, dtype=torch.uint8, device=gpu)
    ws = raw[(-raw.data_ptr()) % 256:][:need]
    ref = bsq.bsq_gemm(cfg, codec, layer, X, lora=(A, B), y_dtype=torch.float32, ws=ws, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ws[:256].fill_(1)  # the header (a GEMV workspace's poison word sits there)
    prev = bsq.bsq_debug_set_wait_limit(0)
    try:
        Y = bsq.bsq_gemm(cfg, codec, layer, X, lora=(A, B), y_dtype=torch.float32, ws=ws, err=err)
    finally:
        bsq.bsq_debug_set_wait_limit(-1)
    torch.cuda.synchronize()
    assert prev >= 0
    assert int(err.item()) == 0
    assert torch.equal(Y, ref)
