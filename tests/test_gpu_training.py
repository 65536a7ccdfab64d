"""Codec training on the GPU (bsq_train_grad, bsq_train_adam) against the
oracle's fp64 step (oracle/train.py; Section III-C, eq. codec_loss and
eq. codec_loss_terms), on weight chunks gathered from a stack of layers of one
category (Section III-G).

Bar: both sides take the same decisions (code bits of E x and the decoder's
ReLU mask, fp32 fmaf chains), so what differs is fp32 against fp64
arithmetic. The loss terms agree to 1e-5 relative (the entropy term relative
to the two entropy sums it is the difference of); each parameter block's
gradient (E, W1, b1, W2, b2) to 1e-4 of its 2-norm (fp32 evaluation of
chains of a few hundred operations and sums of up to 2^16 terms in a fixed
order, about 1700 units of 2^-24, and a norm-wise bound because the
straight-through projection of the encoder gradient cancels); one Adam step to
16 units of 2^-24 of its update plus two of the parameter. A training run lowers
the loss, runs bit-identically twice, and the trained codec encodes on the
product path exactly as the oracle encodes with the same parameters.
"""
import numpy as np
import pytest
import torch

import oracle
import oracle.train as OT
import paper_2607_08643_amd as bsq
import synth
from parity_bounds import say
from test_gpu_parity import assert_layer_equal

pytestmark = pytest.mark.gpu

HP = dict(lambda_c=0.25, lambda_e=0.1, gamma=1.0, tau=1.0, lr=2e-3)


def _theta0(d, b, h, seed):
    dec = synth.decoder_params(synth.DEC_MLP, d, b, h, 1, seed=seed, encoder=True)[0]
    return OT.pack(dec.E, dec.W1, dec.b1, dec.W2, dec.b2)


def _blocks(d, b, h):
    sizes = [b * d, h * b, h, d * h, d]
    out, o = [], 0
    for n in sizes:
        out.append(slice(o, o + n))
        o += n
    return out


def _stack(n_mats, d_out, d_in, seed, dtype):
    W, _ = synth.weight(d_out, d_in, seed, k_outliers=0, dtype=dtype, n_mats=n_mats)
    return W


@pytest.mark.parametrize("d,b,h", [(8, 8, 8), (8, 16, 16), (16, 8, 8), (16, 16, 16), (8, 8, 24)])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_loss_and_gradient_match_oracle(d, b, h, dtype, gpu):
    say(f"train grad d={d} b={b} h={h} {dtype}")
    cfg = bsq.Config(d=d, codebook_bits=b, hidden=h, encoder=bsq.ENC_LINEAR)
    hp = bsq.TrainHyper(**HP)
    W = _stack(4, 256, 512, seed=50 + d + b + h, dtype=dtype)         # 4 layers of one category
    chunks = W.reshape(-1, d)
    n_total = chunks.shape[0]
    g = torch.Generator().manual_seed(7)
    idx = torch.randint(0, n_total, (16384,), generator=g, dtype=torch.int64)
    theta0 = _theta0(d, b, h, seed=60 + d)
    theta = torch.from_numpy(theta0.astype(np.float32))
    err = torch.zeros(1, dtype=torch.int32, device=gpu)
    loss, grad = bsq.bsq_train_grad(cfg, hp, W.to(gpu), theta.to(gpu), idx=idx.to(gpu), err=err)
    loss2, grad2 = bsq.bsq_train_grad(cfg, hp, W.to(gpu), theta.to(gpu), idx=idx.to(gpu))
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    assert torch.equal(grad.view(torch.int32), grad2.view(torch.int32)) and torch.equal(loss, loss2)
    X = oracle.to_f32(chunks)[idx.numpy()]
    (L, L_rec, L_com, L_ent), g_ref = OT.loss_and_grad(theta.numpy().astype(np.float64), X, d, b, h,
                                                        OT.Hyper(**HP))
    got = loss.cpu().numpy().astype(np.float64)
    # L_ent is the difference of two sums of entropies, each at most
    # b ln 2 (and times gamma), which cancel: its error is relative to them
    ent_mag = b * np.log(2.0) * (1.0 + HP["gamma"])
    mags = (abs(L) + HP["lambda_e"] * ent_mag, abs(L_rec), abs(L_com), ent_mag)
    for k, (a, r, mag) in enumerate(zip(got, (L, L_rec, L_com, L_ent), mags)):
        assert abs(a - r) <= 1e-5 * mag, (k, a, r)
    gg = grad.cpu().numpy().astype(np.float64)
    for name, sl in zip(("E", "W1", "b1", "W2", "b2"), _blocks(d, b, h)):
        ref = g_ref[sl]
        rel = np.linalg.norm(gg[sl] - ref) / max(np.linalg.norm(ref), 1e-30)
        say(f"  {name}: |grad - ref| / |ref| = {rel:.2e}")
        assert rel <= 1e-4, name


def test_out_of_range_index_is_reported_and_safe(gpu):
    cfg = bsq.Config(d=8, hidden=8, encoder=bsq.ENC_LINEAR)
    W = _stack(1, 64, 64, seed=3, dtype=torch.float32).to(gpu)
    idx = torch.tensor([0, 5, 512, -1], dtype=torch.int64, device=gpu)     # 512 chunks: 512 and -1 are out of range
    err = torch.zeros(1, dtype=torch.int32, device=gpu)
    theta = torch.from_numpy(_theta0(8, 8, 8, 1).astype(np.float32)).to(gpu)
    bsq.bsq_train_grad(cfg, bsq.TrainHyper(), W, theta, idx=idx, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & bsq.DEVERR_BAD_SET


def test_adam_step_matches_oracle(gpu):
    cfg = bsq.Config(d=8, codebook_bits=16, hidden=16, encoder=bsq.ENC_LINEAR)
    hp = bsq.TrainHyper(**HP)
    P = bsq.bsq_train_param_count(cfg)
    r = np.random.default_rng(5)
    theta = r.normal(0, 0.3, P).astype(np.float32)
    m = r.normal(0, 1e-3, P).astype(np.float32)
    v = np.abs(r.normal(0, 1e-5, P)).astype(np.float32)
    g = r.normal(0, 1e-2, P).astype(np.float32)
    td, md, vd, gd = (torch.from_numpy(a).to(gpu) for a in (theta, m, v, g))
    bsq.bsq_train_adam(cfg, hp, 7, td, gd, md, vd)
    torch.cuda.synchronize()
    # the oracle takes the hyperparameters the kernel receives: fp32 numbers
    # (1 - beta2 of fp32(0.999) differs from 0.001 by 1.3e-5 relative)
    hp32 = OT.Hyper(**{k: float(np.float32(v_)) for k, v_ in hp.__dict__.items()})
    t_ref, m_ref, v_ref = OT.adam(theta.astype(np.float64), g.astype(np.float64), m.astype(np.float64),
                                  v.astype(np.float64), 7, hp32)
    # fp32: about ten roundings in the update, and the rounding of the new
    # parameter and of the subtraction
    u = 2.0 ** -24
    upd = np.abs(t_ref - theta.astype(np.float64))
    bound = 16 * u * upd + 2 * u * np.abs(theta) + 1e-30
    assert np.all(np.abs(td.cpu().numpy() - t_ref) <= bound)
    assert np.all(np.abs(md.cpu().numpy() - m_ref) <= 8 * u * (np.abs(m) + np.abs(g)) + 1e-30)
    assert np.all(np.abs(vd.cpu().numpy() - v_ref) <= 8 * u * (np.abs(v) + g.astype(np.float64) ** 2) + 1e-37)


@pytest.mark.parametrize("d,b", [(8, 8), (8, 16)])
def test_training_run_lowers_loss_and_feeds_the_encoder(d, b, gpu):
    """Category-batched training: 8 layers' chunks of one category, 150 Adam
    steps on mini-batches drawn from the whole stack. The loss falls; the run
    is deterministic; the trained (E, decoder) prepared as a codec encodes a
    layer on the product path bit-exactly as the oracle does with the same
    parameters, with a lower reconstruction error than the untrained codec."""
    say(f"train run d={d} b={b}")
    h = b
    cfg = bsq.Config(d=d, codebook_bits=b, hidden=h, encoder=bsq.ENC_LINEAR, stages=1, protect_num=0)
    hp = bsq.TrainHyper(**HP)
    W = _stack(8, 256, 512, seed=70, dtype=torch.bfloat16).to(gpu)
    n_total = W.numel() // d
    P = bsq.bsq_train_param_count(cfg)
    theta_init = torch.from_numpy(_theta0(d, b, h, seed=71).astype(np.float32)).to(gpu)

    def run(steps, batch=8192):
        theta = theta_init.clone()
        m = torch.zeros(P, device=gpu)
        v = torch.zeros(P, device=gpu)
        gen = torch.Generator(device=gpu).manual_seed(72)
        ws = torch.empty(bsq.bsq_train_workspace_bytes(cfg, batch) + 256, dtype=torch.uint8, device=gpu)
        ws = ws[(-ws.data_ptr()) % 256:]
        losses = []
        for step in range(1, steps + 1):
            idx = torch.randint(0, n_total, (batch,), generator=gen, device=gpu, dtype=torch.int64)
            loss, grad = bsq.bsq_train_grad(cfg, hp, W, theta, idx=idx, ws=ws)
            bsq.bsq_train_adam(cfg, hp, step, theta, grad, m, v)
            losses.append(loss.clone())
        torch.cuda.synchronize()
        return theta, torch.stack(losses).cpu().numpy()

    theta, losses = run(150)
    theta_b, _ = run(150)
    assert torch.equal(theta.view(torch.int32), theta_b.view(torch.int32))
    assert losses[-1, 0] < 0.5 * losses[0, 0]
    say(f"  loss {losses[0, 0]:.4g} -> {losses[-1, 0]:.4g}")

    def codec_of(th):
        E, W1, b1, W2, b2 = OT.unpack(th.cpu().numpy().astype(np.float64), d, b, h)
        dec = synth.StageDecoder(W1=W1.astype(np.float32), b1=b1.astype(np.float32), W2=W2.astype(np.float32),
                                 b2=b2.astype(np.float32))
        dec.E = E.astype(np.float32)
        return [dec]

    oc = oracle.Config(d=d, b=b, stages=1, kind=oracle.KIND_MLP, hidden=h, protect_num=0, encoder=oracle.ENC_LINEAR)
    Wl = W[3]
    errs = []
    for th in (theta_init, theta):
        decs = codec_of(th)
        codec = bsq.bsq_codec_prepare(cfg, decs, device=gpu)
        layer = bsq.bsq_encode(cfg, codec, Wl)
        w_hat = bsq.bsq_decode(cfg, codec, layer, dtype=torch.float32)
        torch.cuda.synchronize()
        enc = oracle.encode(oc, decs, oracle.to_f32(Wl))
        assert_layer_equal(layer, enc, cfg)
        errs.append(float(((w_hat - Wl.float()) ** 2).sum()))
    say(f"  reconstruction error untrained {errs[0]:.4g}, trained {errs[1]:.4g}")
    assert errs[1] < errs[0]
