"""The step's callback input (`control_outputs`): per-block residuals added to
the residual stream partway through the forward, each optionally gated by a
producer's event that the step waits for only at the consuming block.

* fp32 model: the velocity with residuals after both blocks against the
  oracle's forward with the same control input (1e-4);
* 512-px bf16 model: a producer on a second stream writes the residuals
  after a long-running kernel and records events; the step, launched right
  away, must give bitwise the result of a call whose residuals were written
  beforehand; the residual stream after the injecting block differs from the
  one without control by exactly the residual (fp32 rounding);
* reduced MMDiT: residual on the image stream against the oracle."""
import gc

import numpy as np
import pytest
import torch

import synth
import paper_2607_26566_amd as t2i
from oracle import dit, mmdit
from gpu_common import DEV, Model, rel_l2, say

pytestmark = pytest.mark.gpu


def step_v(M, lats, hw, t, tx, **kw):
    x = M.latents_dev(lats)
    npred = torch.zeros_like(x)
    t2i.t2i_dit_step(M.m, x, hw, t, tx, noise_pred=npred, **kw)
    torch.cuda.synchronize()
    return npred.cpu().numpy().astype(np.float64)


def test_control_fp32_against_oracle():
    w = synth.workload("tiny_f32")
    M = Model(w)
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    N, D = w.tokens(0), w.hidden
    rs = [synth.normal(w.seed, (9, b), (N, D), 0.1) for b in range(w.depth)]
    ctl = [(b, torch.from_numpy(rs[b]).to(DEV), None) for b in range(w.depth)]
    v = step_v(M, lats, hw, [0.6], M.text_dev(texts), control=ctl)
    ref = dit.forward(M.W, w, lats[0], 0.6, texts[0],
                      control={b: rs[b].astype(np.float64) for b in range(w.depth)}).ravel()
    err = rel_l2(v, ref)
    say(f"control fp32: v rel_l2 {err:.2e}")
    assert err < 1e-4
    v0 = step_v(M, lats, hw, [0.6], M.text_dev(texts))
    assert rel_l2(v0, ref) > 1e-3          # the residuals do change the result


def test_control_events_from_a_producer_stream():
    w = synth.workload("dit512")
    M = Model(w)
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    tx = M.text_dev(texts)
    N, D = w.tokens(0), w.hidden
    blocks = (3, 20)
    vals = {b: torch.from_numpy(synth.normal(w.seed, (9, b), (N, D), 0.05)).to(DEV)
            for b in blocks}
    # reference: residuals in place before the call
    bufs = {b: vals[b].clone() for b in blocks}
    torch.cuda.synchronize()
    v_ref = step_v(M, lats, hw, [0.7], tx, control=[(b, bufs[b], None) for b in blocks])
    # producer: a long matmul chain, then the residual copies, on its own stream
    for b in blocks:
        bufs[b].zero_()
    torch.cuda.synchronize()
    a = torch.randn(4096, 4096, device=DEV)
    prod = torch.cuda.Stream()
    events = {}
    with torch.cuda.stream(prod):
        for b in blocks:
            for _ in range(8):
                a = a @ a * 1e-3
            bufs[b].copy_(vals[b])
            events[b] = torch.cuda.Event()
            events[b].record(prod)
    v_ev = step_v(M, lats, hw, [0.7], tx, control=[(b, bufs[b], events[b]) for b in blocks])
    say(f"control events: max |diff| vs pre-written {np.abs(v_ev - v_ref).max():.3e}")
    assert np.array_equal(v_ev, v_ref)
    # the residual stream after block 3 moves by exactly the residual
    hid = torch.zeros((N, D), dtype=torch.float32, device=DEV)
    outs = []
    for ctl in (None, [(3, vals[3], None)]):
        x = M.latents_dev(lats)
        t2i.t2i_dit_step(M.m, x, hw, [0.7], tx, n_blocks=4, hidden_out=hid, control=ctl)
        torch.cuda.synchronize()
        outs.append(hid.cpu().numpy().astype(np.float64))
    r = vals[3].cpu().numpy().astype(np.float64)
    assert rel_l2(outs[1] - outs[0], r) < 1e-6
    del M
    gc.collect()
    torch.cuda.empty_cache()


def test_control_mmdit_image_stream():
    w = synth.reduced(synth.workload("mmdit1024"), name="mmdit_ctl", hidden=256, heads=2,
                      head_dim=128, depth=3, mlp_hidden=512, text_dim=128, text_tokens=64,
                      requests=((32, 32),))
    M = Model(w)
    lats, texts = synth.latents(w), synth.texts(w)
    N, D = w.tokens(0), w.hidden
    r = synth.normal(w.seed, (9, 1), (N, D), 0.1)
    v = step_v(M, lats, list(w.requests), [0.5], M.text_dev(texts),
               control=[(1, torch.from_numpy(r).to(DEV), None)])
    ref = mmdit.forward(M.W, w, lats[0], 0.5, texts[0], control={1: r.astype(np.float64)})[0].ravel()
    err = rel_l2(v, ref)
    say(f"control mmdit: v rel_l2 {err:.2e}")
    assert err < 1e-2
