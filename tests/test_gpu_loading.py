"""First-layers caching with progressive loading on the GPU (Sec. 5.1 "Caching
the first layers"; Sec. 5.3 layer lookup table and elastic eviction).

Parity bar: a step or sampling loop that starts while evicted blocks are
still being copied from the host tier gives bitwise the result of the same
call on a resident model (the deferred per-block modulation and text K/V use
the same kernels and arguments).  The copies are held behind a long GPU job
on another stream, so every call here is enqueued while its loads are
pending and the per-block waits are what orders them.

* 512-px DiT (28 blocks of 58 MB), guidance + Euler update, prefixes
  L_e = 0, 11, 27, 28, evicting and reloading between them;
* the sampling loop with the step-skip cache (block 0 deferred: the cache
  check needs its modulation first);
* reduced MMDiT and the fp32 model;
* error paths: a call that needs an evicted block fails before launching;
  fewer blocks than the resident prefix run without a load."""
import gc

import numpy as np
import pytest
import torch

import synth
import paper_2607_26566_amd as t2i
from gpu_common import DEV, Model, say

pytestmark = pytest.mark.gpu


def gated_copy_stream():
    """A copy stream whose work starts only after ~tens of ms of matmuls."""
    gate, copy = torch.cuda.Stream(), torch.cuda.Stream()
    a = torch.randn(4096, 4096, device=DEV)
    with torch.cuda.stream(gate):
        for _ in range(24):
            a = a @ a * 1e-3
    copy.wait_stream(gate)
    return copy, a


def step_out(M, lats, hw, tx, t=0.7, t_next=0.65, guidance=None):
    x = M.latents_dev(lats)
    v = torch.zeros_like(x)
    g = M.w.guidance if guidance is None else guidance
    t2i.t2i_dit_step(M.m, x, hw, [t] * len(hw), tx, guidance=g, t_next=[t_next] * len(hw),
                     noise_pred=v)
    return x, v


def host_tier(M):
    host = t2i.pack_blocks(M.cfg, M.dev)
    t2i.t2i_dit_host_tier(M.m, host)
    return host


def test_progressive_step_bitwise_dit512():
    w = synth.workload("dit512")
    M = Model(w)
    lats, texts = synth.latents(w), synth.texts(w)
    hw, tx = list(w.requests), M.text_dev(texts)
    x_ref, v_ref = step_out(M, lats, hw, tx)
    torch.cuda.synchronize()
    x_ref, v_ref = x_ref.cpu(), v_ref.cpu()
    host_tier(M)
    L = w.depth
    for keep in (0, 11, 27, 28):
        t2i.t2i_dit_evict(M.m, keep)
        assert t2i.t2i_dit_block_state(M.m) == [0] * keep + [2] * (L - keep)
        copy, _ = gated_copy_stream()
        assert t2i.t2i_dit_load_async(M.m, copy) == L - keep
        st = t2i.t2i_dit_block_state(M.m)
        assert st[:keep] == [0] * keep and all(s == 1 for s in st[keep:]), st
        x, v = step_out(M, lats, hw, tx)
        torch.cuda.synchronize()
        assert t2i.t2i_dit_block_state(M.m) == [0] * L
        say(f"progressive keep={keep}: max |dv| {float((v.cpu() - v_ref).abs().max()):.1e}")
        assert torch.equal(v.cpu(), v_ref) and torch.equal(x.cpu(), x_ref)
    # the reloaded model (arena-resident) is an ordinary resident model now
    x, v = step_out(M, lats, hw, tx)
    torch.cuda.synchronize()
    assert torch.equal(v.cpu(), v_ref)
    del M
    gc.collect()
    torch.cuda.empty_cache()


def test_progressive_sample_with_cache():
    w = synth.reduced(synth.workload("dit512"), name="dit512_d6", depth=6,
                      requests=((32, 32), (24, 40)), guidance=4.5)
    M = Model(w, max_steps=8)
    lats, texts = synth.latents(w), synth.texts(w)
    hw, tx = list(w.requests), M.text_dev(texts)
    toks = [(h // w.patch) * (ww // w.patch) for h, ww in hw]
    n = 8

    def run():
        x = M.latents_dev(lats)
        state = M.m.new_cache_state(toks, 2)
        log, rel = t2i.t2i_dit_sample(M.m, x, hw, tx, n, guidance=w.guidance, cache_tau=0.3,
                                      cache_state=state)
        torch.cuda.synchronize()
        return x.cpu(), np.asarray(log)

    x_ref, log_ref = run()
    host_tier(M)
    for keep in (0, 3):
        t2i.t2i_dit_evict(M.m, keep)
        copy, _ = gated_copy_stream()
        t2i.t2i_dit_load_async(M.m, copy)
        x, log = run()
        say(f"progressive sample keep={keep}: skips {int(log.sum())} of {log.size}")
        assert np.array_equal(log, log_ref) and torch.equal(x, x_ref)
    assert log_ref.sum() > 0          # the cache did skip steps


def test_progressive_mmdit_and_fp32():
    cases = [
        synth.reduced(synth.workload("mmdit1024"), name="mmdit_load", hidden=256, heads=2,
                      head_dim=128, depth=4, mlp_hidden=512, text_dim=128, text_tokens=64,
                      requests=((32, 32),)),
        synth.workload("tiny_f32"),
    ]
    for w in cases:
        M = Model(w)
        lats, texts = synth.latents(w), synth.texts(w)
        hw, tx = list(w.requests), M.text_dev(texts)
        _, v_ref = step_out(M, lats, hw, tx, guidance=w.guidance)
        torch.cuda.synchronize()
        v_ref = v_ref.cpu()
        host_tier(M)
        t2i.t2i_dit_evict(M.m, 1)
        copy, _ = gated_copy_stream()
        t2i.t2i_dit_load_async(M.m, copy)
        _, v = step_out(M, lats, hw, tx, guidance=w.guidance)
        torch.cuda.synchronize()
        say(f"progressive {w.name}: equal={torch.equal(v.cpu(), v_ref)}")
        assert torch.equal(v.cpu(), v_ref)


def test_evicted_blocks_are_rejected():
    w = synth.reduced(synth.workload("dit512"), name="dit512_d4", depth=4, requests=((32, 32),))
    M = Model(w)
    lats, texts = synth.latents(w), synth.texts(w)
    hw, tx = list(w.requests), M.text_dev(texts)
    x = M.latents_dev(lats)
    hid = torch.zeros((w.tokens(0) * w.branches, w.hidden), device=DEV)
    t2i.t2i_dit_step(M.m, x, hw, [0.5], tx, n_blocks=2, hidden_out=hid)
    torch.cuda.synchronize()
    ref = hid.clone()
    host_tier(M)
    t2i.t2i_dit_evict(M.m, 2)
    hid.zero_()
    # blocks 0, 1 are resident: a two-block call needs no load
    t2i.t2i_dit_step(M.m, x, hw, [0.5], tx, n_blocks=2, hidden_out=hid)
    torch.cuda.synchronize()
    assert torch.equal(hid, ref)
    with pytest.raises(t2i.T2IError, match="evicted"):
        t2i.t2i_dit_step(M.m, x, hw, [0.5], tx)
    state = M.m.new_cache_state([w.tokens(0)], 1)
    with pytest.raises(t2i.T2IError, match="evicted"):
        t2i.t2i_dit_sample(M.m, x, hw, tx, 1)
    t2i.t2i_dit_evict(M.m, 0)
    with pytest.raises(t2i.T2IError, match="evicted"):
        t2i.t2i_cache_check(M.m, x, hw, [0.5], 0, 4, 0.1, state)
    with pytest.raises(t2i.T2IError):
        t2i.t2i_dit_evict(M.m, 5)
    assert t2i.t2i_dit_load_async(M.m) == 4
    t2i.t2i_dit_step(M.m, x, hw, [0.5], tx, n_blocks=2, hidden_out=hid)
    torch.cuda.synchronize()
    assert torch.equal(hid, ref)
    # pageable host memory is refused, and so is an arena outside device memory
    hb = M.m.host_blocks
    with pytest.raises(t2i.T2IError, match="page-locked"):
        t2i.t2i_dit_host_tier(M.m, torch.zeros_like(hb, pin_memory=False))
    lib = t2i.load()
    assert lib.t2i_dit_host_tier(M.m.h, hb.data_ptr(), hb.data_ptr(), hb.numel()) == 1
    assert b"device memory" in lib.t2i_last_error(M.m.h)
