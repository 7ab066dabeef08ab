"""Parity of the joint-attention (MMDiT-style) HIP path with the oracle.

* Reduced width, full structure (3 joint blocks, d = 128, 16-channel latents,
  two requests of different grid shapes packed together, one of them
  non-square): velocity of every request with and without guidance against
  the oracle's model velocity; packed == each request alone, bitwise; the
  sampling loop with the step-skip cache against step-by-step calls (bitwise)
  and its decisions against the oracle's rule.
* Full size (3072 wide, 24 heads of 128, 4096 image + 512 text tokens): the
  residual streams after the embeddings, the update of blocks 0, 1 and 18 on
  sampled rows of both streams, and the final layer + Euler update of a whole
  19-block step.  Only blocks 0 and 1 hold their own weights; blocks 2..18
  reuse them alternately (the oracle is given the same aliasing), which keeps
  the host copy of the weights small.

Tolerances: relative L2 1e-2 per bf16 block update / velocity (as for the
cross-attention model), 1e-5 for the fp32 embeddings, 1e-4 for the final
layer evaluated from the GPU's own residual stream."""
import gc

import numpy as np
import pytest
import torch

import synth
import paper_2607_26566_amd as t2i
from oracle import dit, mmdit, sampler
from gpu_common import DEV, Model, rel_l2, say, to_dev

pytestmark = pytest.mark.gpu

# MLP width 2048: the text stream's down-projection (64 rows, K = 2048) takes
# the split-K path
SMALL = synth.reduced(synth.workload("mmdit1024"), name="mmdit_small", hidden=256, heads=2,
                      head_dim=128, depth=3, mlp_hidden=2048, text_dim=128, text_tokens=64,
                      requests=((32, 32), (16, 48)), guidance=4.5, steps=8)


def step_gpu(M, lats_dev, hw, t, texts_dev, guidance=1.0, t_next=None, **kw):
    npred = torch.zeros_like(lats_dev)
    t2i.t2i_dit_step(M.m, lats_dev, hw, t, texts_dev, guidance=guidance, t_next=t_next,
                     noise_pred=npred, **kw)
    torch.cuda.synchronize()
    return npred.cpu().numpy().astype(np.float64)


@pytest.fixture(scope="module")
def small():
    M = Model(SMALL)
    yield M
    del M
    gc.collect()
    torch.cuda.empty_cache()


def test_mmdit_small_velocity_with_and_without_guidance(small):
    M, w = small, small.w
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    ts = [0.9, 0.35]
    tx = M.text_dev(texts)
    shapes = [l.shape for l in lats]
    for g in (1.0, w.guidance):
        x = M.latents_dev(lats)
        v = M.split(step_gpu(M, x, hw, ts, tx, guidance=g), shapes)
        for r in range(w.n_req):
            ref, _ = sampler.model_velocity(M.W, w, lats[r], ts[r], texts[r], g)
            err = rel_l2(v[r], ref)
            say(f"mmdit small guidance {g} request {r}: v rel_l2 {err:.2e}")
            assert err < 1e-2


def test_mmdit_small_packed_equals_alone(small):
    M, w = small, small.w
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    ts = [0.6, 0.45]
    x = M.latents_dev(lats)
    v = M.split(step_gpu(M, x, hw, ts, M.text_dev(texts), guidance=w.guidance),
                [l.shape for l in lats])
    for r in range(w.n_req):
        xr = M.latents_dev([lats[r]])
        vr = step_gpu(M, xr, [hw[r]], [ts[r]], M.text_dev([texts[r]]), guidance=w.guidance)
        assert np.array_equal(vr, v[r].ravel()), r


def test_mmdit_small_hidden_streams_and_block_updates(small):
    """hidden_out holds [image rows; text rows]; each block's update of both
    streams matches the oracle's block on the GPU's own input."""
    M, w = small, small.w
    lats, texts = synth.latents(w)[:1], synth.texts(w)[:1]
    hw = [w.requests[0]]
    N, T, D = w.tokens(0), w.text_tokens, w.hidden
    t = 0.7
    hid = torch.zeros((N + T, D), dtype=torch.float32, device=DEV)
    got = {}
    for nb in range(w.depth + 1):
        x = M.latents_dev(lats)
        t2i.t2i_dit_step(M.m, x, hw, [t], M.text_dev(texts), n_blocks=nb, hidden_out=hid)
        torch.cuda.synchronize()
        got[nb] = hid.cpu().numpy().astype(np.float64)
    xt0, xi0 = mmdit.embed(M.W, w, lats[0], texts[0])
    assert rel_l2(got[0][:N], xi0) < 1e-5 and rel_l2(got[0][N:], xt0) < 1e-5
    c = dit.conditioning(M.W, w, t)
    rows, cols = mmdit.grid_positions(hw[0][0] // w.patch, hw[0][1] // w.patch)
    for b in range(w.depth):
        xi, xt = got[b][:N], got[b][N:]
        nt, ni = mmdit.joint_block(M.W, w, b, xt, xi, c, rows, cols)
        ei = rel_l2(got[b + 1][:N] - xi, ni - xi)
        et = rel_l2(got[b + 1][N:] - xt, nt - xt)
        say(f"mmdit small block {b}: image update {ei:.2e} text update {et:.2e}")
        assert ei < 1e-2 and et < 1e-2


def test_mmdit_small_cached_sampling(small):
    """8 steps with the step-skip rule: decisions equal the oracle's rule on
    the GPU's own latents; the sampling loop equals step-by-step calls."""
    M, w = small, small.w
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    n, tau = w.steps, 0.3
    sched = np.stack([sampler.schedule(n) for _ in lats], axis=1)
    tx = M.text_dev(texts)
    x = M.latents_dev(lats)
    toks = [w.tokens(r) for r in range(w.n_req)]
    state = M.m.new_cache_state(toks, 2)
    shapes = [l.shape for l in lats]
    states = [sampler.CacheState() for _ in lats]
    vstates = [sampler.CacheState() for _ in lats]   # the oracle's cached residuals
    skips = []
    n_vel_skips = 0
    for k in range(n):
        xk = M.split(x.cpu().numpy(), shapes)
        rel, skip = t2i.t2i_cache_check(M.m, x, hw, sched[k], k, n, tau, state, branches=2)
        for r in range(w.n_req):
            m = np.asarray(mmdit.cache_signal(M.W, w, xk[r].astype(np.float64), sched[k, r]),
                           dtype=np.float32)
            st = states[r]
            d = float("nan") if st.m_prev is None else sampler.rel_l1(m, st.m_prev)
            has_r = st.residual is not None and st.m_prev is not None
            sk, st.acc = sampler.cache_rule(st.acc, d, k, n, tau, sampler.MODE_ACCUMULATE, has_r)
            if not sk:
                st.residual = True
            st.m_prev = m
            if k > 0:
                assert abs(rel[r] - d) <= 1e-6 * abs(d) + 1e-12, (k, r, rel[r], d)
            assert bool(skip[r]) == sk, (k, r)
        skips.append(skip)
        npred = torch.zeros_like(x)
        t2i.t2i_dit_step(M.m, x, hw, sched[k], tx, guidance=w.guidance, t_next=sched[k + 1],
                         skip=skip, cache_state=state, noise_pred=npred)
        torch.cuda.synchronize()
        # guided velocity of every request, computed or skipped (teacher-forced:
        # the oracle refreshes its own residual at each computed step)
        vk = M.split(npred.cpu().numpy().astype(np.float64), shapes)
        for r in range(w.n_req):
            ref, _ = sampler.model_velocity(M.W, w, xk[r].astype(np.float64), sched[k, r],
                                            texts[r], w.guidance, vstates[r], skip=bool(skip[r]))
            err = rel_l2(vk[r], ref)
            assert err < 1e-2, (k, r, bool(skip[r]), err)
            if skip[r]:
                n_vel_skips += 1
                say(f"mmdit small cache step {k} request {r}: skipped-step v rel_l2 {err:.2e}")
    assert n_vel_skips > 0
    say(f"mmdit small cache: {int(np.sum(skips))} skipped request-steps of {n * w.n_req}")
    x2 = M.latents_dev(lats)
    state2 = M.m.new_cache_state(toks, 2)
    log, _ = t2i.t2i_dit_sample(M.m, x2, hw, tx, n, guidance=w.guidance, timesteps=sched,
                                cache_tau=tau, cache_state=state2)
    torch.cuda.synchronize()
    assert np.array_equal(log, np.array(skips, dtype=np.uint8))
    assert np.array_equal(x2.cpu().numpy(), x.cpu().numpy())


# ---------------------------------------------------------------- full size

def test_mmdit1024_full_size_sampled():
    w = synth.workload("mmdit1024")
    cfg = t2i.Config.from_shape(w)
    table = t2i.weight_table(cfg)
    assert table == [(n, tuple(s)) for n, s in mmdit.weight_layout(w)]
    per, nreal = 20, 2
    n_tab = len(table)
    head, tail = list(range(8)), list(range(n_tab - 4, n_tab))
    real = list(range(8, 8 + nreal * per))
    host = synth.weights(w, table, pick=head + real + tail)
    by_index = dict(zip(head + real + tail, host))

    def alias(i):
        if 8 <= i < n_tab - 4:
            return 8 + (i - 8) % (nreal * per)
        return i

    dev_of = {i: to_dev(a, "bf16") for i, a in by_index.items()}
    m = t2i.t2i_dit_init(cfg, [dev_of[alias(i)] for i in range(n_tab)])
    # oracle weights: embeddings, final layer, blocks 0, 1 and 18 (= block 0's)
    f64 = {}
    W = {}
    for i, (name, shape) in enumerate(table):
        if name.startswith("blocks.") and name.split(".")[1] not in ("0", "1", "18"):
            continue
        j = alias(i)
        if j not in f64:
            f64[j] = np.asarray(by_index[j], dtype=np.float64).reshape(shape)
        W[name] = f64[j]
    del host, by_index
    say("mmdit1024 weights ready")
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    tx = to_dev(np.stack(texts), "bf16")
    N, T, D = w.tokens(0), w.text_tokens, w.hidden
    t, tn = 1.0, 1.0 - 1.0 / w.steps
    hid = torch.zeros((N + T, D), dtype=torch.float32, device=DEV)
    got = {}
    for nb in (0, 1, 2, 18, 19):
        x = torch.from_numpy(lats[0].ravel().astype(np.float32)).to(DEV)
        t2i.t2i_dit_step(m, x, hw, [t], tx, n_blocks=nb, hidden_out=hid)
        torch.cuda.synchronize()
        got[nb] = hid.cpu().numpy().astype(np.float64)
    xt0, xi0 = mmdit.embed(W, w, lats[0], texts[0])
    assert rel_l2(got[0][:N], xi0) < 1e-5 and rel_l2(got[0][N:], xt0) < 1e-5
    c = dit.conditioning(W, w, t)
    rows, cols = mmdit.grid_positions(hw[0][0] // w.patch, hw[0][1] // w.patch)
    sel_i = np.r_[np.arange(0, N, 61), N - 1]
    sel_t = np.r_[np.arange(0, T, 29), T - 1]
    for b in (0, 1, 18):
        xi, xt = got[b][:N], got[b][N:]
        rt, ri = mmdit.joint_block_rows(W, w, b, xt, xi, c, rows, cols, sel_t, sel_i)
        ei = rel_l2(got[b + 1][:N][sel_i] - xi[sel_i], ri - xi[sel_i])
        et = rel_l2(got[b + 1][N:][sel_t] - xt[sel_t], rt - xt[sel_t])
        say(f"mmdit1024 block {b}: image update {ei:.2e} text update {et:.2e}")
        assert ei < 1e-2 and et < 1e-2
    # the whole step: final layer and Euler from the GPU's final image stream
    x = torch.from_numpy(lats[0].ravel().astype(np.float32)).to(DEV)
    npred = torch.zeros_like(x)
    t2i.t2i_dit_step(m, x, hw, [t], tx, t_next=[tn], noise_pred=npred)
    torch.cuda.synchronize()
    ref = dit.final_layer(W, w, got[19][:N], c, hw[0][0], hw[0][1])
    assert rel_l2(npred.cpu().numpy(), ref.ravel()) < 1e-4
    xr = sampler.euler_update(lats[0].astype(np.float64), ref, t, tn)
    assert rel_l2(x.cpu().numpy(), xr.ravel()) < 1e-5
    del m, dev_of
    gc.collect()
    torch.cuda.empty_cache()
