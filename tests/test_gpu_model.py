"""Step- and sample-level parity of the HIP path (through the C ABI) with the
oracle, on the seeded workloads.

Tolerances (relative L2 per output tensor): the fp32 model 1e-4, free running
over the whole sample; bf16 models 1e-2 per step output, teacher-forced (the
oracle starts every compared step from the GPU's latent).  Cache-skip
decisions must be identical."""
import gc
import math

import numpy as np
import pytest
import torch

import synth
import paper_2607_26566_amd as t2i
from oracle import dit, sampler
from gpu_common import DEV, Model, rel_l2, say, to_host

pytestmark = pytest.mark.gpu


def step_gpu(M, lats_dev, hw, t, texts_dev, guidance=1.0, t_next=None, **kw):
    npred = torch.zeros_like(lats_dev)
    t2i.t2i_dit_step(M.m, lats_dev, hw, t, texts_dev, guidance=guidance, t_next=t_next,
                     noise_pred=npred, **kw)
    torch.cuda.synchronize()
    return npred.cpu().numpy().astype(np.float64)


# ---------------------------------------------------------------- fp32 model

def test_tiny_f32_free_running_sample():
    w = synth.workload("tiny_f32")
    M = Model(w)
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    # oracle, free running
    ref_x, log = sampler.sample(M.W, w, lats, texts, [1.0], w.steps, keep=True)
    # GPU step by step from its own latents
    x = M.latents_dev(lats)
    tx = M.text_dev(texts)
    s = sampler.schedule(w.steps)
    for k in range(w.steps):
        v = step_gpu(M, x, hw, [s[k]], tx, t_next=[s[k + 1]])
        err = rel_l2(v, log["v"][k][0].ravel())
        say(f"tiny step {k}: v rel_l2 {err:.2e}")
        assert err < 1e-4
    x_step = x.cpu().numpy()
    assert rel_l2(x_step, ref_x[0].ravel()) < 1e-4
    # the sampling loop gives the same result as the step-by-step calls, bitwise
    x2 = M.latents_dev(lats)
    skips, _ = t2i.t2i_dit_sample(M.m, x2, hw, tx, w.steps)
    torch.cuda.synchronize()
    assert np.array_equal(x2.cpu().numpy(), x_step)
    assert not skips.any()


# ---------------------------------------------------------------- 512 px bf16

@pytest.fixture(scope="module")
def dit512():
    M = Model(synth.workload("dit512"))
    yield M
    del M
    gc.collect()
    torch.cuda.empty_cache()


def test_dit512_teacher_forced_steps(dit512):
    M, w = dit512, dit512.w
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    x = M.latents_dev(lats)
    tx = M.text_dev(texts)
    s = sampler.schedule(w.steps)
    check = {0, 4, 8, 12, 16, w.steps - 1}
    for k in range(w.steps):
        x_k = x.cpu().numpy().astype(np.float64).reshape(lats[0].shape)
        v = step_gpu(M, x, hw, [s[k]], tx, t_next=[s[k + 1]])
        if k in check:
            ref = dit.forward(M.W, w, x_k, s[k], texts[0])
            err = rel_l2(v, ref.ravel())
            say(f"dit512 step {k}: v rel_l2 {err:.2e}")
            assert err < 1e-2


@pytest.mark.parametrize("text_tokens", [8, 64, 128, 200])
def test_cross_dit_text_lengths(text_tokens):
    """Cross-attention over one key tile (8), one full tile (64), two full
    tiles (128) and four tiles, the last ragged (200: text longer than 128
    keys runs the pipelined attention kernel), two requests and guidance 4.5,
    at full width, 2 blocks."""
    w = synth.reduced(synth.workload("dit512"), depth=2, text_tokens=text_tokens,
                      requests=((32, 32), (16, 48)), guidance=4.5)
    M = Model(w)
    lats, texts = synth.latents(w), synth.texts(w)
    tx = M.text_dev(texts)
    x = M.latents_dev(lats)
    v = step_gpu(M, x, list(w.requests), [0.7, 0.3], tx, guidance=w.guidance)
    parts = M.split(v, [l.shape for l in lats])
    for r, t in enumerate((0.7, 0.3)):
        vc = dit.forward(M.W, w, lats[r], t, texts[r])
        vu = dit.forward(M.W, w, lats[r], t, None)
        err = rel_l2(parts[r].ravel(), sampler.cfg_combine(vc, vu, w.guidance).ravel())
        say(f"cross text {text_tokens} request {r}: v rel_l2 {err:.2e}")
        assert err < 1e-2
    del M
    gc.collect()
    torch.cuda.empty_cache()


def test_dit512_determinism_and_block_updates(dit512):
    M, w = dit512, dit512.w
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    tx = M.text_dev(texts)
    outs = []
    for _ in range(2):
        x = M.latents_dev(lats)
        outs.append(step_gpu(M, x, hw, [0.7], tx, t_next=[0.65]) )
        outs.append(x.cpu().numpy())
    assert np.array_equal(outs[0], outs[2]) and np.array_equal(outs[1], outs[3])
    # block-by-block: GPU residual stream before/after blocks b, compared as updates
    N = w.tokens(0)
    hid = torch.zeros((N, w.hidden), dtype=torch.float32, device=DEV)
    c = dit.conditioning(M.W, w, 0.7)
    y = dit.text_project(M.W, w, texts[0])
    prev = None
    for nb in (0, 1, 2, 14, 15, 27, 28):
        x = M.latents_dev(lats)
        t2i.t2i_dit_step(M.m, x, hw, [0.7], tx, n_blocks=nb, hidden_out=hid)
        torch.cuda.synchronize()
        cur = hid.cpu().numpy().astype(np.float64)
        if nb == 0:
            ref0 = dit.embed(M.W, w, lats[0])
            assert rel_l2(cur, ref0) < 1e-5
        elif prev is not None and prev[0] == nb - 1:
            b = nb - 1
            ref = dit.block(M.W, w, b, prev[1], y, dit.block_modulation(M.W, w, c, b))
            err = rel_l2(cur - prev[1], ref - prev[1])
            say(f"dit512 block {b}: update rel_l2 {err:.2e}")
            assert err < 1e-2
        prev = (nb, cur)


# ---------------------------------------------------------------- 1024 px CFG bf16

@pytest.fixture(scope="module")
def dit1024():
    M = Model(synth.workload("dit1024_cfg"))
    yield M
    del M
    gc.collect()
    torch.cuda.empty_cache()


def test_dit1024_cfg_reduced_resolution_step(dit1024):
    """Full width and depth, 256 px image (256 tokens per branch), guidance 4.5."""
    M, w = dit1024, dit1024.w
    lat = synth.normal(w.seed, (0, 7), (4, 32, 32))
    text = synth.texts(w)[0]
    tx = M.text_dev([text])
    for g in (4.5, 1.0):
        x = M.latents_dev([lat])
        v = step_gpu(M, x, [(32, 32)], [0.6], tx, guidance=g, t_next=[0.55])
        vc = dit.forward(M.W, w, lat, 0.6, text)
        vu = dit.forward(M.W, w, lat, 0.6, None) if g != 1.0 else None
        ref = vc if g == 1.0 else sampler.cfg_combine(vc, vu, g)
        err = rel_l2(v, ref.ravel())
        say(f"dit1024 256px guidance {g}: v rel_l2 {err:.2e}")
        assert err < 1e-2
        # x_{k+1} = x_k + dt v: its error is |dt| times the velocity's
        xr = sampler.euler_update(lat.astype(np.float64), ref, 0.6, 0.55)
        dx = np.linalg.norm(x.cpu().numpy() - xr.ravel())
        assert dx <= 0.05 * 1e-2 * np.linalg.norm(ref) + 1e-6 * np.linalg.norm(xr)


def test_dit1024_cfg_full_size_sampled(dit1024):
    """4096 tokens x 2 branches: embed exactly, blocks 0 and 27 on sampled rows,
    final layer + guidance + Euler on every element."""
    M, w = dit1024, dit1024.w
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    tx = M.text_dev(texts)
    N, D = w.tokens(0), w.hidden
    t, tn = 1.0, 0.95
    hid = torch.zeros((2 * N, D), dtype=torch.float32, device=DEV)
    c = dit.conditioning(M.W, w, t)
    ys = [dit.text_project(M.W, w, texts[0]),
          dit.text_project(M.W, w, np.zeros((w.text_tokens, w.text_dim)))]
    rows = np.r_[np.arange(0, N, 131), N - 1]
    got = {}
    for nb in (0, 1, 27, 28):
        x = M.latents_dev(lats)
        t2i.t2i_dit_step(M.m, x, hw, [t], tx, guidance=w.guidance, n_blocks=nb, hidden_out=hid)
        torch.cuda.synchronize()
        got[nb] = hid.cpu().numpy().astype(np.float64)
    x0 = dit.embed(M.W, w, lats[0])
    assert rel_l2(got[0][:N], x0) < 1e-5 and np.array_equal(got[0][:N], got[0][N:])
    for b in (0, 27):
        mod = dit.block_modulation(M.W, w, c, b)
        for br in range(2):
            xin = got[b][br * N:(br + 1) * N]
            ref = dit.block_rows(M.W, w, b, xin, ys[br], mod, rows)
            out = got[b + 1][br * N:(br + 1) * N][rows]
            err = rel_l2(out - xin[rows], ref - xin[rows])
            say(f"dit1024 block {b} branch {br}: update rel_l2 {err:.2e}")
            assert err < 1e-2
    # the full step: final layer, guidance and Euler from the GPU's final stream
    x = M.latents_dev(lats)
    v = step_gpu(M, x, hw, [t], tx, guidance=w.guidance, t_next=[tn])
    h, ww = hw[0]
    vc = dit.final_layer(M.W, w, got[28][:N], c, h, ww)
    vu = dit.final_layer(M.W, w, got[28][N:], c, h, ww)
    ref = sampler.cfg_combine(vc, vu, w.guidance)
    assert rel_l2(v, ref.ravel()) < 1e-4
    assert rel_l2(x.cpu().numpy(), sampler.euler_update(lats[0].astype(np.float64), ref, t, tn).ravel()) < 1e-5


def _oracle_blocks_threaded(M, w, x_k, t, texts):
    """The oracle's residual stream after every block for both guidance
    branches (conditional, unconditional), each branch in its own thread so
    that their single-threaded elementwise parts overlap; progress per block."""
    import threading
    c = dit.conditioning(M.W, w, t)
    x0 = dit.embed(M.W, w, x_k)
    out = [None, None]

    def run(br):
        txt = texts if br == 0 else np.zeros((w.text_tokens, w.text_dim))
        y = dit.text_project(M.W, w, txt)
        x = x0
        for b in range(w.depth):
            x = dit.block(M.W, w, b, x, y, dit.block_modulation(M.W, w, c, b))
            if b % 7 == 6:
                say(f"  oracle branch {br}: {b + 1} blocks")
        out[br] = x
    th = [threading.Thread(target=run, args=(br,)) for br in (0, 1)]
    for t_ in th:
        t_.start()
    for t_ in th:
        t_.join()
    return c, x0, out


def _per_row_rel(got, ref):
    """Relative L2 error of every row (last axis)."""
    num = np.linalg.norm(got - ref, axis=-1)
    den = np.linalg.norm(ref, axis=-1)
    return num / den


@pytest.mark.timeout(900)
def test_dit1024_cfg_full_step_every_element(dit1024):
    """The headline step at full size, teacher-forced: 4096 tokens x 2
    guidance branches through all 28 blocks.  The GPU runs steps 0..9 on its
    own, then step 10 is compared with the oracle started from the GPU's x_10:
    every element of the residual stream after the blocks (each branch, also
    row by row), of each branch's velocity before guidance, of the guided
    velocity and of x_11."""
    M, w = dit1024, dit1024.w
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    tx = M.text_dev(texts)
    N, D, g = w.tokens(0), w.hidden, w.guidance
    s = sampler.schedule(w.steps)
    k = 10
    x = M.latents_dev(lats)
    for j in range(k):
        t2i.t2i_dit_step(M.m, x, hw, [s[j]], tx, guidance=g, t_next=[s[j + 1]])
    torch.cuda.synchronize()
    x_k = x.cpu().numpy().astype(np.float64).reshape(lats[0].shape)
    hid = torch.zeros((2 * N, D), dtype=torch.float32, device=DEV)
    xg = x.clone()
    v = step_gpu(M, xg, hw, [s[k]], tx, guidance=g, t_next=[s[k + 1]], hidden_out=hid)
    x_next = xg.cpu().numpy().astype(np.float64)
    hid_g = hid.cpu().numpy().astype(np.float64)
    # guidance 0 returns the unconditional branch of the same two-branch step
    v_u = step_gpu(M, x.clone(), hw, [s[k]], tx, guidance=0.0)
    v_c = v_u + (v - v_u) / g
    say("dit1024 full step: GPU done, oracle running")
    c, x0, xl = _oracle_blocks_threaded(M, w, x_k, s[k], texts[0])
    h, ww = hw[0]
    for br in range(2):
        got = hid_g[br * N:(br + 1) * N]
        err = rel_l2(got - x0, xl[br] - x0)
        rows = _per_row_rel(got - x0, xl[br] - x0)
        say(f"dit1024 full step branch {br}: block residual rel_l2 {err:.2e}, "
            f"worst row {rows.max():.2e} (row {int(rows.argmax())})")
        assert err < 1e-2 and rows.max() < 3e-2
    vc_ref = dit.final_layer(M.W, w, xl[0], c, h, ww)
    vu_ref = dit.final_layer(M.W, w, xl[1], c, h, ww)
    v_ref = sampler.cfg_combine(vc_ref, vu_ref, g)
    for name, got, ref in (("v_c", v_c, vc_ref), ("v_u", v_u, vu_ref), ("v", v, v_ref)):
        err = rel_l2(got, ref.ravel())
        # per token: the p x p x C values of one patch
        tok = _per_row_rel(dit.patchify(got.reshape(ref.shape), w.patch),
                           dit.patchify(ref, w.patch))
        say(f"dit1024 full step {name}: rel_l2 {err:.2e}, worst token {tok.max():.2e}")
        assert err < 1e-2 and tok.max() < 3e-2
    xr = sampler.euler_update(x_k, v_ref, s[k], s[k + 1])
    err = rel_l2(x_next, xr.ravel())
    say(f"dit1024 full step x_k+1: rel_l2 {err:.2e}")
    assert err < 1e-2
    assert np.linalg.norm(x_next - xr.ravel()) <= \
        abs(s[k + 1] - s[k]) * 1e-2 * np.linalg.norm(v_ref) + 1e-6 * np.linalg.norm(xr)


# ---------------------------------------------------------------- packed multi-request

@pytest.fixture(scope="module")
def packed8():
    w = synth.workload("packed8")
    M = Model(w)
    yield M
    del M
    gc.collect()
    torch.cuda.empty_cache()


def test_packed_equals_each_request_alone(packed8):
    M, w = packed8, packed8.w
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    ts = list(synth.start_times(w))
    tx = M.text_dev(texts)
    x = M.latents_dev(lats)
    v_packed = step_gpu(M, x, hw, ts, tx)
    shapes = [l.shape for l in lats]
    parts = M.split(v_packed, shapes)
    for r in range(w.n_req):
        xr = M.latents_dev([lats[r]])
        vr = step_gpu(M, xr, [hw[r]], [ts[r]], M.text_dev([texts[r]]))
        assert np.array_equal(vr, parts[r].ravel()), r
    # oracle parity on the 256 px and 512 px requests
    for r in range(6):
        ref = dit.forward(M.W, w, lats[r], ts[r], texts[r])
        err = rel_l2(parts[r], ref)
        say(f"packed request {r}: v rel_l2 {err:.2e}")
        assert err < 1e-2


def test_packed_cache_decisions_match_oracle(packed8):
    """20 steps, tau = 0.1: the GPU decides from its own latents; the oracle
    recomputes m_k from the same latents and applies the rule on its own."""
    M, w = packed8, packed8.w
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    t0 = synth.start_times(w)
    n = w.steps
    sched = np.stack([sampler.schedule(n, a) for a in t0], axis=1)   # [n+1, R]
    tx = M.text_dev(texts)
    x = M.latents_dev(lats)
    toks = [w.tokens(r) for r in range(w.n_req)]
    state = M.m.new_cache_state(toks, 1)
    shapes = [l.shape for l in lats]
    states = [sampler.CacheState() for _ in lats]
    gpu_skips, margins = [], []
    # velocity parity of the 256-px requests on every step, computed or
    # skipped: the oracle keeps its own cached residual, refreshed at each
    # computed step from the GPU's latent (teacher-forced)
    vel_req = [r for r in range(w.n_req) if w.tokens(r) <= 256]
    vstates = {r: sampler.CacheState() for r in vel_req}
    n_vel_skips = 0
    for k in range(n):
        xk = M.split(x.cpu().numpy(), shapes)
        rel, skip = t2i.t2i_cache_check(M.m, x, hw, sched[k], k, n, w.cache_tau, state)
        for r in range(w.n_req):
            m = dit.cache_signal(M.W, w, xk[r].astype(np.float64), sched[k, r])
            st = states[r]
            m32 = np.asarray(m, dtype=np.float32)
            d = float("nan") if st.m_prev is None else sampler.rel_l1(m32, st.m_prev)
            has_r = st.residual is not None and st.m_prev is not None
            active = k not in (0, n - 1) and has_r
            acc_before = st.acc
            sk, st.acc = sampler.cache_rule(st.acc, d, k, n, w.cache_tau, sampler.MODE_ACCUMULATE, has_r)
            if not sk:
                st.residual = True
            st.m_prev = m32
            if k > 0:
                assert abs(rel[r] - d) <= 1e-6 * abs(d) + 1e-12, (k, r, rel[r], d)
            if active:
                margins.append(abs(acc_before + d - w.cache_tau))
            assert bool(skip[r]) == sk, (k, r)
        gpu_skips.append(skip)
        npred = torch.zeros_like(x)
        t2i.t2i_dit_step(M.m, x, hw, sched[k], tx, t_next=sched[k + 1], skip=skip, cache_state=state,
                         noise_pred=npred)
        torch.cuda.synchronize()
        vk = M.split(npred.cpu().numpy().astype(np.float64), shapes)
        for r in vel_req:
            ref, _ = sampler.model_velocity(M.W, w, xk[r].astype(np.float64), sched[k, r], texts[r],
                                            1.0, vstates[r], skip=bool(skip[r]))
            err = rel_l2(vk[r], ref)
            assert err < 1e-2, (k, r, bool(skip[r]), err)
            if skip[r]:
                n_vel_skips += 1
                say(f"packed cache step {k} request {r}: skipped-step v rel_l2 {err:.2e}")
    assert n_vel_skips > 0, "no skipped step among the requests compared"
    n_skip = int(np.sum(gpu_skips))
    say(f"packed cache: {n_skip} skipped request-steps of {n * w.n_req}; min margin {min(margins):.3e}")
    # the sampling loop reproduces the step-by-step run bitwise
    x2 = M.latents_dev(lats)
    state2 = M.m.new_cache_state(toks, 1)
    skip_log, _ = t2i.t2i_dit_sample(M.m, x2, hw, tx, n, timesteps=sched, cache_tau=w.cache_tau,
                                     cache_state=state2)
    torch.cuda.synchronize()
    assert np.array_equal(skip_log, np.array(gpu_skips, dtype=np.uint8))
    assert np.array_equal(x2.cpu().numpy(), x.cpu().numpy())


def test_packed_per_step_cache_mode_and_resume(packed8):
    """The per-step reading of the cache rule (skip iff d_k < tau) on the GPU:
    decisions equal the oracle's rule applied to the GPU's latents.  Then a
    sample interrupted after step k -- latents and cache state saved to host
    memory, restored into fresh buffers, resumed with start_step = k on a
    second handle over the same weights -- equals the uninterrupted sample
    bitwise, decisions included."""
    M, w = packed8, packed8.w
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    t0 = synth.start_times(w)
    n, tau, mode = w.steps, w.cache_tau, t2i.T2I_CACHE_PER_STEP
    sched = np.stack([sampler.schedule(n, a) for a in t0], axis=1)
    tx = M.text_dev(texts)
    toks = [w.tokens(r) for r in range(w.n_req)]
    shapes = [l.shape for l in lats]
    # uninterrupted sample in per-step mode
    x_full = M.latents_dev(lats)
    st_full = M.m.new_cache_state(toks, 1)
    log_full, rel_full = t2i.t2i_dit_sample(M.m, x_full, hw, tx, n, timesteps=sched,
                                            cache_tau=tau, cache_mode=mode, cache_state=st_full)
    torch.cuda.synchronize()
    # the same loop step by step, decisions checked against the oracle's rule
    x = M.latents_dev(lats)
    state = M.m.new_cache_state(toks, 1)
    states = [sampler.CacheState() for _ in lats]
    k_stop = n // 2
    for k in range(k_stop):
        xk = M.split(x.cpu().numpy(), shapes)
        rel, skip = t2i.t2i_cache_check(M.m, x, hw, sched[k], k, n, tau, state, mode=mode)
        for r in range(w.n_req):
            m = dit.cache_signal(M.W, w, xk[r].astype(np.float64), sched[k, r])
            st = states[r]
            sk, d = sampler.cache_decide(st, m, k, n, tau, sampler.MODE_PER_STEP)
            if not sk:
                st.residual = True
            if k > 0:
                assert abs(rel[r] - d) <= 1e-6 * abs(d) + 1e-12, (k, r, rel[r], d)
            assert bool(skip[r]) == sk, (k, r)
            assert log_full[k, r] == skip[r], (k, r)
        t2i.t2i_dit_step(M.m, x, hw, sched[k], tx, t_next=sched[k + 1], skip=skip,
                         cache_state=state)
    torch.cuda.synchronize()
    say(f"per-step cache: {int(log_full.sum())} skipped request-steps of {n * w.n_req}")
    assert log_full.sum() > 0
    # checkpoint to host, restore into fresh buffers, resume on a second handle
    ck_x, ck_state = x.cpu().numpy().copy(), state.cpu().numpy().copy()
    del x, state
    m2 = t2i.t2i_dit_init(M.cfg, M.dev)
    x2 = torch.from_numpy(ck_x).to(DEV)
    st2 = torch.from_numpy(ck_state).to(DEV)
    log2, _ = t2i.t2i_dit_sample(m2, x2, hw, tx, n, timesteps=sched, start_step=k_stop,
                                 cache_tau=tau, cache_mode=mode, cache_state=st2)
    torch.cuda.synchronize()
    assert np.array_equal(log2[k_stop:], log_full[k_stop:])
    assert np.array_equal(x2.cpu().numpy(), x_full.cpu().numpy())
    m2.close()
    del m2
    gc.collect()
    torch.cuda.empty_cache()


def test_packed_mixed_skip_runs_blocks_on_computing_requests_only(packed8):
    """A step in which some requests reuse their cached residual and the
    others compute runs the blocks on the computing requests' rows alone.
    Their velocities and updated latents equal, bitwise, those of the same
    step with every request computing; the skipped requests' equal those of
    the step with every request skipping."""
    M, w = packed8, packed8.w
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    n = w.n_req
    ts = list(synth.start_times(w))
    t1 = [0.9 * t for t in ts]
    t2 = [0.85 * t for t in ts]
    tx = M.text_dev(texts)
    toks = [w.tokens(r) for r in range(n)]
    state = M.m.new_cache_state(toks, 1)
    x = M.latents_dev(lats)
    t2i.t2i_dit_step(M.m, x.clone(), hw, ts, tx, skip=[0] * n, cache_state=state)
    shapes = [l.shape for l in lats]

    def run(skip):
        st, xx = state.clone(), x.clone()
        v = torch.zeros_like(xx)
        t2i.t2i_dit_step(M.m, xx, hw, t1, tx, t_next=t2, skip=skip, cache_state=st, noise_pred=v)
        torch.cuda.synchronize()
        return M.split(v.cpu().numpy(), shapes), M.split(xx.cpu().numpy(), shapes)

    for mixed in ([0, 1, 1, 0, 1, 0, 1, 1], [1, 1, 1, 1, 1, 1, 0, 1], [0, 1, 0, 1, 0, 1, 0, 1]):
        v_mix, x_mix = run(mixed)
        v_all, x_all = run([0] * n)
        v_none, x_none = run([1] * n)
        for r in range(n):
            v_ref, x_ref = (v_none, x_none) if mixed[r] else (v_all, x_all)
            assert np.array_equal(v_mix[r], v_ref[r]), (mixed, r)
            assert np.array_equal(x_mix[r], x_ref[r]), (mixed, r)
        say(f"mixed skip {mixed}: computing and skipped requests bitwise as in the uniform steps")
