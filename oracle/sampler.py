"""Guidance, Euler sampler, cache-skip rule and the sampling loop (float64).

Test infrastructure only.  The paper's workflow (Sec. 4, Fig. "workflow
definition") draws a Gaussian latent, then for every denoising step calls the
base model on ``(latents, prompt_embeds)`` and feeds ``noise_pred`` to a
``denoise`` update.  Readings for what the paper leaves open:

* classifier-free guidance: ``v = v_u + g (v_c - v_u)``, the unconditional
  branch sees all-zero text embeddings, the same latent and the same ``t``;
* schedule: ``t_k = t0 (1 - k/N)``, ``k = 0 ... N`` (``t0 = 1`` unless a
  request starts at its own time); the model output is the velocity dx/dt and
  ``x_{k+1} = x_k + (t_{k+1} - t_k) v_k``;
* step-skip cache (named in the paper's preamble, described nowhere in its
  text; readings follow the published TeaCache rule without its polynomial
  rescaling): per request, ``m_k`` is block 0's modulated input, rounded to
  float32, ``d_k = sum|m_k - m_{k-1}| / sum|m_{k-1}|`` in float64.
  In accumulate mode ``A += d_k`` and the step skips iff it is neither the
  first nor the last step, ``A < tau`` and a residual exists; a computed step
  stores ``R = x_L - x_0`` per guidance branch and resets ``A = 0``; a skipped
  step uses ``x_L = x_0 + R``.  In per-step mode the test is ``d_k < tau``.
  ``m_{k-1}`` is replaced every step.  ``tau <= 0`` disables the rule.  The
  final layer always runs at the current ``t``.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np

from . import dit, mmdit

F64 = np.float64

MODE_ACCUMULATE = 0
MODE_PER_STEP = 1


def cfg_combine(v_c, v_u, g):
    return v_u + g * (v_c - v_u)


def euler_update(x, v, t, t_next):
    return x + (t_next - t) * v


def schedule(n_steps, t0=1.0):
    """``t_k = t0 (1 - k/N)`` for ``k = 0 ... N``."""
    k = np.arange(n_steps + 1, dtype=F64)
    return float(t0) * (1.0 - k / n_steps)


def rel_l1(m, m_prev):
    """``sum|m - m_prev| / sum|m_prev|`` accumulated in float64."""
    m = np.asarray(m, dtype=F64)
    m_prev = np.asarray(m_prev, dtype=F64)
    return float(np.abs(m - m_prev).sum() / np.abs(m_prev).sum())


@dataclasses.dataclass
class CacheState:
    """Per-request cache state between steps."""
    m_prev: Optional[np.ndarray] = None
    residual: Optional[List[np.ndarray]] = None   # one per guidance branch
    acc: float = 0.0


def cache_rule(acc, d, k, n_steps, tau, mode, has_residual):
    """The skip decision of step ``k`` given its relative-L1 change ``d``.

    Returns ``(skip, acc')``.  The rule is active only when ``tau > 0``, the
    step is neither the first nor the last, and a residual exists; a computed
    step resets the accumulator."""
    skip = False
    if tau > 0 and k not in (0, n_steps - 1) and has_residual:
        if mode == MODE_ACCUMULATE:
            acc = acc + d
            skip = acc < tau
        else:
            acc = d
            skip = d < tau
    if not skip:
        acc = 0.0
    return skip, acc


def cache_decide(state: CacheState, m, k, n_steps, tau, mode=MODE_ACCUMULATE):
    """Decide whether step ``k`` skips the blocks; updates ``acc`` and ``m_prev``.

    ``m`` is rounded to float32 first.  Returns ``(skip, d_k)``; ``d_k`` is NaN
    on the first step (no predecessor)."""
    m = np.asarray(m, dtype=np.float32)
    d = float("nan") if state.m_prev is None else rel_l1(m, state.m_prev)
    has_r = state.residual is not None and state.m_prev is not None
    skip, state.acc = cache_rule(state.acc, d, k, n_steps, tau, mode, has_r)
    state.m_prev = m
    return skip, d


def model_velocity(W, w, lat, t, text, guidance, state: CacheState = None,
                   skip=False, n_blocks=None):
    """Guided velocity of one request; uses or refreshes the cached residual.

    Returns ``(v, v_branches)`` where ``v_branches`` lists the conditional and,
    under guidance, the unconditional velocity."""
    C, h, ww = lat.shape
    mm = getattr(w, "arch", "cross") == "mmdit"
    c = dit.conditioning(W, w, t)
    x0 = mmdit.embed_image(W, w, lat) if mm else dit.embed(W, w, lat)
    nb = w.depth if n_blocks is None else n_blocks
    branches = [text] if guidance == 1.0 else [text, None]
    vs, resid = [], []
    for bi, txt in enumerate(branches):
        if txt is None:
            txt = np.zeros((w.text_tokens, w.text_dim))
        if skip:
            xl = x0 + state.residual[bi]
        else:
            if mm:   # joint blocks; the residual is the image stream's
                _, xl = mmdit.run_blocks(W, w, mmdit.embed_text(W, w, txt), x0, c, (h, ww), 0, nb)
            else:
                y = dit.text_project(W, w, txt)
                xl = dit.run_blocks(W, w, x0, y, c, 0, nb)
            resid.append(xl - x0)
        vs.append(dit.final_layer(W, w, xl, c, h, ww))
    if state is not None and not skip:
        state.residual = resid
    v = vs[0] if guidance == 1.0 else cfg_combine(vs[0], vs[1], guidance)
    return v, vs


def step(W, w, lats, texts, ts, t_nexts, guidance=1.0, states=None, k=0,
         n_steps=1, tau=0.0, mode=MODE_ACCUMULATE):
    """One denoising step for every request (requests are independent).

    Returns ``(new_lats, vs, branch_vs, skips, ds)``."""
    new, vs, bvs, skips, ds = [], [], [], [], []
    for r, lat in enumerate(lats):
        lat = np.asarray(lat, dtype=F64)
        st = None if states is None else states[r]
        skip, d = False, float("nan")
        if st is not None:
            sig = mmdit.cache_signal if getattr(w, "arch", "cross") == "mmdit" else dit.cache_signal
            m = sig(W, w, lat, ts[r])
            skip, d = cache_decide(st, m, k, n_steps, tau, mode)
        v, vb = model_velocity(W, w, lat, ts[r], texts[r], guidance, st, skip)
        new.append(euler_update(lat, v, ts[r], t_nexts[r]))
        vs.append(v)
        bvs.append(vb)
        skips.append(skip)
        ds.append(d)
    return new, vs, bvs, skips, ds


def sample(W, w, lats, texts, t_starts, n_steps, guidance=1.0, tau=0.0,
           mode=MODE_ACCUMULATE, keep=False):
    """The denoising loop of every request from its start time down to 0.

    Returns ``(final_lats, log)`` where ``log`` holds per-step skip decisions
    and relative-L1 values (and the latents/velocities when ``keep``)."""
    scheds = [schedule(n_steps, t0) for t0 in t_starts]
    states = [CacheState() for _ in lats]
    lats = [np.asarray(l, dtype=F64) for l in lats]
    log = {"skip": [], "d": [], "acc": [], "x": [], "v": []}
    for k in range(n_steps):
        ts = [s[k] for s in scheds]
        tn = [s[k + 1] for s in scheds]
        if keep:
            log["x"].append([l.copy() for l in lats])
        new, vs, _, skips, ds = step(W, w, lats, texts, ts, tn, guidance,
                                     states, k, n_steps, tau, mode)
        log["skip"].append(skips)
        log["d"].append(ds)
        log["acc"].append([s.acc for s in states])
        if keep:
            log["v"].append(vs)
        lats = new
    return lats, log
