"""Pins of the oracle against things other than itself (CPU only).

Each test checks an oracle function against a brute-force loop written from
the definition, a library routine computing the same textbook operation
(PyTorch CPU in float64), a closed form, an invariant, or a hand-worked
fixture under ``tests/golden/``.
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as TF

import synth
from oracle import dit, sampler

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

TINY = synth.reduced(synth.workload("tiny_f32"), hidden=8, heads=2, head_dim=4,
                     depth=2, mlp_hidden=16, text_dim=6, text_tokens=3,
                     latent_channels=2, requests=((4, 6),), freq_dim=8)


def tiny_weights(w=TINY, std=None, seed=11):
    lay = dit.weight_layout(w)
    rng = np.random.default_rng(seed)
    ts = []
    for name, shape in lay:
        s = std if std is not None else (0.5 if name.endswith(".b") else 0.4)
        ts.append(rng.standard_normal(shape) * s)
    return dit.as_dict(w, ts)


def T(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


# ---------------------------------------------------------------- patchify

def test_patchify_index_map_brute_force():
    C, h, w, p = 3, 4, 6, 2
    lat = np.arange(C * h * w, dtype=np.float64).reshape(C, h, w)
    tok = dit.patchify(lat, p)
    gw = w // p
    for i in range(h // p):
        for j in range(w // p):
            for a in range(p):
                for b in range(p):
                    for c in range(C):
                        assert tok[i * gw + j, (a * p + b) * C + c] == lat[c, i * p + a, j * p + b]
    assert np.array_equal(dit.unpatchify(tok, p, C, h, w), lat)


# ---------------------------------------------------------------- embeddings

def test_pos_embed_structure():
    gh, gw, D = 3, 5, 16
    pe = dit.pos_embed_2d(gh, gw, D)
    q = D // 4
    # origin: sin halves 0, cos halves 1
    assert np.allclose(pe[0], np.r_[np.zeros(q), np.ones(q), np.zeros(q), np.ones(q)])
    for i in range(gh):
        for j in range(gw):
            row = pe[i * gw + j]
            # the first half depends on the row only, the second on the column only
            assert np.allclose(row[:D // 2], pe[i * gw][:D // 2])
            assert np.allclose(row[D // 2:], pe[j][D // 2:])
            # sin^2 + cos^2 = 1 per frequency, in both halves
            assert np.allclose(row[:q] ** 2 + row[q:2 * q] ** 2, 1)
            assert np.allclose(row[2 * q:3 * q] ** 2 + row[3 * q:] ** 2, 1)
            # lowest index is 1 rad per position, highest 10000^(-(q-1)/q)
            assert math.isclose(row[0], math.sin(i), abs_tol=1e-12)
            assert math.isclose(row[2 * q], math.sin(j), abs_tol=1e-12)
            assert math.isclose(row[q - 1], math.sin(i * 10000.0 ** (-(q - 1) / q)), abs_tol=1e-12)


def test_timestep_frequencies_closed_forms():
    w = synth.workload("dit512")
    e0 = dit.timestep_frequencies(0.0, w)
    assert np.array_equal(e0, np.r_[np.ones(128), np.zeros(128)])
    e = dit.timestep_frequencies(0.37, w)
    assert np.allclose(e[:128] ** 2 + e[128:] ** 2, 1)
    assert math.isclose(e[0], math.cos(370.0), abs_tol=1e-12)
    assert math.isclose(e[128], math.sin(370.0), abs_tol=1e-12)
    assert math.isclose(e[127], math.cos(370.0 * 10000.0 ** (-127 / 128)), abs_tol=1e-12)


def test_conditioning_mlp_brute_force():
    W = tiny_weights()
    c = dit.conditioning(W, TINY, 0.6)
    e = dit.timestep_frequencies(0.6, TINY)
    D = TINY.hidden
    h = []
    for o in range(D):
        s = W["t_embed.b1"][o] + sum(W["t_embed.w1"][o, i] * e[i] for i in range(len(e)))
        h.append(s / (1 + math.exp(-s)))
    for o in range(D):
        s = W["t_embed.b2"][o] + sum(W["t_embed.w2"][o, i] * h[i] for i in range(D))
        assert math.isclose(c[o], s, rel_tol=1e-12, abs_tol=1e-12)


# ---------------------------------------------------------------- pointwise ops

def test_layer_norm_matches_torch():
    x = np.random.default_rng(0).standard_normal((7, 40)) * 3 + 1
    ref = TF.layer_norm(T(x), (40,), eps=1e-6).numpy()
    assert np.allclose(dit.layer_norm(x, 1e-6), ref, rtol=1e-12, atol=1e-12)


def test_layer_norm_zero_modulation_moments():
    x = np.random.default_rng(1).standard_normal((5, 64)) * 0.01
    eps = 1e-6
    h = dit.modulate(dit.layer_norm(x, eps), 0.0, 0.0)
    var = x.var(axis=1)
    assert np.allclose(h.mean(axis=1), 0, atol=1e-12)
    assert np.allclose(h.var(axis=1), var / (var + eps), rtol=1e-10)


def test_gelu_tanh_matches_torch_and_erf_gelu():
    u = np.linspace(-8, 8, 2001)
    g = dit.gelu_tanh(u)
    assert np.allclose(g, TF.gelu(T(u), approximate="tanh").numpy(), rtol=1e-12, atol=1e-14)
    from scipy.special import erf
    exact = 0.5 * u * (1 + erf(u / math.sqrt(2)))
    assert np.max(np.abs(g - exact)) < 1e-3        # known bound of the tanh form
    assert dit.gelu_tanh(np.array(0.0)) == 0.0
    assert np.allclose(g - dit.gelu_tanh(-u), u, atol=1e-12)


def test_silu_matches_torch():
    u = np.linspace(-30, 30, 601)
    assert np.allclose(dit.silu(u), TF.silu(T(u)).numpy(), rtol=1e-12, atol=1e-15)


# ---------------------------------------------------------------- attention

def brute_attention(q, k, v, heads):
    nq, dm = q.shape
    nk = k.shape[0]
    d = dm // heads
    out = np.zeros((nq, dm))
    for h in range(heads):
        for i in range(nq):
            s = [sum(q[i, h * d + c] * k[j, h * d + c] for c in range(d)) / math.sqrt(d)
                 for j in range(nk)]
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            z = sum(e)
            for c in range(d):
                out[i, h * d + c] = sum(e[j] / z * v[j, h * d + c] for j in range(nk))
    return out


def test_attention_brute_force():
    rng = np.random.default_rng(2)
    q, k, v = rng.standard_normal((5, 12)), rng.standard_normal((7, 12)), rng.standard_normal((7, 12))
    assert np.allclose(dit.attention(q, k, v, 3), brute_attention(q, k, v, 3), rtol=1e-12, atol=1e-13)


def test_attention_matches_torch_sdpa_head_layout():
    rng = np.random.default_rng(3)
    H, d, nq, nk = 4, 18, 33, 20
    q, k, v = (rng.standard_normal((n, H * d)) for n in (nq, nk, nk))
    tq = T(q).view(nq, H, d).transpose(0, 1)
    tk = T(k).view(nk, H, d).transpose(0, 1)
    tv = T(v).view(nk, H, d).transpose(0, 1)
    ref = TF.scaled_dot_product_attention(tq, tk, tv).transpose(0, 1).reshape(nq, H * d)
    assert np.allclose(dit.attention(q, k, v, H), ref.numpy(), rtol=1e-12, atol=1e-13)


def test_softmax_rows_sum_to_one():
    s = np.random.default_rng(4).standard_normal((9, 31)) * 20
    p = dit.softmax_rows(s)
    assert np.allclose(p.sum(axis=1), 1, atol=1e-14)
    assert (p >= 0).all()


def test_identical_keys_give_mean_of_values():
    rng = np.random.default_rng(5)
    q = rng.standard_normal((6, 8))
    k = np.tile(rng.standard_normal((1, 8)), (10, 1))
    v = rng.standard_normal((10, 8))
    o = dit.attention(q, k, v, 2)
    assert np.allclose(o, np.tile(v.mean(axis=0), (6, 1)), atol=1e-13)


def test_single_key_returns_value_and_key_permutation_invariance():
    rng = np.random.default_rng(6)
    q, k, v = rng.standard_normal((4, 8)), rng.standard_normal((1, 8)), rng.standard_normal((1, 8))
    assert np.allclose(dit.attention(q, k, v, 2), np.tile(v, (4, 1)), atol=1e-14)
    k, v = rng.standard_normal((9, 8)), rng.standard_normal((9, 8))
    perm = rng.permutation(9)
    assert np.allclose(dit.attention(q, k, v, 2), dit.attention(q, k[perm], v[perm], 2), atol=1e-13)


# ---------------------------------------------------------------- transformer block

def brute_block(W, w, b, x, y, c):
    """The block written with scalar loops from the definitions."""
    D, H, F = w.hidden, w.heads, w.mlp_hidden
    d = D // H
    p = f"blocks.{b}."

    def lin(vec, Wm, bv):
        return [bv[o] + sum(Wm[o][i] * vec[i] for i in range(len(vec))) for o in range(len(bv))]

    def ln(vec):
        mu = sum(vec) / len(vec)
        var = sum((a - mu) ** 2 for a in vec) / len(vec)
        return [(a - mu) / math.sqrt(var + w.ln_eps) for a in vec]

    def attend(qs, ks, vs):
        out = []
        for qi in qs:
            row = [0.0] * D
            for h in range(H):
                s = [sum(qi[h * d + c] * kj[h * d + c] for c in range(d)) / math.sqrt(d) for kj in ks]
                mx = max(s)
                e = [math.exp(a - mx) for a in s]
                z = sum(e)
                for c in range(d):
                    row[h * d + c] = sum(e[j] * vs[j][h * d + c] for j in range(len(ks))) / z
            out.append(row)
        return out

    sc = [a / (1 + math.exp(-a)) for a in c]
    mod = lin(sc, W[p + "ada.w"], W[p + "ada.b"])
    sh1, s1, g1, sh2, s2, g2 = (mod[i * D:(i + 1) * D] for i in range(6))
    xs = [list(r) for r in x]
    hs = [[n * (1 + s1[i]) + sh1[i] for i, n in enumerate(ln(r))] for r in xs]
    qkv = [lin(h, W[p + "attn.qkv.w"], W[p + "attn.qkv.b"]) for h in hs]
    o = attend([r[:D] for r in qkv], [r[D:2 * D] for r in qkv], [r[2 * D:] for r in qkv])
    for t in range(len(xs)):
        po = lin(o[t], W[p + "attn.o.w"], W[p + "attn.o.b"])
        xs[t] = [xs[t][i] + g1[i] * po[i] for i in range(D)]
    qs = [lin(r, W[p + "xattn.q.w"], W[p + "xattn.q.b"]) for r in xs]
    kv = [lin(r, W[p + "xattn.kv.w"], W[p + "xattn.kv.b"]) for r in y]
    o = attend(qs, [r[:D] for r in kv], [r[D:] for r in kv])
    for t in range(len(xs)):
        po = lin(o[t], W[p + "xattn.o.w"], W[p + "xattn.o.b"])
        xs[t] = [xs[t][i] + po[i] for i in range(D)]
    for t in range(len(xs)):
        h = [n * (1 + s2[i]) + sh2[i] for i, n in enumerate(ln(xs[t]))]
        u = lin(h, W[p + "mlp.fc1.w"], W[p + "mlp.fc1.b"])
        u = [0.5 * a * (1 + math.tanh(math.sqrt(2 / math.pi) * (a + 0.044715 * a ** 3))) for a in u]
        f = lin(u, W[p + "mlp.fc2.w"], W[p + "mlp.fc2.b"])
        xs[t] = [xs[t][i] + g2[i] * f[i] for i in range(D)]
    return np.array(xs)


def test_block_brute_force():
    W = tiny_weights()
    rng = np.random.default_rng(7)
    x = rng.standard_normal((5, TINY.hidden))
    y = rng.standard_normal((3, TINY.hidden))
    c = rng.standard_normal(TINY.hidden)
    for b in range(TINY.depth):
        got = dit.block(W, TINY, b, x, y, dit.block_modulation(W, TINY, c, b))
        assert np.allclose(got, brute_block(W, TINY, b, x, y, c), rtol=1e-11, atol=1e-12)


def test_block_rows_equals_block_subset():
    W = tiny_weights()
    rng = np.random.default_rng(18)
    x = rng.standard_normal((9, TINY.hidden))
    y = rng.standard_normal((3, TINY.hidden))
    mod = dit.block_modulation(W, TINY, rng.standard_normal(TINY.hidden), 1)
    full = dit.block(W, TINY, 1, x, y, mod)
    rows = np.array([7, 0, 4])
    assert np.allclose(dit.block_rows(W, TINY, 1, x, y, mod, rows), full[rows], rtol=1e-13, atol=1e-14)


def test_zero_gates_make_block_identity():
    """adaLN-Zero with zero gates is an identity block.

    The cross-attention path is ungated in this architecture, so its output
    projection is zeroed as well (adapted form of the identity pin)."""
    W = tiny_weights()
    D = TINY.hidden
    for b in range(TINY.depth):
        p = f"blocks.{b}."
        for chunk in (2, 5):                       # gate_msa, gate_mlp
            W[p + "ada.w"][chunk * D:(chunk + 1) * D] = 0
            W[p + "ada.b"][chunk * D:(chunk + 1) * D] = 0
        W[p + "xattn.o.w"][:] = 0
        W[p + "xattn.o.b"][:] = 0
    rng = np.random.default_rng(8)
    x = rng.standard_normal((6, D))
    y = rng.standard_normal((3, D))
    c = rng.standard_normal(D)
    assert np.array_equal(dit.run_blocks(W, TINY, x, y, c), x)


def test_control_residuals_through_identity_blocks():
    """Callback input: with identity blocks (zero gates, zero ungated
    cross-attention output) the stream after the blocks is x0 plus the sum of
    the injected residuals; injection after the last block that runs shows in
    the output, injection past it does not."""
    W = tiny_weights()
    D = TINY.hidden
    for b in range(TINY.depth):
        p = f"blocks.{b}."
        for chunk in (2, 5):
            W[p + "ada.w"][chunk * D:(chunk + 1) * D] = 0
            W[p + "ada.b"][chunk * D:(chunk + 1) * D] = 0
        W[p + "xattn.o.w"][:] = 0
        W[p + "xattn.o.b"][:] = 0
    rng = np.random.default_rng(19)
    x = rng.standard_normal((6, D))
    y = rng.standard_normal((3, D))
    c = rng.standard_normal(D)
    r0, r1 = rng.standard_normal((6, D)), rng.standard_normal((6, D))
    out = dit.run_blocks(W, TINY, x, y, c, control={0: r0, TINY.depth - 1: r1})
    assert np.allclose(out, x + r0 + r1, rtol=0, atol=1e-14)
    out = dit.run_blocks(W, TINY, x, y, c, 0, 1, control={0: r0, 1: r1})
    assert np.allclose(out, x + r0, rtol=0, atol=1e-14)
    # a zero residual changes nothing in a real (non-identity) model
    W2 = tiny_weights()
    assert np.array_equal(dit.run_blocks(W2, TINY, x, y, c, control={1: np.zeros((6, D))}),
                          dit.run_blocks(W2, TINY, x, y, c))


def test_unconditional_cross_attention_closed_form():
    """All-zero text makes every key equal, so each query gets the value row."""
    W = tiny_weights()
    D = TINY.hidden
    y = dit.text_project(W, TINY, np.zeros((TINY.text_tokens, TINY.text_dim)))
    assert np.array_equal(y, np.tile(W["y_embed.b"], (TINY.text_tokens, 1)))
    p = "blocks.0."
    kv = dit.linear(y, W[p + "xattn.kv.w"], W[p + "xattn.kv.b"])
    rng = np.random.default_rng(9)
    q = rng.standard_normal((5, D)) * 3
    o = dit.attention(q, kv[:, :D], kv[:, D:], TINY.heads)
    v_row = W["y_embed.b"] @ W[p + "xattn.kv.w"][D:].T + W[p + "xattn.kv.b"][D:]
    assert np.allclose(o, np.tile(v_row, (5, 1)), atol=1e-13)


def test_forward_matches_brute_force_composition():
    """Embed -> blocks -> final layer composed from independent pieces."""
    W = tiny_weights()
    rng = np.random.default_rng(10)
    lat = rng.standard_normal((TINY.latent_channels, 4, 6))
    text = rng.standard_normal((TINY.text_tokens, TINY.text_dim))
    t = 0.73
    v, hid = dit.forward(W, TINY, lat, t, text, return_hidden=True)
    # embedding by loops
    p, C, D = TINY.patch, TINY.latent_channels, TINY.hidden
    gh, gw = 2, 3
    x = np.zeros((gh * gw, D))
    q = D // 4
    for i in range(gh):
        for j in range(gw):
            for o in range(D):
                s = W["x_embed.b"][o]
                for a in range(p):
                    for bb in range(p):
                        for c in range(C):
                            s += W["x_embed.w"][o, (a * p + bb) * C + c] * lat[c, i * p + a, j * p + bb]
                half, k = divmod(o, D // 2)
                pos = i if half == 0 else j
                f = 10000.0 ** (-(k % q) / q)
                s += math.sin(pos * f) if k < q else math.cos(pos * f)
                x[i * gw + j, o] = s
    c = dit.conditioning(W, TINY, t)
    y = [[W["y_embed.b"][o] + sum(W["y_embed.w"][o, i] * text[r, i] for i in range(TINY.text_dim))
          for o in range(D)] for r in range(TINY.text_tokens)]
    for b in range(TINY.depth):
        x = brute_block(W, TINY, b, x, y, c)
    assert np.allclose(hid, x, rtol=1e-10, atol=1e-11)
    # final layer by loops
    sc = [a / (1 + math.exp(-a)) for a in c]
    fm = [W["final.ada.b"][o] + sum(W["final.ada.w"][o, i] * sc[i] for i in range(D)) for o in range(2 * D)]
    out = np.zeros((C, 4, 6))
    for i in range(gh):
        for j in range(gw):
            r = x[i * gw + j]
            mu = r.mean()
            sd = math.sqrt(((r - mu) ** 2).mean() + TINY.ln_eps)
            hmod = [(r[k] - mu) / sd * (1 + fm[D + k]) + fm[k] for k in range(D)]
            for a in range(p):
                for bb in range(p):
                    for cc in range(C):
                        f = (a * p + bb) * C + cc
                        out[cc, i * p + a, j * p + bb] = W["final.out.b"][f] + sum(
                            W["final.out.w"][f, k] * hmod[k] for k in range(D))
    assert np.allclose(v, out, rtol=1e-10, atol=1e-11)


# ---------------------------------------------------------------- sampler

def test_zero_velocity_euler_leaves_latent():
    x = np.random.default_rng(12).standard_normal((4, 8, 8))
    for t, tn in zip(sampler.schedule(7)[:-1], sampler.schedule(7)[1:]):
        assert np.array_equal(sampler.euler_update(x, np.zeros_like(x), t, tn), x)


def test_constant_velocity_integrates_to_minus_v():
    x0 = np.random.default_rng(13).standard_normal(50)
    v = np.random.default_rng(14).standard_normal(50)
    x = x0.copy()
    s = sampler.schedule(20)
    assert s[0] == 1.0 and s[-1] == 0.0
    for k in range(20):
        x = sampler.euler_update(x, v, s[k], s[k + 1])
    assert np.allclose(x, x0 - v, atol=1e-13)
    s = sampler.schedule(20, 0.25)
    assert math.isclose(s[0], 0.25) and s[-1] == 0.0


def test_cfg_special_cases():
    rng = np.random.default_rng(15)
    vc, vu = rng.standard_normal(9), rng.standard_normal(9)
    assert np.allclose(sampler.cfg_combine(vc, vu, 1.0), vc, rtol=0, atol=1e-15)
    assert np.array_equal(sampler.cfg_combine(vc, vu, 0.0), vu)
    assert np.allclose(sampler.cfg_combine(vc, vu, 4.5), 4.5 * vc - 3.5 * vu, atol=1e-14)


def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line)
    return rows


def test_rel_l1_golden():
    for row in _read_golden("cache_rel_l1.txt"):
        a, b, d = (s.strip() for s in row.split("|"))
        m_prev = np.array([float(v) for v in a.split()])
        m = np.array([float(v) for v in b.split()])
        assert math.isclose(sampler.rel_l1(m, m_prev), float(d), abs_tol=1e-15)
        assert sampler.rel_l1(m_prev, m_prev) == 0.0


def test_cache_rule_golden_sequence():
    rows = [r.split() for r in _read_golden("cache_decisions.txt")]
    n = len(rows)
    for mode, col in ((sampler.MODE_ACCUMULATE, 2), (sampler.MODE_PER_STEP, 4)):
        acc = 0.0
        for k, r in enumerate(rows):
            d = float(r[1])
            skip, acc = sampler.cache_rule(acc, d, k, n, 0.1, mode, has_residual=k > 0)
            assert ("S" if skip else "C") == r[col], (mode, k)
            if mode == sampler.MODE_ACCUMULATE:
                assert math.isclose(acc, float(r[3]), abs_tol=1e-15)
    # disabled rule never skips
    for k in range(n):
        assert sampler.cache_rule(0.0, 0.0, k, n, 0.0, sampler.MODE_ACCUMULATE, True) == (False, 0.0)


def _tiny_problem(guidance=1.0):
    w = synth.reduced(TINY, guidance=guidance, steps=5)
    W = tiny_weights(w, std=0.3)
    rng = np.random.default_rng(16)
    lats = [rng.standard_normal((w.latent_channels, 4, 6))]
    texts = [rng.standard_normal((w.text_tokens, w.text_dim))]
    return w, W, lats, texts


def test_disabled_cache_equals_plain_loop():
    w, W, lats, texts = _tiny_problem(guidance=3.0)
    out_a, log_a = sampler.sample(W, w, lats, texts, [1.0], 5, 3.0, tau=0.0)
    x = np.asarray(lats[0], dtype=np.float64)
    s = sampler.schedule(5)
    for k in range(5):
        vc = dit.forward(W, w, x, s[k], texts[0])
        vu = dit.forward(W, w, x, s[k], None)
        x = x + (s[k + 1] - s[k]) * (vu + 3.0 * (vc - vu))
    assert np.array_equal(out_a[0], x)
    assert not any(any(r) for r in log_a["skip"])


def test_infinite_tau_reuses_first_residual():
    """tau = inf skips every middle step, each using step 0's residual."""
    w, W, lats, texts = _tiny_problem(guidance=2.0)
    n = 5
    out, log = sampler.sample(W, w, lats, texts, [1.0], n, 2.0, tau=np.inf)
    assert [r[0] for r in log["skip"]] == [False, True, True, True, False]
    s = sampler.schedule(n)
    x = np.asarray(lats[0], dtype=np.float64)
    c0 = dit.conditioning(W, w, s[0])
    x00 = dit.embed(W, w, x)
    R = [dit.run_blocks(W, w, x00, dit.text_project(W, w, t), c0) - x00
         for t in (texts[0], np.zeros((w.text_tokens, w.text_dim)))]
    for k in range(n):
        c = dit.conditioning(W, w, s[k])
        x0 = dit.embed(W, w, x)
        if k in (0, n - 1):
            vc = dit.forward(W, w, x, s[k], texts[0])
            vu = dit.forward(W, w, x, s[k], None)
        else:
            vc = dit.final_layer(W, w, x0 + R[0], c, 4, 6)
            vu = dit.final_layer(W, w, x0 + R[1], c, 4, 6)
        x = x + (s[k + 1] - s[k]) * (vu + 2.0 * (vc - vu))
    assert np.allclose(out[0], x, rtol=1e-12, atol=1e-12)


def test_cache_signal_is_block0_modulated_input():
    w, W, lats, _ = _tiny_problem()
    m = dit.cache_signal(W, w, lats[0], 0.4)
    c = dit.conditioning(W, w, 0.4)
    mod = dit.block_modulation(W, w, c, 0)
    ref = TF.layer_norm(T(dit.embed(W, w, lats[0])), (w.hidden,), eps=w.ln_eps).numpy()
    assert np.allclose(m, ref * (1 + mod["scale_msa"]) + mod["shift_msa"], atol=1e-12)


def test_oracle_is_deterministic():
    w, W, lats, texts = _tiny_problem(guidance=4.5)
    a, la = sampler.sample(W, w, lats, texts, [1.0], 5, 4.5, tau=0.3)
    b, lb = sampler.sample(W, w, lats, texts, [1.0], 5, 4.5, tau=0.3)
    assert np.array_equal(a[0], b[0]) and la["skip"] == lb["skip"]


# ---------------------------------------------------------------- inputs

def test_inputs_regenerate_bitwise_and_have_recipe_moments():
    w = synth.workload("dit512")
    lay = dit.weight_layout(w)
    a = synth.weights(w, lay, only=4)
    b = synth.weights(w, lay, only=4)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    big = a[0]                                      # x_embed.w, bf16-rounded
    assert np.array_equal(big, synth.round_bf16(big))
    assert abs(big.std() - 0.02) < 5 * 0.02 / math.sqrt(big.size) + 1e-3
    lat = synth.latents(w)[0]
    assert lat.dtype == np.float32 and lat.shape == (4, 64, 64)
    assert abs(lat.mean()) < 5 / math.sqrt(lat.size)


def test_bf16_rounding_is_nearest_even():
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -9], dtype=np.float32)
    got = synth.round_bf16(vals)
    ref = torch.from_numpy(vals).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(got, ref)


# ---------------------------------------------------------------- pin power

def _block_error(W, x, y, c):
    got = dit.block(W, TINY, 0, x, y, dit.block_modulation(W, TINY, c, 0))
    return float(np.max(np.abs(got - brute_block(W, TINY, 0, x, y, c))))


@pytest.mark.parametrize("mutation", ["modulate_drops_one", "gelu_drops_cubic",
                                      "attention_scale_d", "linear_transposed",
                                      "layer_norm_no_eps", "silu_sign"])
def test_pins_catch_planted_oracle_mistakes(monkeypatch, mutation):
    """Plant a plausible mistake in the oracle; the brute-force pin must see it."""
    W = tiny_weights()
    rng = np.random.default_rng(17)
    x = rng.standard_normal((5, TINY.hidden)) * 0.05
    y = rng.standard_normal((3, TINY.hidden))
    c = rng.standard_normal(TINY.hidden)
    assert _block_error(W, x, y, c) < 1e-11
    orig_attn, orig_ln = dit.attention, dit.layer_norm
    if mutation == "modulate_drops_one":
        monkeypatch.setattr(dit, "modulate", lambda xn, sh, sc: xn * sc + sh)
    elif mutation == "gelu_drops_cubic":
        monkeypatch.setattr(dit, "gelu_tanh", lambda u: 0.5 * u * (1 + np.tanh(math.sqrt(2 / math.pi) * u)))
    elif mutation == "attention_scale_d":
        monkeypatch.setattr(dit, "attention", lambda q, k, v, h: orig_attn(q / math.sqrt(q.shape[1] // h), k, v, h))
    elif mutation == "linear_transposed":
        sq = lambda wt: wt.T if wt.shape[0] == wt.shape[1] else wt
        monkeypatch.setattr(dit, "linear", lambda a, wt, b: a @ sq(wt).T + b)
    elif mutation == "layer_norm_no_eps":
        monkeypatch.setattr(dit, "layer_norm", lambda a, eps: orig_ln(a, 0.0))
    elif mutation == "silu_sign":
        monkeypatch.setattr(dit, "silu", lambda a: a / (1 + np.exp(a)))
    assert _block_error(W, x, y, c) > 1e-9
