"""Pins of the joint-attention (MMDiT-style) oracle, CPU only."""
import math

import numpy as np
import pytest

import synth
from oracle import dit, mmdit
from test_oracle_pins import brute_attention

TINY = synth.reduced(synth.workload("mmdit1024"), hidden=16, heads=2, head_dim=8,
                     depth=2, mlp_hidden=32, text_dim=6, text_tokens=3,
                     latent_channels=2, requests=((4, 6),), freq_dim=8)


def weights(w=TINY, seed=21, std=0.3):
    rng = np.random.default_rng(seed)
    return mmdit.as_dict(w, [rng.standard_normal(s) * std for _, s in mmdit.weight_layout(w)])


def brute_rope(x, rows, cols, heads):
    n, dm = x.shape
    d = dm // heads
    out = np.zeros_like(x)
    for t in range(n):
        for h in range(heads):
            for half in range(2):
                pos = rows[t] if half == 0 else cols[t]
                for j in range(d // 4):
                    a = h * d + half * (d // 2) + 2 * j
                    ang = pos * 10000.0 ** (-j / (d // 4))
                    out[t, a] = x[t, a] * math.cos(ang) - x[t, a + 1] * math.sin(ang)
                    out[t, a + 1] = x[t, a] * math.sin(ang) + x[t, a + 1] * math.cos(ang)
    return out


def test_rope_brute_force_identity_and_norm():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((12, 16))
    rows, cols = mmdit.grid_positions(3, 4)
    r = mmdit.rope_2d(x, rows, cols, 2)
    assert np.allclose(r, brute_rope(x, rows, cols, 2), atol=1e-13)
    assert np.allclose(r[0], x[0])                       # position (0, 0)
    assert np.allclose(np.linalg.norm(r, axis=1), np.linalg.norm(x, axis=1))
    # per-head, per-pair norms are preserved too
    assert np.allclose(r[:, 0::2] ** 2 + r[:, 1::2] ** 2, x[:, 0::2] ** 2 + x[:, 1::2] ** 2)


def test_rope_scores_depend_on_relative_position_only():
    rng = np.random.default_rng(1)
    q, k = rng.standard_normal((1, 16)), rng.standard_normal((1, 16))

    def score(p, pp):
        a = mmdit.rope_2d(q, [p[0]], [p[1]], 2)
        b = mmdit.rope_2d(k, [pp[0]], [pp[1]], 2)
        return float((a * b).sum())

    base = score((1, 2), (4, 7))
    assert math.isclose(base, score((3, 5), (6, 10)), rel_tol=1e-11)
    assert math.isclose(base, score((0, 0), (3, 5)), rel_tol=1e-11)
    assert not math.isclose(base, score((0, 0), (3, 6)), rel_tol=1e-6)


def test_zero_gates_identity_both_streams():
    W = weights()
    D = TINY.hidden
    for b in range(TINY.depth):
        for s in mmdit.STREAMS:
            for chunk in (2, 5):
                W[f"blocks.{b}.{s}.ada.w"][chunk * D:(chunk + 1) * D] = 0
                W[f"blocks.{b}.{s}.ada.b"][chunk * D:(chunk + 1) * D] = 0
    rng = np.random.default_rng(2)
    xt, xi = rng.standard_normal((3, D)), rng.standard_normal((6, D))
    c = rng.standard_normal(D)
    rows, cols = mmdit.grid_positions(2, 3)
    for b in range(TINY.depth):
        nt, ni = mmdit.joint_block(W, TINY, b, xt, xi, c, rows, cols)
        assert np.array_equal(nt, xt) and np.array_equal(ni, xi)


def test_joint_attention_brute_force_and_empty_text():
    """Joint block attention equals brute-force attention over [text; image]."""
    W = weights()
    D, H = TINY.hidden, TINY.heads
    rng = np.random.default_rng(3)
    xt, xi = rng.standard_normal((3, D)), rng.standard_normal((6, D))
    c = rng.standard_normal(D)
    rows, cols = mmdit.grid_positions(2, 3)
    nt, ni = mmdit.joint_block(W, TINY, 0, xt, xi, c, rows, cols)
    # rebuild the image-stream output by brute force
    qs, ks, vs = [], [], []
    for s, x in (("txt", xt), ("img", xi)):
        md = mmdit.stream_modulation(W, TINY, c, 0, s)
        h = dit.modulate(dit.layer_norm(x, TINY.ln_eps), md["shift_msa"], md["scale_msa"])
        qkv = h @ W[f"blocks.0.{s}.qkv.w"].T + W[f"blocks.0.{s}.qkv.b"]
        q, k, v = qkv[:, :D], qkv[:, D:2 * D], qkv[:, 2 * D:]
        if s == "img":
            q, k = brute_rope(q, rows, cols, H), brute_rope(k, rows, cols, H)
        qs.append(q), ks.append(k), vs.append(v)
    o = brute_attention(np.vstack(qs), np.vstack(ks), np.vstack(vs), H)
    md = mmdit.stream_modulation(W, TINY, c, 0, "img")
    x = xi + md["gate_msa"] * (o[3:] @ W["blocks.0.img.o.w"].T + W["blocks.0.img.o.b"])
    h = dit.modulate(dit.layer_norm(x, TINY.ln_eps), md["shift_mlp"], md["scale_mlp"])
    u = dit.gelu_tanh(h @ W["blocks.0.img.fc1.w"].T + W["blocks.0.img.fc1.b"])
    x = x + md["gate_mlp"] * (u @ W["blocks.0.img.fc2.w"].T + W["blocks.0.img.fc2.b"])
    assert np.allclose(ni, x, atol=1e-12)
    # no text tokens: the image stream is plain self-attention with RoPE
    nt0, ni0 = mmdit.joint_block(W, TINY, 0, np.zeros((0, D)), xi, c, rows, cols)
    assert nt0.shape == (0, D)
    o = brute_attention(qs[1], ks[1], vs[1], H)
    x = xi + md["gate_msa"] * (o @ W["blocks.0.img.o.w"].T + W["blocks.0.img.o.b"])
    h = dit.modulate(dit.layer_norm(x, TINY.ln_eps), md["shift_mlp"], md["scale_mlp"])
    u = dit.gelu_tanh(h @ W["blocks.0.img.fc1.w"].T + W["blocks.0.img.fc1.b"])
    x = x + md["gate_mlp"] * (u @ W["blocks.0.img.fc2.w"].T + W["blocks.0.img.fc2.b"])
    assert np.allclose(ni0, x, atol=1e-12)


def test_forward_runs_and_embeds():
    W = weights()
    rng = np.random.default_rng(4)
    lat = rng.standard_normal((2, 4, 6))
    text = rng.standard_normal((3, 6))
    v, xt, xi = mmdit.forward(W, TINY, lat, 1.0, text)
    assert v.shape == lat.shape and xt.shape == (3, 16) and xi.shape == (6, 16)
    _, xt0, xi0 = mmdit.forward(W, TINY, lat, 1.0, text, n_blocks=0)
    assert np.allclose(xi0, dit.patchify(lat, 2) @ W["x_embed.w"].T + W["x_embed.b"])
    assert np.allclose(xt0, text @ W["y_embed.w"].T + W["y_embed.b"])


def test_layout_sizes():
    w = synth.workload("mmdit1024")
    n = sum(int(np.prod(s)) for _, s in mmdit.weight_layout(w))
    D, F = 3072, 12288
    per_block = 2 * (6 * D * D + 6 * D + 3 * D * D + 3 * D + D * D + D + F * D + F + D * F + D)
    assert n == per_block * 19 + (D * 64 + D) + (D * 256 + D + D * D + D) + (D * 4096 + D) \
        + (2 * D * D + 2 * D) + (64 * D + 64)


def _stream_inputs(seed=5):
    rng = np.random.default_rng(seed)
    D = TINY.hidden
    return rng.standard_normal((3, D)), rng.standard_normal((6, D)), rng.standard_normal(D)


def test_joint_block_rows_matches_full_block():
    W = weights()
    xt, xi, c = _stream_inputs()
    rows, cols = mmdit.grid_positions(2, 3)
    nt, ni = mmdit.joint_block(W, TINY, 1, xt, xi, c, rows, cols)
    at, ai = mmdit.joint_block_rows(W, TINY, 1, xt, xi, c, rows, cols, range(3), range(6))
    assert np.allclose(at, nt, atol=1e-12) and np.allclose(ai, ni, atol=1e-12)
    st, si = [2, 0], [5, 1, 3]
    bt, bi = mmdit.joint_block_rows(W, TINY, 1, xt, xi, c, rows, cols, st, si)
    assert np.allclose(bt, nt[st], atol=1e-12) and np.allclose(bi, ni[si], atol=1e-12)


def test_cache_signal_is_image_block0_modulated_input():
    import torch
    import torch.nn.functional as TF
    W = weights()
    lat = np.random.default_rng(6).standard_normal((2, 4, 6))
    m = mmdit.cache_signal(W, TINY, lat, 0.3)
    c = dit.conditioning(W, TINY, 0.3)
    a = dit.silu(c) @ W["blocks.0.img.ada.w"].T + W["blocks.0.img.ada.b"]
    D = TINY.hidden
    x = torch.from_numpy(dit.patchify(lat, 2) @ W["x_embed.w"].T + W["x_embed.b"])
    ln = TF.layer_norm(x, (D,), eps=TINY.ln_eps).numpy()
    assert np.allclose(m, ln * (1 + a[D:2 * D]) + a[:D], atol=1e-12)


def test_sampler_runs_mmdit_velocity_guidance_and_cached_residual():
    from oracle import sampler
    W = weights()
    rng = np.random.default_rng(7)
    lat = rng.standard_normal((2, 4, 6))
    text = rng.standard_normal((3, 6))
    vc = mmdit.forward(W, TINY, lat, 0.8, text)[0]
    vu = mmdit.forward(W, TINY, lat, 0.8, None)[0]
    v1, _ = sampler.model_velocity(W, TINY, lat, 0.8, text, 1.0)
    assert np.allclose(v1, vc, atol=1e-12)
    st = sampler.CacheState()
    v2, vb = sampler.model_velocity(W, TINY, lat, 0.8, text, 3.0, st)
    assert np.allclose(vb[0], vc, atol=1e-12) and np.allclose(vb[1], vu, atol=1e-12)
    assert np.allclose(v2, vu + 3.0 * (vc - vu), atol=1e-12)
    # a skipped step reuses the image-stream residual: same velocity here
    v3, _ = sampler.model_velocity(W, TINY, lat, 0.8, text, 3.0, st, skip=True)
    assert np.allclose(v3, v2, atol=1e-10)
    # the unconditional text stream starts from the bias alone
    assert np.allclose(mmdit.embed_text(W, TINY, None), np.tile(W["y_embed.b"], (3, 1)))


# ---------------------------------------------------------------- both streams by scalar loops

def brute_joint_block(W, w, b, x_txt, x_img, c, rows, cols):
    """One joint block written with scalar loops from its definition, returning
    BOTH streams: per-stream adaLN-Zero, LN-modulate, q|k|v projection, RoPE on
    the image queries and keys only, one softmax attention over the text rows
    followed by the image rows, then per stream the gated output projection and
    the gated tanh-GELU MLP with that stream's own weights and gates."""
    D, H, F = w.hidden, w.heads, w.mlp_hidden
    d = D // H

    def lin(vec, Wm, bv):
        return [bv[o] + sum(Wm[o][i] * vec[i] for i in range(len(vec))) for o in range(len(bv))]

    def ln(vec):
        mu = sum(vec) / len(vec)
        var = sum((a - mu) ** 2 for a in vec) / len(vec)
        return [(a - mu) / math.sqrt(var + w.ln_eps) for a in vec]

    def rot(vec, r, cc):
        out = list(vec)
        for h in range(H):
            for half, pos in ((0, r), (1, cc)):
                for j in range(d // 4):
                    a = h * d + half * (d // 2) + 2 * j
                    ang = pos * 10000.0 ** (-j / (d // 4))
                    out[a] = vec[a] * math.cos(ang) - vec[a + 1] * math.sin(ang)
                    out[a + 1] = vec[a] * math.sin(ang) + vec[a + 1] * math.cos(ang)
        return out

    sc = [a / (1 + math.exp(-a)) for a in c]
    xs = {"txt": [list(r) for r in x_txt], "img": [list(r) for r in x_img]}
    mod, qs, ks, vs = {}, [], [], []
    for s in mmdit.STREAMS:
        p = f"blocks.{b}.{s}."
        m = lin(sc, W[p + "ada.w"], W[p + "ada.b"])
        mod[s] = [m[i * D:(i + 1) * D] for i in range(6)]
        for t, row in enumerate(xs[s]):
            hv = [n * (1 + mod[s][1][i]) + mod[s][0][i] for i, n in enumerate(ln(row))]
            qkv = lin(hv, W[p + "qkv.w"], W[p + "qkv.b"])
            q, k, v = qkv[:D], qkv[D:2 * D], qkv[2 * D:]
            if s == "img":
                q, k = rot(q, rows[t], cols[t]), rot(k, rows[t], cols[t])
            qs.append(q), ks.append(k), vs.append(v)
    o = []
    for qi in qs:
        out = [0.0] * D
        for h in range(H):
            sc_ = [sum(qi[h * d + e] * kj[h * d + e] for e in range(d)) / math.sqrt(d) for kj in ks]
            mx = max(sc_)
            ex = [math.exp(a - mx) for a in sc_]
            z = sum(ex)
            for e in range(d):
                out[h * d + e] = sum(ex[j] * vs[j][h * d + e] for j in range(len(ks))) / z
        o.append(out)
    nt = len(xs["txt"])
    outs = {"txt": o[:nt], "img": o[nt:]}
    new = {}
    for s in mmdit.STREAMS:
        p = f"blocks.{b}.{s}."
        sh1, s1, g1, sh2, s2, g2 = mod[s]
        res = []
        for t, row in enumerate(xs[s]):
            po = lin(outs[s][t], W[p + "o.w"], W[p + "o.b"])
            r = [row[i] + g1[i] * po[i] for i in range(D)]
            hv = [n * (1 + s2[i]) + sh2[i] for i, n in enumerate(ln(r))]
            u = lin(hv, W[p + "fc1.w"], W[p + "fc1.b"])
            u = [0.5 * a * (1 + math.tanh(math.sqrt(2 / math.pi) * (a + 0.044715 * a ** 3)))
                 for a in u]
            f = lin(u, W[p + "fc2.w"], W[p + "fc2.b"])
            res.append([r[i] + g2[i] * f[i] for i in range(D)])
        new[s] = np.array(res).reshape(len(res), D)
    return new["txt"], new["img"]


def _joint_inputs(seed=31):
    rng = np.random.default_rng(seed)
    D = TINY.hidden
    return (rng.standard_normal((3, D)), rng.standard_normal((6, D)) * 0.7,
            rng.standard_normal(D))


def test_joint_block_both_streams_brute_force():
    """Text and image stream outputs of joint_block against scalar loops."""
    W = weights()
    xt, xi, c = _joint_inputs()
    rows, cols = mmdit.grid_positions(2, 3)
    for b in range(TINY.depth):
        nt, ni = mmdit.joint_block(W, TINY, b, xt, xi, c, rows, cols)
        bt, bi = brute_joint_block(W, TINY, b, xt, xi, c, rows, cols)
        assert np.allclose(nt, bt, rtol=1e-11, atol=1e-12), b
        assert np.allclose(ni, bi, rtol=1e-11, atol=1e-12), b


def test_forward_two_blocks_brute_force_composition():
    """mmdit.forward = embed (loops) -> 2 brute joint blocks -> final layer
    (loops) on the image stream; the text stream after the blocks too."""
    W = weights()
    rng = np.random.default_rng(32)
    C, p, D = TINY.latent_channels, TINY.patch, TINY.hidden
    lat = rng.standard_normal((C, 4, 6))
    text = rng.standard_normal((TINY.text_tokens, TINY.text_dim))
    t = 0.61
    v, xt_o, xi_o = mmdit.forward(W, TINY, lat, t, text)
    gh, gw = 2, 3
    xi = np.zeros((gh * gw, D))
    for i in range(gh):
        for j in range(gw):
            for o in range(D):
                s = W["x_embed.b"][o]
                for a in range(p):
                    for bb in range(p):
                        for cc in range(C):
                            s += W["x_embed.w"][o, (a * p + bb) * C + cc] * lat[cc, i * p + a, j * p + bb]
                xi[i * gw + j, o] = s
    xt = np.array([[W["y_embed.b"][o] + sum(W["y_embed.w"][o, k] * text[r, k]
                                             for k in range(TINY.text_dim))
                    for o in range(D)] for r in range(TINY.text_tokens)])
    # conditioning by loops (sinusoid, Linear, SiLU, Linear)
    half = TINY.freq_dim // 2
    s_t = TINY.t_scale * t
    e = [math.cos(s_t * math.exp(-math.log(10000.0) * k / half)) for k in range(half)] + \
        [math.sin(s_t * math.exp(-math.log(10000.0) * k / half)) for k in range(half)]
    h1 = [W["t_embed.b1"][o] + sum(W["t_embed.w1"][o, k] * e[k] for k in range(len(e)))
          for o in range(D)]
    h1 = [a / (1 + math.exp(-a)) for a in h1]
    c = [W["t_embed.b2"][o] + sum(W["t_embed.w2"][o, k] * h1[k] for k in range(D)) for o in range(D)]
    rows, cols = mmdit.grid_positions(gh, gw)
    for b in range(TINY.depth):
        xt, xi = brute_joint_block(W, TINY, b, xt, xi, c, rows, cols)
    assert np.allclose(xt_o, xt, rtol=1e-10, atol=1e-11)
    assert np.allclose(xi_o, xi, rtol=1e-10, atol=1e-11)
    sc = [a / (1 + math.exp(-a)) for a in c]
    fm = [W["final.ada.b"][o] + sum(W["final.ada.w"][o, k] * sc[k] for k in range(D))
          for o in range(2 * D)]
    out = np.zeros_like(lat)
    for i in range(gh):
        for j in range(gw):
            r = xi[i * gw + j]
            mu = r.mean()
            sd = math.sqrt(((r - mu) ** 2).mean() + TINY.ln_eps)
            hm = [(r[k] - mu) / sd * (1 + fm[D + k]) + fm[k] for k in range(D)]
            for a in range(p):
                for bb in range(p):
                    for cc in range(C):
                        f = (a * p + bb) * C + cc
                        out[cc, i * p + a, j * p + bb] = W["final.out.b"][f] + sum(
                            W["final.out.w"][f, k] * hm[k] for k in range(D))
    assert np.allclose(v, out, rtol=1e-10, atol=1e-11)


class _Redirect(dict):
    """A weight dict that answers reads of one stream's tensors with another
    stream's: simulates an oracle that indexes the wrong parameter."""

    def __init__(self, base, frm, to):
        super().__init__(base)
        self.frm, self.to = frm, to

    def __getitem__(self, k):
        for part in self.frm:
            if part in k:
                k = k.replace(part, self.to[part])
        return dict.__getitem__(self, k)


@pytest.mark.parametrize("mutation", ["txt_uses_img_o_proj", "txt_uses_img_modulation",
                                      "txt_uses_img_mlp", "o_rows_shifted", "rope_on_text",
                                      "txt_uses_img_qkv"])
def test_pins_catch_planted_text_stream_mistakes(monkeypatch, mutation):
    """Plant a plausible text-stream mistake in the MMDiT oracle; the
    scalar-loop pin of the text stream must see it."""
    W = weights()
    xt, xi, c = _joint_inputs(33)
    rows, cols = mmdit.grid_positions(2, 3)
    bt, bi = brute_joint_block(W, TINY, 0, xt, xi, c, rows, cols)
    nt, _ = mmdit.joint_block(W, TINY, 0, xt, xi, c, rows, cols)
    assert np.max(np.abs(nt - bt)) < 1e-11
    Wm = W
    if mutation == "txt_uses_img_o_proj":
        Wm = _Redirect(W, ["txt.o."], {"txt.o.": "img.o."})
    elif mutation == "txt_uses_img_modulation":
        Wm = _Redirect(W, ["txt.ada."], {"txt.ada.": "img.ada."})
    elif mutation == "txt_uses_img_mlp":
        Wm = _Redirect(W, ["txt.fc2."], {"txt.fc2.": "img.fc2."})
    elif mutation == "txt_uses_img_qkv":
        Wm = _Redirect(W, ["txt.qkv."], {"txt.qkv.": "img.qkv."})
    elif mutation == "o_rows_shifted":
        orig = mmdit.attention
        monkeypatch.setattr(mmdit, "attention", lambda q, k, v, h: np.roll(orig(q, k, v, h), 1, axis=0))
    elif mutation == "rope_on_text":
        # the text rows rotated as if they were tokens (i, 0) of the grid
        orig = mmdit.attention
        nt_rows = xt.shape[0]

        def attn_rot(q, k, v, h):
            q, k = np.array(q), np.array(k)
            pos = np.arange(nt_rows)
            q[:nt_rows] = mmdit.rope_2d(q[:nt_rows], pos + 1, pos * 0, h)
            k[:nt_rows] = mmdit.rope_2d(k[:nt_rows], pos + 1, pos * 0, h)
            return orig(q, k, v, h)
        monkeypatch.setattr(mmdit, "attention", attn_rot)
    mt, _ = mmdit.joint_block(Wm, TINY, 0, xt, xi, c, rows, cols)
    assert np.max(np.abs(mt - bt)) > 1e-6
