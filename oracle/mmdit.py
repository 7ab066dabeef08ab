"""Joint-attention (MMDiT-style) transformer in float64 -- test infrastructure only.

The second model family served by the paper's workflows (SD3.5, Flux, Sec. 8.1)
concatenates text and image tokens into one attention.  Readings for what the
paper leaves open:

* text ``y`` is projected ``y W_ctx^T + b`` to the model width; the image is
  patchified as in :mod:`oracle.dit` with no absolute position embedding;
* conditioning ``c`` is the timestep embedding; each block owns one
  adaLN-Zero projection per stream, chunks ordered as in :mod:`oracle.dit`;
* per stream: ``h = LNmod(x)``, ``qkv = h W_qkv^T + b``; image q and k are
  rotated by a 2D RoPE; attention runs over the concatenation ``[text; image]``;
  outputs split back; ``x += g_msa * (o W_o^T + b)``;
  ``x += g_mlp * MLP(LNmod(x))``; no QK-norm; the last block computes the text
  stream in full;
* 2D RoPE per head of width d: the first d/2 dimensions rotate by the token's
  row, the last d/2 by its column; within a half, dimensions ``(2j, 2j+1)``,
  ``j < d/4``, rotate by ``pos * 10000^(-j/(d/4))``:
  ``(a, b) -> (a cos - b sin, a sin + b cos)``; text tokens are not rotated;
* the final layer acts on the image stream only;
* classifier-free guidance runs the unconditional branch with an all-zero
  prompt, whose text stream then evolves through the blocks like any other;
* the step-skip signal is block 0's first modulated input of the image
  stream, and the cached residual is that of the image stream.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

from .dit import (F64, silu, gelu_tanh, linear, layer_norm, modulate,
                  attention, patchify, unpatchify, conditioning, final_layer)

STREAMS = ("txt", "img")


def weight_layout(w) -> List[Tuple[str, Tuple[int, ...]]]:
    D, F, P = w.hidden, w.mlp_hidden, w.patch_dim
    L = [("x_embed.w", (D, P)), ("x_embed.b", (D,)),
         ("t_embed.w1", (D, w.freq_dim)), ("t_embed.b1", (D,)),
         ("t_embed.w2", (D, D)), ("t_embed.b2", (D,)),
         ("y_embed.w", (D, w.text_dim)), ("y_embed.b", (D,))]
    for b in range(w.depth):
        for s in STREAMS:
            p = f"blocks.{b}.{s}."
            L += [(p + "ada.w", (6 * D, D)), (p + "ada.b", (6 * D,)),
                  (p + "qkv.w", (3 * D, D)), (p + "qkv.b", (3 * D,)),
                  (p + "o.w", (D, D)), (p + "o.b", (D,)),
                  (p + "fc1.w", (F, D)), (p + "fc1.b", (F,)),
                  (p + "fc2.w", (D, F)), (p + "fc2.b", (D,))]
    L += [("final.ada.w", (2 * D, D)), ("final.ada.b", (2 * D,)),
          ("final.out.w", (P, D)), ("final.out.b", (P,))]
    return L


def as_dict(w, tensors: Sequence[np.ndarray]) -> Dict[str, np.ndarray]:
    """Name a (possibly leading-prefix) list of tensors and widen to float64."""
    lay = weight_layout(w)
    out = {}
    for (name, shape), t in zip(lay, tensors):
        out[name] = np.asarray(t, dtype=F64).reshape(shape)
    return out


def rope_2d(x, rows, cols, heads):
    """Rotate every head of ``x [N, H*d]`` by the token grid positions."""
    n, dm = x.shape
    d = dm // heads
    q = d // 4
    theta = 10000.0 ** (-np.arange(q, dtype=F64) / q)
    out = np.array(x, dtype=F64, copy=True)
    for h in range(heads):
        for half, pos in ((0, rows), (1, cols)):
            base = h * d + half * (d // 2)
            ang = np.asarray(pos, dtype=F64)[:, None] * theta[None, :]
            c, s = np.cos(ang), np.sin(ang)
            a = x[:, base + 0:base + d // 2:2]
            b = x[:, base + 1:base + d // 2:2]
            out[:, base + 0:base + d // 2:2] = a * c - b * s
            out[:, base + 1:base + d // 2:2] = a * s + b * c
    return out


def grid_positions(gh, gw):
    ii, jj = np.meshgrid(np.arange(gh), np.arange(gw), indexing="ij")
    return ii.ravel(), jj.ravel()


def stream_modulation(W, w, c, b, s):
    m = linear(silu(c), W[f"blocks.{b}.{s}.ada.w"], W[f"blocks.{b}.{s}.ada.b"])
    names = ("shift_msa", "scale_msa", "gate_msa", "shift_mlp", "scale_mlp", "gate_mlp")
    D = w.hidden
    return {n: m[i * D:(i + 1) * D] for i, n in enumerate(names)}


def joint_block(W, w, b, x_txt, x_img, c, rows, cols):
    D, H = w.hidden, w.heads
    xs = {"txt": x_txt, "img": x_img}
    mods, q, k, v = {}, {}, {}, {}
    for s in STREAMS:
        p = f"blocks.{b}.{s}."
        mods[s] = stream_modulation(W, w, c, b, s)
        h = modulate(layer_norm(xs[s], w.ln_eps), mods[s]["shift_msa"], mods[s]["scale_msa"])
        qkv = linear(h, W[p + "qkv.w"], W[p + "qkv.b"])
        q[s], k[s], v[s] = qkv[:, :D], qkv[:, D:2 * D], qkv[:, 2 * D:]
    q["img"] = rope_2d(q["img"], rows, cols, H)
    k["img"] = rope_2d(k["img"], rows, cols, H)
    o = attention(np.concatenate([q["txt"], q["img"]]),
                  np.concatenate([k["txt"], k["img"]]),
                  np.concatenate([v["txt"], v["img"]]), H)
    nt = x_txt.shape[0]
    outs = {"txt": o[:nt], "img": o[nt:]}
    new = {}
    for s in STREAMS:
        p = f"blocks.{b}.{s}."
        md = mods[s]
        x = xs[s] + md["gate_msa"] * linear(outs[s], W[p + "o.w"], W[p + "o.b"])
        h = modulate(layer_norm(x, w.ln_eps), md["shift_mlp"], md["scale_mlp"])
        u = gelu_tanh(linear(h, W[p + "fc1.w"], W[p + "fc1.b"]))
        new[s] = x + md["gate_mlp"] * linear(u, W[p + "fc2.w"], W[p + "fc2.b"])
    return new["txt"], new["img"]


def joint_block_rows(W, w, b, x_txt, x_img, c, rows, cols, sel_txt, sel_img):
    """:func:`joint_block` evaluated for the selected output rows only.

    Keys and values come from every row of both streams; queries, the output
    projection and the MLP from the selected rows (``sel_txt`` index text
    rows, ``sel_img`` image rows).  Returns the selected rows' new values."""
    D, H = w.hidden, w.heads
    xs = {"txt": x_txt, "img": x_img}
    sel = {"txt": np.asarray(sel_txt, dtype=int), "img": np.asarray(sel_img, dtype=int)}
    mods, q, k, v = {}, {}, {}, {}
    for s in STREAMS:
        p = f"blocks.{b}.{s}."
        mods[s] = stream_modulation(W, w, c, b, s)
        h = modulate(layer_norm(xs[s], w.ln_eps), mods[s]["shift_msa"], mods[s]["scale_msa"])
        wq, bq = W[p + "qkv.w"], W[p + "qkv.b"]
        q[s] = linear(h[sel[s]], wq[:D], bq[:D])
        k[s] = linear(h, wq[D:2 * D], bq[D:2 * D])
        v[s] = linear(h, wq[2 * D:], bq[2 * D:])
    rows, cols = np.asarray(rows), np.asarray(cols)
    q["img"] = rope_2d(q["img"], rows[sel["img"]], cols[sel["img"]], H)
    k["img"] = rope_2d(k["img"], rows, cols, H)
    o = attention(np.concatenate([q["txt"], q["img"]]),
                  np.concatenate([k["txt"], k["img"]]),
                  np.concatenate([v["txt"], v["img"]]), H)
    ns = len(sel["txt"])
    outs = {"txt": o[:ns], "img": o[ns:]}
    new = {}
    for s in STREAMS:
        p = f"blocks.{b}.{s}."
        md = mods[s]
        x = xs[s][sel[s]] + md["gate_msa"] * linear(outs[s], W[p + "o.w"], W[p + "o.b"])
        h = modulate(layer_norm(x, w.ln_eps), md["shift_mlp"], md["scale_mlp"])
        u = gelu_tanh(linear(h, W[p + "fc1.w"], W[p + "fc1.b"]))
        new[s] = x + md["gate_mlp"] * linear(u, W[p + "fc2.w"], W[p + "fc2.b"])
    return new["txt"], new["img"]


def embed_image(W, w, lat):
    return linear(patchify(np.asarray(lat, dtype=F64), w.patch), W["x_embed.w"], W["x_embed.b"])


def embed_text(W, w, text):
    """Initial text stream; ``None`` is the unconditional (all-zero) prompt."""
    if text is None:
        text = np.zeros((w.text_tokens, w.text_dim))
    return linear(np.asarray(text, dtype=F64), W["y_embed.w"], W["y_embed.b"])


def embed(W, w, lat, text):
    return embed_text(W, w, text), embed_image(W, w, lat)


def run_blocks(W, w, x_txt, x_img, c, lat_hw, b0, b1, control=None):
    """Joint blocks ``b0 .. b1-1`` for a latent of spatial size ``lat_hw``;
    ``control`` residuals (block -> array) are added to the image stream."""
    rows, cols = grid_positions(lat_hw[0] // w.patch, lat_hw[1] // w.patch)
    for b in range(b0, b1):
        x_txt, x_img = joint_block(W, w, b, x_txt, x_img, c, rows, cols)
        if control is not None and b in control:
            x_img = x_img + control[b]
    return x_txt, x_img


def cache_signal(W, w, lat, t):
    """Block 0's first modulated input of the image stream ``[N, D]`` (the
    quantity the step-skip rule compares between steps)."""
    c = conditioning(W, w, t)
    md = stream_modulation(W, w, c, 0, "img")
    return modulate(layer_norm(embed_image(W, w, lat), w.ln_eps),
                    md["shift_msa"], md["scale_msa"])


def forward(W, w, lat, t, text, n_blocks=None, control=None):
    """Returns ``(v, x_txt, x_img)``; ``v`` is None unless all blocks ran.
    ``text`` None is the unconditional prompt."""
    C, h, ww = lat.shape
    c = conditioning(W, w, t)
    x_txt, x_img = embed(W, w, lat, text)
    nb = w.depth if n_blocks is None else n_blocks
    x_txt, x_img = run_blocks(W, w, x_txt, x_img, c, (h, ww), 0, nb, control)
    v = final_layer(W, w, x_img, c, h, ww) if nb == w.depth else None
    return v, x_txt, x_img
