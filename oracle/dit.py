"""Cross-attention DiT forward in float64 -- test infrastructure only.

One call of the base diffusion model (the ``execute`` of a model function,
ServerlessT2I Sec. 4, Fig. "Flux function"): a latent ``[C, h, w]``, a
timestep ``t`` and text embeddings ``[M, Dt]`` in, a velocity ``[C, h, w]``
out.  The paper leaves the architecture open; the readings used here:

* patchify: token ``i*(w/p)+j``, feature ``(a*p+b)*C+c`` <- latent
  ``[c, i*p+a, j*p+b]`` (channel fastest);
* fixed 2D sin-cos position embedding added after the patch embedding: the
  first D/2 channels encode the token's row, the last D/2 its column, each
  half ``[sin(pos*w_k) ..., cos(pos*w_k) ...]`` with ``w_k = 10000^(-k/(D/4))``;
* timestep: ``s = t_scale*t``, ``[cos(s f_k) ..., sin(s f_k) ...]`` with
  ``f_k = exp(-ln(10000) k / (freq_dim/2))``, then Linear -> SiLU -> Linear;
* conditioning ``c`` is the timestep embedding alone; every block owns an
  adaLN-Zero projection ``SiLU(c) W^T + b`` split as
  ``[shift_msa, scale_msa, gate_msa, shift_mlp, scale_mlp, gate_mlp]``;
  the final layer's projection splits as ``[shift, scale]``;
* LayerNorm without affine, biased variance, eps ``ln_eps``;
  modulation ``h = LN(x) * (1 + scale) + shift``;
* block: ``x += g_msa * SelfAttn(LNmod_msa(x))``;
  ``x += CrossAttn(x, y')`` (query from the raw residual, ungated);
  ``x += g_mlp * MLP(LNmod_mlp(x))`` with a tanh-approximate GELU;
* fused projections: qkv columns ``[q | k | v]``, cross kv columns ``[k | v]``,
  head ``h`` at columns ``h*d ... h*d+d-1``; no mask, no QK-norm;
* text ``y' = y W_cap^T + b_cap`` once per request;
* final layer ``LNmod(x; shift, scale) W_out^T + b_out`` then unpatchify, the
  output read as the velocity dx/dt.
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence, Tuple

import numpy as np

F64 = np.float64


# --------------------------------------------------------------------------
# weight table

def weight_layout(w) -> List[Tuple[str, Tuple[int, ...]]]:
    """(name, shape) of every parameter, in table order.

    Linear weights are ``[out, in]``; the table is the per-layer lookup of
    parameter tensors the model function reads (Sec. 5.3)."""
    D, F, P = w.hidden, w.mlp_hidden, w.patch_dim
    L = [("x_embed.w", (D, P)), ("x_embed.b", (D,)),
         ("t_embed.w1", (D, w.freq_dim)), ("t_embed.b1", (D,)),
         ("t_embed.w2", (D, D)), ("t_embed.b2", (D,)),
         ("y_embed.w", (D, w.text_dim)), ("y_embed.b", (D,))]
    for b in range(w.depth):
        p = f"blocks.{b}."
        L += [(p + "ada.w", (6 * D, D)), (p + "ada.b", (6 * D,)),
              (p + "attn.qkv.w", (3 * D, D)), (p + "attn.qkv.b", (3 * D,)),
              (p + "attn.o.w", (D, D)), (p + "attn.o.b", (D,)),
              (p + "xattn.q.w", (D, D)), (p + "xattn.q.b", (D,)),
              (p + "xattn.kv.w", (2 * D, D)), (p + "xattn.kv.b", (2 * D,)),
              (p + "xattn.o.w", (D, D)), (p + "xattn.o.b", (D,)),
              (p + "mlp.fc1.w", (F, D)), (p + "mlp.fc1.b", (F,)),
              (p + "mlp.fc2.w", (D, F)), (p + "mlp.fc2.b", (D,))]
    L += [("final.ada.w", (2 * D, D)), ("final.ada.b", (2 * D,)),
          ("final.out.w", (P, D)), ("final.out.b", (P,))]
    return L


def as_dict(w, tensors: Sequence[np.ndarray]) -> Dict[str, np.ndarray]:
    """Name the tensors of a weight table and widen them to float64."""
    lay = weight_layout(w)
    return {name: np.asarray(t, dtype=F64).reshape(shape)
            for (name, shape), t in zip(lay, tensors)}


# --------------------------------------------------------------------------
# elementary operations

def silu(x):
    return x / (1.0 + np.exp(-x))


def gelu_tanh(u):
    """Tanh approximation of GELU (Hendrycks and Gimpel)."""
    return 0.5 * u * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (u + 0.044715 * u ** 3)))


def linear(x, weight, bias):
    """``x W^T + b`` with ``W`` stored ``[out, in]``."""
    return x @ weight.T + bias


def layer_norm(x, eps):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def modulate(xn, shift, scale):
    return xn * (1.0 + scale) + shift


def softmax_rows(s):
    s = s - s.max(axis=-1, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=-1, keepdims=True)


def attention(q, k, v, heads):
    """Multi-head scaled dot-product attention, no mask.

    ``q [Nq, H*d]``, ``k, v [Nk, H*d]``; head ``h`` occupies columns
    ``h*d ... h*d+d-1``; each head computes ``softmax(Q K^T / sqrt(d)) V``."""
    nq, dm = q.shape
    d = dm // heads
    out = np.empty((nq, dm), dtype=F64)
    for h in range(heads):
        cols = slice(h * d, (h + 1) * d)
        p = softmax_rows((q[:, cols] @ k[:, cols].T) / math.sqrt(d))
        out[:, cols] = p @ v[:, cols]
    return out


# --------------------------------------------------------------------------
# embeddings

def patchify(lat, p):
    """``[C, h, w]`` -> ``[(h/p)(w/p), p*p*C]``, channel fastest."""
    C, h, w = lat.shape
    t = lat.reshape(C, h // p, p, w // p, p)          # c, i, a, j, b
    return t.transpose(1, 3, 2, 4, 0).reshape((h // p) * (w // p), p * p * C)


def unpatchify(tok, p, C, h, w):
    """Inverse of :func:`patchify`."""
    t = tok.reshape(h // p, w // p, p, p, C)            # i, j, a, b, c
    return t.transpose(4, 0, 2, 1, 3).reshape(C, h, w)


def sincos_1d(pos, dim):
    """``[sin(pos w_k) for k < dim/2] + [cos(pos w_k) ...]``, ``w_k = 10000^(-k/(dim/2))``."""
    half = dim // 2
    omega = 10000.0 ** (-np.arange(half, dtype=F64) / half)
    ang = np.asarray(pos, dtype=F64)[:, None] * omega[None, :]
    return np.concatenate([np.sin(ang), np.cos(ang)], axis=1)


def pos_embed_2d(gh, gw, D):
    """Fixed 2D sin-cos position embedding ``[gh*gw, D]``: rows then columns."""
    ii, jj = np.meshgrid(np.arange(gh), np.arange(gw), indexing="ij")
    return np.concatenate([sincos_1d(ii.ravel(), D // 2),
                           sincos_1d(jj.ravel(), D // 2)], axis=1)


def timestep_frequencies(t, w):
    """``[cos(s f_k) ..., sin(s f_k) ...]`` for ``s = t_scale * t``."""
    half = w.freq_dim // 2
    f = np.exp(-math.log(10000.0) * np.arange(half, dtype=F64) / half)
    s = w.t_scale * float(t)
    return np.concatenate([np.cos(s * f), np.sin(s * f)])


def conditioning(W, w, t):
    """Timestep embedding ``c [D]``: Linear -> SiLU -> Linear."""
    e = timestep_frequencies(t, w)
    h = silu(linear(e, W["t_embed.w1"], W["t_embed.b1"]))
    return linear(h, W["t_embed.w2"], W["t_embed.b2"])


def block_modulation(W, w, c, b):
    """adaLN-Zero chunks of block ``b``: dict of six ``[D]`` vectors."""
    m = linear(silu(c), W[f"blocks.{b}.ada.w"], W[f"blocks.{b}.ada.b"])
    names = ("shift_msa", "scale_msa", "gate_msa", "shift_mlp", "scale_mlp", "gate_mlp")
    D = w.hidden
    return {n: m[i * D:(i + 1) * D] for i, n in enumerate(names)}


def final_modulation(W, w, c):
    m = linear(silu(c), W["final.ada.w"], W["final.ada.b"])
    return m[:w.hidden], m[w.hidden:]


def embed(W, w, lat):
    """Patch embedding plus position embedding: residual stream ``x0 [N, D]``."""
    C, h, ww = lat.shape
    tok = patchify(np.asarray(lat, dtype=F64), w.patch)
    pe = pos_embed_2d(h // w.patch, ww // w.patch, w.hidden)
    return linear(tok, W["x_embed.w"], W["x_embed.b"]) + pe


def text_project(W, w, text):
    return linear(np.asarray(text, dtype=F64), W["y_embed.w"], W["y_embed.b"])


# --------------------------------------------------------------------------
# transformer block and final layer

def block(W, w, b, x, y, mod):
    """One adaLN-Zero block with self-attention, cross-attention and MLP."""
    p = f"blocks.{b}."
    D, H = w.hidden, w.heads
    h = modulate(layer_norm(x, w.ln_eps), mod["shift_msa"], mod["scale_msa"])
    qkv = linear(h, W[p + "attn.qkv.w"], W[p + "attn.qkv.b"])
    o = attention(qkv[:, :D], qkv[:, D:2 * D], qkv[:, 2 * D:], H)
    x = x + mod["gate_msa"] * linear(o, W[p + "attn.o.w"], W[p + "attn.o.b"])

    q = linear(x, W[p + "xattn.q.w"], W[p + "xattn.q.b"])
    kv = linear(y, W[p + "xattn.kv.w"], W[p + "xattn.kv.b"])
    o = attention(q, kv[:, :D], kv[:, D:], H)
    x = x + linear(o, W[p + "xattn.o.w"], W[p + "xattn.o.b"])

    h = modulate(layer_norm(x, w.ln_eps), mod["shift_mlp"], mod["scale_mlp"])
    u = gelu_tanh(linear(h, W[p + "mlp.fc1.w"], W[p + "mlp.fc1.b"]))
    return x + mod["gate_mlp"] * linear(u, W[p + "mlp.fc2.w"], W[p + "mlp.fc2.b"])


def block_rows(W, w, b, x, y, mod, rows):
    """Output rows ``rows`` of :func:`block` (self-attention keys and values
    from every row of ``x``); every other step acts on each row alone, so this
    equals ``block(...)[rows]`` while evaluating far fewer rows."""
    p = f"blocks.{b}."
    D, H = w.hidden, w.heads
    h = modulate(layer_norm(x, w.ln_eps), mod["shift_msa"], mod["scale_msa"])
    qkv = linear(h, W[p + "attn.qkv.w"], W[p + "attn.qkv.b"])
    xr = x[rows]
    o = attention(qkv[rows, :D], qkv[:, D:2 * D], qkv[:, 2 * D:], H)
    xr = xr + mod["gate_msa"] * linear(o, W[p + "attn.o.w"], W[p + "attn.o.b"])
    q = linear(xr, W[p + "xattn.q.w"], W[p + "xattn.q.b"])
    kv = linear(y, W[p + "xattn.kv.w"], W[p + "xattn.kv.b"])
    o = attention(q, kv[:, :D], kv[:, D:], H)
    xr = xr + linear(o, W[p + "xattn.o.w"], W[p + "xattn.o.b"])
    h = modulate(layer_norm(xr, w.ln_eps), mod["shift_mlp"], mod["scale_mlp"])
    u = gelu_tanh(linear(h, W[p + "mlp.fc1.w"], W[p + "mlp.fc1.b"]))
    return xr + mod["gate_mlp"] * linear(u, W[p + "mlp.fc2.w"], W[p + "mlp.fc2.b"])


def run_blocks(W, w, x, y, c, first=0, last=None, control=None):
    """Blocks ``first ... last-1`` on the residual stream.

    ``control`` maps a block index to a residual added to the stream right
    after that block: the model function's callback input ``control_outputs``
    (Sec. 4), the per-layer outputs a ControlNet feeds into the base model."""
    last = w.depth if last is None else last
    for b in range(first, last):
        x = block(W, w, b, x, y, block_modulation(W, w, c, b))
        if control is not None and b in control:
            x = x + control[b]
    return x


def final_layer(W, w, x, c, h, ww):
    shift, scale = final_modulation(W, w, c)
    out = linear(modulate(layer_norm(x, w.ln_eps), shift, scale),
                 W["final.out.w"], W["final.out.b"])
    return unpatchify(out, w.patch, w.latent_channels, h, ww)


def forward(W, w, lat, t, text, n_blocks=None, return_hidden=False, control=None):
    """Velocity of one request: ``[C, h, w]`` latent at time ``t``.

    ``text`` ``None`` means the unconditional (all-zero) text; ``control`` as
    in :func:`run_blocks`."""
    C, h, ww = lat.shape
    if text is None:
        text = np.zeros((w.text_tokens, w.text_dim))
    c = conditioning(W, w, t)
    x = embed(W, w, lat)
    y = text_project(W, w, text)
    x = run_blocks(W, w, x, y, c, 0, w.depth if n_blocks is None else n_blocks, control)
    v = final_layer(W, w, x, c, h, ww)
    return (v, x) if return_hidden else v


def cache_signal(W, w, lat, t):
    """Modulated input of block 0: ``LNmod(x0; shift_msa, scale_msa)`` ``[N, D]``.

    The quantity whose step-to-step relative L1 change drives the cache-skip
    rule (see :mod:`oracle.sampler`)."""
    c = conditioning(W, w, t)
    mod = block_modulation(W, w, c, 0)
    return modulate(layer_norm(embed(W, w, lat), w.ln_eps),
                    mod["shift_msa"], mod["scale_msa"])
