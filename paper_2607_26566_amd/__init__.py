"""MI355X-native diffusion-transformer denoising step (ServerlessT2I's hot path).

Thin Python binding of ``libt2i_dit.so``.  PyTorch provides device memory and
the HIP stream; every step of the computation runs in the library's gfx950
kernels.  The functions below carry the C ABI's names:

* :func:`t2i_dit_init`   -> :class:`DiT` (binds weights and a workspace)
* :func:`t2i_dit_step`   one model evaluation (+ guidance, + Euler update)
* :func:`t2i_dit_sample` the whole denoising loop with the optional cache skip
* :func:`t2i_cache_check` the cache-skip decision of one step
* :func:`t2i_dit_host_tier`, :func:`t2i_dit_evict`, :func:`t2i_dit_load_async`,
  :func:`t2i_dit_block_state`: first-layers caching with progressive loading
"""
from __future__ import annotations

import ctypes as C
from typing import List, Optional, Sequence

import numpy as np
import torch

from . import _lib
from ._lib import (T2I_F32, T2I_BF16, T2I_ARCH_CROSS_DIT, T2I_ARCH_MMDIT,
                   T2I_CACHE_ACCUMULATE, T2I_CACHE_PER_STEP, T2IError, check, load)

__all__ = ["Config", "DiT", "t2i_dit_init", "t2i_dit_init_static", "t2i_dit_step", "t2i_dit_sample",
           "t2i_cache_check", "weight_table", "upload", "T2IError", "load",
           "t2i_dit_block_layout", "pack_blocks", "t2i_dit_host_tier", "t2i_dit_evict",
           "t2i_dit_load_async", "t2i_dit_block_state", "t2i_first_layers"]


def _stream(stream=None) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _arr(ctype, values):
    n = len(values)
    return (ctype * n)(*values)


class Config:
    """Model shape (``t2i_dit_config``)."""

    def __init__(self, *, arch="cross", dtype="bf16", latent_channels, patch, hidden,
                 heads, head_dim, depth, mlp_hidden, text_dim, text_tokens, freq_dim=256,
                 max_tokens, max_requests=1, max_steps=1, ln_eps=1e-6, t_scale=1000.0):
        self.c = _lib.t2i_dit_config(
            C.sizeof(_lib.t2i_dit_config),
            T2I_ARCH_CROSS_DIT if arch == "cross" else T2I_ARCH_MMDIT,
            T2I_BF16 if dtype == "bf16" else T2I_F32,
            latent_channels, patch, hidden, heads, head_dim, depth, mlp_hidden, text_dim,
            text_tokens, freq_dim, max_tokens, max_requests, max_steps, ln_eps, t_scale)
        self.dtype = dtype

    @classmethod
    def from_shape(cls, w, max_tokens=None, max_requests=None, max_steps=None):
        """Build from any object with the workload attributes (arch, dtype, ...)."""
        return cls(arch=w.arch, dtype=w.dtype, latent_channels=w.latent_channels,
                   patch=w.patch, hidden=w.hidden, heads=w.heads, head_dim=w.head_dim,
                   depth=w.depth, mlp_hidden=w.mlp_hidden, text_dim=w.text_dim,
                   text_tokens=w.text_tokens, freq_dim=w.freq_dim,
                   max_tokens=max_tokens if max_tokens else w.image_tokens * w.branches,
                   max_requests=max_requests if max_requests else w.n_req,
                   max_steps=max_steps if max_steps else w.steps,
                   ln_eps=w.ln_eps, t_scale=w.t_scale)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def ref(self):
        return C.byref(self.c)


def weight_table(cfg: Config):
    """[(name, shape)] of the library's weight table for ``cfg``."""
    lib = load()
    n = lib.t2i_dit_weight_count(cfg.ref())
    if n == 0:
        raise T2IError(1, "invalid config")
    out = []
    name = C.create_string_buffer(64)
    shape = (C.c_int64 * 4)()
    dt = C.c_int32()
    for i in range(n):
        check(lib.t2i_dit_weight_desc(cfg.ref(), i, name, shape, C.byref(dt)))
        out.append((name.value.decode(), tuple(int(s) for s in shape if s)))
    return out


def upload(arrays: Sequence[np.ndarray], dtype: str, device="cuda") -> List[torch.Tensor]:
    """Copy host arrays (float32 values, already bf16-representable for bf16)
    to device tensors of the model dtype."""
    out = []
    for a in arrays:
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
        out.append(t.to(device=device, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32))
    return out


class DiT:
    """A bound model: weights + workspace + library handle (``t2i_dit_init``)."""

    def __init__(self, cfg: Config, weights: Sequence[torch.Tensor], device="cuda", stream=None,
                 static_workspace=False):
        lib = load()
        self.cfg = cfg
        self.lib = lib
        table = weight_table(cfg)
        if len(weights) != len(table):
            raise T2IError(2, f"expected {len(table)} weight tensors, got {len(weights)}")
        for (name, shape), w in zip(table, weights):
            if tuple(w.shape) != shape or w.dtype != cfg.torch_dtype or not w.is_contiguous():
                raise T2IError(2, f"weight {name}: expected {shape} {cfg.torch_dtype} contiguous")
        self.weights = list(weights)
        ptrs = (C.c_void_p * len(self.weights))(*[w.data_ptr() for w in self.weights])
        h = C.c_void_p()
        if static_workspace:
            # the library's static device array (t2i_dit_init_static): nothing allocated
            self.workspace = None
            st = lib.t2i_dit_init_static(cfg.ref(), ptrs, C.c_void_p(_stream(stream)), C.byref(h))
            if st != 0:
                raise T2IError(st, "t2i_dit_init_static failed")
        else:
            ws = lib.t2i_dit_workspace_bytes(cfg.ref())
            self.workspace = torch.empty(ws, dtype=torch.uint8, device=device)
            check(lib.t2i_dit_init(cfg.ref(), ptrs, C.c_void_p(self.workspace.data_ptr()), ws,
                                   C.c_void_p(_stream(stream)), C.byref(h)))
        self.h = h

    def close(self):
        if getattr(self, "h", None):
            self.lib.t2i_dit_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def cache_state_bytes(self, tokens_per_req: Sequence[int], branches: int) -> int:
        return int(self.lib.t2i_cache_state_bytes(self.cfg.ref(), len(tokens_per_req),
                                                  _arr(C.c_int32, tokens_per_req), branches))

    def new_cache_state(self, tokens_per_req, branches, device="cuda"):
        n = self.cache_state_bytes(tokens_per_req, branches)
        if n == 0:
            raise T2IError(1, "invalid cache state request")
        return torch.zeros(n, dtype=torch.uint8, device=device)


def t2i_dit_init(cfg: Config, weights: Sequence[torch.Tensor], device="cuda", stream=None) -> DiT:
    return DiT(cfg, weights, device, stream)


def t2i_dit_init_static(cfg: Config, weights: Sequence[torch.Tensor], stream=None) -> DiT:
    """A handle on the library's static workspace of the current device (no
    device allocation; calls on such handles must not overlap in time)."""
    return DiT(cfg, weights, stream=stream, static_workspace=True)


# ---------------------------------------------------------------- layer residency

def t2i_dit_block_layout(cfg: Config):
    """(first_index, n_tensors, offsets, block_bytes) of the packed per-block
    weight record (``t2i_dit_block_layout``)."""
    lib = load()
    first, n = C.c_int32(), C.c_int32()
    bb = lib.t2i_dit_block_layout(cfg.ref(), C.byref(first), C.byref(n), None)
    if bb == 0:
        raise T2IError(1, "invalid config")
    offs = (C.c_size_t * n.value)()
    lib.t2i_dit_block_layout(cfg.ref(), C.byref(first), C.byref(n), offs)
    return first.value, n.value, list(offs), int(bb)


def pack_blocks(cfg: Config, weights: Sequence[torch.Tensor]) -> torch.Tensor:
    """The host tier: every block's tensors (weight-table order) copied into a
    page-locked uint8 [depth, block_bytes] buffer at the packed offsets."""
    first, n, offs, bb = t2i_dit_block_layout(cfg)
    depth = cfg.c.depth
    out = torch.zeros((depth, bb), dtype=torch.uint8, pin_memory=True)
    for b in range(depth):
        for j in range(n):
            t = weights[first + b * n + j].contiguous().reshape(-1).view(torch.uint8)
            out[b, offs[j]:offs[j] + t.numel()].copy_(t)
    return out


def t2i_dit_host_tier(m: DiT, host_blocks: torch.Tensor, arena: Optional[torch.Tensor] = None):
    """Register the host tier (pinned, from :func:`pack_blocks`) and the device
    arena blocks load into (allocated here when not given)."""
    if not host_blocks.is_pinned():
        raise T2IError(1, "host_blocks must be page-locked (pin_memory)")
    if arena is None:
        arena = torch.empty(host_blocks.numel(), dtype=torch.uint8, device="cuda")
    check(m.lib.t2i_dit_host_tier(m.h, C.c_void_p(host_blocks.data_ptr()),
                                  C.c_void_p(arena.data_ptr()), arena.numel()), m.h)
    m.host_blocks, m.arena = host_blocks, arena
    return arena


def t2i_dit_evict(m: DiT, keep: int):
    """Evict blocks [keep, depth), last first."""
    check(m.lib.t2i_dit_evict(m.h, int(keep)), m.h)


def t2i_dit_load_async(m: DiT, stream=None) -> int:
    """Queue the loads of every evicted block on ``stream``; returns how many."""
    n = C.c_int32()
    check(m.lib.t2i_dit_load_async(m.h, C.c_void_p(_stream(stream)), C.byref(n)), m.h)
    return n.value


def t2i_first_layers(L: int, t_load: float, t_comp: float) -> int:
    """Resident prefix that hides loading (Eq. 2; see the header)."""
    return int(load().t2i_first_layers(int(L), float(t_load), float(t_comp)))


def t2i_dit_block_state(m: DiT) -> List[int]:
    """Per block: 0 resident, 1 loading, 2 evicted."""
    st = (C.c_int32 * m.cfg.c.depth)()
    check(m.lib.t2i_dit_block_state(m.h, st), m.h)
    return list(st)


def _check_lat(latents: torch.Tensor):
    if latents.dtype != torch.float32 or not latents.is_cuda or not latents.is_contiguous():
        raise T2IError(1, "latents must be a contiguous fp32 device tensor")


def t2i_dit_step(m: DiT, latents: torch.Tensor, lat_hw: Sequence[tuple], t: Sequence[float],
                 prompt_embeds: torch.Tensor, guidance: float = 1.0,
                 t_next: Optional[Sequence[float]] = None,
                 noise_pred: Optional[torch.Tensor] = None, n_blocks: int = -1,
                 hidden_out: Optional[torch.Tensor] = None,
                 skip: Optional[Sequence[int]] = None,
                 cache_state: Optional[torch.Tensor] = None, stream=None,
                 control: Optional[Sequence[tuple]] = None):
    """One model evaluation on packed fp32 ``latents`` (updated in place when
    ``t_next`` is given).  ``prompt_embeds`` is ``[n_req, text_tokens, text_dim]``.

    ``control``: the callback input, a list of ``(block, residual, event)``:
    ``residual`` (fp32 device tensor ``[rows, hidden]``) is added after block
    ``block``; ``event`` (a recorded ``torch.cuda.Event`` or None) is waited for
    on the step's stream only at that point."""
    _check_lat(latents)
    n = len(lat_hw)
    a = _lib.t2i_step_args()
    a.struct_size = C.sizeof(a)
    a.n_req = n
    a.lat_h = _arr(C.c_int32, [h for h, _ in lat_hw])
    a.lat_w = _arr(C.c_int32, [w for _, w in lat_hw])
    a.t = _arr(C.c_double, list(t))
    a.t_next = _arr(C.c_double, list(t_next)) if t_next is not None else None
    a.latents = latents.data_ptr()
    a.prompt_embeds = prompt_embeds.data_ptr()
    a.guidance = guidance
    a.noise_pred = noise_pred.data_ptr() if noise_pred is not None else None
    a.n_blocks = n_blocks
    a.hidden_out = hidden_out.data_ptr() if hidden_out is not None else None
    a.skip = _arr(C.c_uint8, list(skip)) if skip is not None else None
    a.cache_state = cache_state.data_ptr() if cache_state is not None else None
    a.cache_state_bytes = cache_state.numel() if cache_state is not None else 0
    ctl = None
    if control:
        for _, r, _ in control:
            if r.dtype != torch.float32 or not r.is_cuda or not r.is_contiguous():
                raise T2IError(1, "control residuals must be contiguous fp32 device tensors")
        ctl = _lib.t2i_control()
        ctl.struct_size = C.sizeof(ctl)
        ctl.n = len(control)
        ctl.blocks = _arr(C.c_int32, [int(b) for b, _, _ in control])
        ctl.residuals = _arr(C.c_void_p, [r.data_ptr() for _, r, _ in control])
        ctl.ready = _arr(C.c_void_p, [int(ev.cuda_event) if ev is not None else None
                                      for _, _, ev in control])
    a.control_outputs = C.cast(C.byref(ctl), C.c_void_p) if ctl is not None else None
    check(m.lib.t2i_dit_step(m.h, C.byref(a), C.c_void_p(_stream(stream))), m.h)


def lora_merge(W: torch.Tensor, A: torch.Tensor, B: torch.Tensor, alpha: float, stream=None):
    """``W += alpha * B @ A`` in place on the device (``t2i_op_lora_merge``):
    ``W [out, in]``, ``A [rank, in]``, ``B [out, rank]``, one dtype (bf16 or fp32)."""
    for t in (W, A, B):
        if not t.is_cuda or not t.is_contiguous() or t.dtype != W.dtype:
            raise T2IError(1, "W, A, B must be contiguous device tensors of one dtype")
    n_out, n_in = W.shape
    rank = A.shape[0]
    if A.shape != (rank, n_in) or B.shape != (n_out, rank):
        raise T2IError(2, "A must be [rank, in] and B [out, rank]")
    lib = load()
    dt = T2I_BF16 if W.dtype == torch.bfloat16 else T2I_F32
    st = lib.t2i_op_lora_merge(dt, n_out, n_in, rank, float(alpha), W.data_ptr(), n_in,
                               A.data_ptr(), B.data_ptr(), C.c_void_p(_stream(stream)))
    if st != 0:
        raise T2IError(st, lib.t2i_ops_last_error().decode())


def lora_merge_batch(Ws: Sequence[torch.Tensor], As: Sequence[torch.Tensor],
                     Bs: Sequence[torch.Tensor], alpha: float, stream=None):
    """``W_i += alpha * B_i @ A_i`` for weights of one shape and dtype
    (``t2i_op_lora_merge_batch``)."""
    n = len(Ws)
    if n == 0 or len(As) != n or len(Bs) != n:
        raise T2IError(2, "need as many A and B as W (at least one)")
    W0, A0 = Ws[0], As[0]
    n_out, n_in = W0.shape
    rank = A0.shape[0]
    for W, A, B in zip(Ws, As, Bs):
        for t in (W, A, B):
            if not t.is_cuda or not t.is_contiguous() or t.dtype != W0.dtype:
                raise T2IError(1, "W, A, B must be contiguous device tensors of one dtype")
        if W.shape != (n_out, n_in) or A.shape != (rank, n_in) or B.shape != (n_out, rank):
            raise T2IError(2, "every W must be [out, in], A [rank, in], B [out, rank] alike")
    lib = load()
    dt = T2I_BF16 if W0.dtype == torch.bfloat16 else T2I_F32
    ptrs = lambda ts: (C.c_void_p * n)(*[t.data_ptr() for t in ts])
    st = lib.t2i_op_lora_merge_batch(dt, n, n_out, n_in, rank, float(alpha), ptrs(Ws), n_in,
                                     ptrs(As), ptrs(Bs), C.c_void_p(_stream(stream)))
    if st != 0:
        raise T2IError(st, lib.t2i_ops_last_error().decode())


def t2i_cache_check(m: DiT, latents: torch.Tensor, lat_hw, t, step: int, n_steps: int,
                    tau: float, cache_state: torch.Tensor, branches: int = 1,
                    mode: int = T2I_CACHE_ACCUMULATE, stream=None):
    """Cache-skip decision of step ``step``; returns (rel_l1 list, skip list)."""
    _check_lat(latents)
    n = len(lat_hw)
    a = _lib.t2i_cache_args()
    a.struct_size = C.sizeof(a)
    a.n_req = n
    a.lat_h = _arr(C.c_int32, [h for h, _ in lat_hw])
    a.lat_w = _arr(C.c_int32, [w for _, w in lat_hw])
    a.t = _arr(C.c_double, list(t))
    a.latents = latents.data_ptr()
    a.step, a.n_steps, a.tau, a.mode, a.branches = step, n_steps, tau, mode, branches
    a.cache_state = cache_state.data_ptr()
    a.cache_state_bytes = cache_state.numel()
    rel = (C.c_double * n)()
    skip = (C.c_uint8 * n)()
    a.rel_l1 = rel
    a.skip = skip
    check(m.lib.t2i_cache_check(m.h, C.byref(a), C.c_void_p(_stream(stream))), m.h)
    return list(rel), list(skip)


def t2i_dit_sample(m: DiT, latents: torch.Tensor, lat_hw, prompt_embeds: torch.Tensor,
                   n_steps: int, guidance: float = 1.0, timesteps: Optional[np.ndarray] = None,
                   start_step: int = 0, cache_tau: float = 0.0,
                   cache_mode: int = T2I_CACHE_ACCUMULATE,
                   cache_state: Optional[torch.Tensor] = None, stream=None):
    """The denoising loop (latents updated in place).  ``timesteps`` is
    ``[(n_steps+1), n_req]`` float64 or None (uniform from 1 to 0).
    Returns (skip_log, rel_l1_log) as ``[n_steps, n_req]`` numpy arrays."""
    _check_lat(latents)
    n = len(lat_hw)
    a = _lib.t2i_sample_args()
    a.struct_size = C.sizeof(a)
    a.n_req = n
    a.lat_h = _arr(C.c_int32, [h for h, _ in lat_hw])
    a.lat_w = _arr(C.c_int32, [w for _, w in lat_hw])
    a.n_steps, a.start_step = n_steps, start_step
    ts = None
    if timesteps is not None:
        ts = np.ascontiguousarray(timesteps, dtype=np.float64).reshape(n_steps + 1, n)
        a.timesteps = ts.ctypes.data_as(C.POINTER(C.c_double))
    a.latents = latents.data_ptr()
    a.prompt_embeds = prompt_embeds.data_ptr()
    a.guidance = guidance
    a.cache_tau = cache_tau
    a.cache_mode = cache_mode
    a.cache_state = cache_state.data_ptr() if cache_state is not None else None
    a.cache_state_bytes = cache_state.numel() if cache_state is not None else 0
    skip_log = np.zeros((n_steps, n), dtype=np.uint8)
    rel_log = np.zeros((n_steps, n), dtype=np.float64)
    a.skip_log = skip_log.ctypes.data_as(C.POINTER(C.c_uint8))
    a.rel_l1_log = rel_log.ctypes.data_as(C.POINTER(C.c_double))
    check(m.lib.t2i_dit_sample(m.h, C.byref(a), C.c_void_p(_stream(stream))), m.h)
    return skip_log, rel_log
