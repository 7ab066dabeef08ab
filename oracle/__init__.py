"""Plain CPU oracle of the DiT denoising step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import anything from this package.  The product path (the
HIP library and its Python binding) never does, and this package never imports
the product.  The two share nothing but the seeded input generators in
``synth``.

What it computes (ServerlessT2I, Sec. 2.1 and Sec. 4, Fig. "workflow
definition"): the base diffusion model evaluated once per denoising step on a
latent under text conditioning, the ``denoise`` update between steps, and the
step-to-step cache-skip rule.  The paper fixes the role of these pieces (a bf16
diffusion transformer called on ``latents`` and ``prompt_embeds`` returning
``noise_pred``; an iterative loop) but no architectural constant, so every
convention below is a stated reading of it.

Everything is float64 numpy, one request (one sequence) at a time, written as
the definitions read: no blocking, no fusion, no reordering.

Modules:
  dit      cross-attention DiT forward (patch embed, adaLN-Zero blocks with
           self- and cross-attention, final layer)
  mmdit    joint-attention (MMDiT-style) blocks with 2D RoPE
  sampler  classifier-free guidance, Euler update, schedules, cache rule and
           the sampling loop
  lora     weight-update adapter merge W + alpha B A
  sched    the vTime two-layer fair scheduler (control plane)
  loading  the load/compute pipeline of first-layers caching (Eq. 1-2)
"""
from . import dit, sampler, mmdit, lora, sched, loading  # noqa: F401
