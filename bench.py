#!/usr/bin/env python3
"""Denoising steps/s of the 1024-px DiT with classifier-free guidance on one MI355X.

One "step" is one complete model-function call (ServerlessT2I Sec. 4): the
stateless ``t2i_dit_step`` on 2 x 4096 image tokens (conditional + unconditional
branch) -- timestep embedding, every block's adaLN modulation, text projection
and cross K/V, patch embedding, 28 blocks (LN-mod, QKV, self-attention, gated
out-projection, cross-attention, MLP), final layer, guidance and the Euler
update -- on synthetic inputs already resident in HBM.

Prints ONE JSON line.  ``roofline`` is for the kernel with the largest share of
step time, timed with HIP events on the library's stream during the timed
steps; ``cpu_baseline`` is the oracle on the host cores on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
WORKLOAD = "dit1024_cfg"


def class_work(w):
    """Algorithmic work of one launch of each kernel class at workload ``w``
    (FLOPs = 2MNK per GEMM and 4 Nq Nk d per attention head; bytes for the
    HBM-bound LN-mod: read fp32 x, write bf16 h)."""
    R = w.image_tokens * w.branches
    D, F = w.hidden, w.mlp_hidden
    seq = [w.tokens(r) for r in range(w.n_req)] * w.branches
    dh = w.heads * w.head_dim
    return {
        "gemm_qkv": ("flop", 2.0 * R * 3 * D * D),
        "attn_self": ("flop", sum(4.0 * n * n * dh for n in seq)),
        "gemm_o": ("flop", 2.0 * R * D * D),
        "gemm_xq": ("flop", 2.0 * R * D * D),
        "attn_cross": ("flop", sum(4.0 * n * w.text_tokens * dh for n in seq)),
        "gemm_xo": ("flop", 2.0 * R * D * D),
        "ln_mod": ("byte", R * D * (4.0 + 2.0)),
        "gemm_fc1": ("flop", 2.0 * R * F * D),
        "gemm_fc2": ("flop", 2.0 * R * F * D),
    }


def step_flops(w):
    cw = class_work(w)
    per_block = sum(v for k, (kind, v) in cw.items() if kind == "flop")
    return per_block * w.depth


def cpu_baseline(w, host_prefix, n_blocks=1):
    """The oracle on a bounded sample: blocks 0..n_blocks-1 of one 1024-px
    step for both guidance branches, scaled to a whole step."""
    import numpy as np
    import synth
    from oracle import dit
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count()
    wp = synth.reduced(w, depth=n_blocks)
    W = dit.as_dict(wp, host_prefix)
    lat, text = synth.latents(w)[0], synth.texts(w)[0]
    t0 = time.perf_counter()
    c = dit.conditioning(W, wp, 1.0)
    x0 = dit.embed(W, wp, lat)
    for txt in (text, np.zeros((w.text_tokens, w.text_dim))):
        y = dit.text_project(W, wp, txt)
        dit.run_blocks(W, wp, x0, y, c)
    dt = time.perf_counter() - t0
    per_step = dt * w.depth / n_blocks
    return {"value": 1.0 / per_step, "unit": "steps/s", "cores": int(cores), "kind": "oracle",
            "sample": f"float64 numpy oracle, blocks 0-{n_blocks - 1} of one 1024px step for both "
                      f"guidance branches (2x4096 tokens) in {dt:.1f} s, scaled x{w.depth / n_blocks:g} "
                      f"to all {w.depth} blocks"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain 1 GiB device copy (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the denoising step "
              "is not sharded across GPUs in this build", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import synth
    import paper_2607_26566_amd as t2i
    from paper_2607_26566_amd import _lib

    if args.copy_calibration:
        n = 1 << 28                      # 2^28 floats = 1 GiB
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "launches": 5}))
        return

    w = synth.workload(WORKLOAD)
    cfg = t2i.Config.from_shape(w)
    table = t2i.weight_table(cfg)
    host = synth.weights(w, table)
    dev = t2i.upload(host, w.dtype)
    m = t2i.t2i_dit_init(cfg, dev)
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    x = torch.from_numpy(np.concatenate([l.ravel() for l in lats])).cuda()
    tx = torch.from_numpy(np.stack(texts)).to("cuda", torch.bfloat16)
    n = w.steps
    sched = [1.0 - k / n for k in range(n + 1)]

    def run(i):
        k = i % n
        t2i.t2i_dit_step(m, x, hw, [sched[k]], tx, guidance=w.guidance, t_next=[sched[k + 1]])

    lib = t2i.load()
    # warmup; the last warmup pass times every kernel class to find the dominant one
    for i in range(max(args.warmup - 1, 0)):
        run(i)
    _lib.check(lib.t2i_dit_profile(m.h, (1 << len(_lib.KERNEL_CLASSES)) - 1), m.h)
    run(0)
    per_class = {}
    for ci, name in enumerate(_lib.KERNEL_CLASSES):
        tot, cnt = C_double(), C_int64()
        _lib.check(lib.t2i_dit_profile_read(m.h, ci, byref(tot), byref(cnt)), m.h)
        per_class[name] = (tot.value, cnt.value)
    dominant = max(per_class, key=lambda k: per_class[k][0])
    dom_idx = _lib.KERNEL_CLASSES.index(dominant)

    # timed region: events only around the dominant kernel class
    _lib.check(lib.t2i_dit_profile(m.h, 1 << dom_idx), m.h)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        run(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    tot, cnt = C_double(), C_int64()
    _lib.check(lib.t2i_dit_profile_read(m.h, dom_idx, byref(tot), byref(cnt)), m.h)
    _lib.check(lib.t2i_dit_profile(m.h, 0), m.h)
    dom_avg_s = tot.value / 1e3 / max(cnt.value, 1)

    ms = elapsed * 1e3 / args.steps
    sps = args.steps / elapsed
    flops = step_flops(w)
    cw = class_work(w)
    kind, work = cw[dominant]
    if kind == "flop":
        ach = work / dom_avg_s / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4), "traffic": None}
    else:
        ach = work / dom_avg_s / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None}
    roof["kernel"] = dominant
    roof["avg_launch_ms"] = round(dom_avg_s * 1e3, 4)
    roof["launches"] = int(cnt.value)
    roof["work_per_launch"] = work

    kernel_ms = {k: round(v[0] / max(v[1], 1), 4) for k, v in per_class.items()}
    ln_bytes = cw["ln_mod"][1]
    ln_ms = kernel_ms["ln_mod"]
    gemm_attn_ms = sum(v[0] for k, v in per_class.items() if cw[k][0] == "flop")

    # a whole 20-step sample (conditioning and text computed once per sample)
    x.copy_(torch.from_numpy(np.concatenate([l.ravel() for l in lats])).cuda())
    torch.cuda.synchronize()
    ts = time.perf_counter()
    t2i.t2i_dit_sample(m, x, hw, tx, n, guidance=w.guidance)
    torch.cuda.synchronize()
    sample_s = time.perf_counter() - ts

    out = {
        "metric": "denoising steps/s at 1024px DiT (CFG, 2x4096 tokens)",
        "value": round(sps, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "dit1024_cfg: 1024px image, latent 4x128x128, patch 2 -> 4096 "
                               "tokens x 2 guidance branches (g=4.5), hidden 1152, 28 blocks, "
                               "16 heads x 72, MLP 4608, 120 text tokens x 4096, seed 2",
                   "global_batch": 2, "seq_len": 4096, "parallelism": "none (1 GPU)"},
        "roofline": roof,
        "gemm_attn_tflops_step": round(flops * sps / 1e12, 1),
        "gemm_attn_frac_of_peak_step": round(flops * sps / 1e12 / PEAK_BF16_TFLOPS, 4),
        "gemm_attn_tflops_kernels": round(flops / (gemm_attn_ms / 1e3) / 1e12, 1),
        "ln_mod_gbs": round(ln_bytes / (ln_ms / 1e3) / 1e9, 1) if ln_ms > 0 else None,
        "images_per_s": round(1.0 / sample_s, 3),
        "sample_steps_per_s": round(n / sample_s, 3),
        "kernel_avg_ms": kernel_ms,
        "flops_per_step": flops,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, host[:8 + 16] + host[-4:])
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    from ctypes import c_double as C_double, c_int64 as C_int64, byref
    main()
