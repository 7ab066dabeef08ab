"""Helpers shared by the GPU parity tests (not a test module)."""
import sys
import time

import numpy as np
import torch

import synth
import paper_2607_26566_amd as t2i
from oracle import dit, mmdit

DEV = "cuda"


def rel_l2(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(got - ref) / np.linalg.norm(ref))


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


def to_dev(a, dtype):
    """numpy float32 (bf16-representable for bf16) -> device tensor."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(DEV).to(torch.bfloat16 if dtype == "bf16" else torch.float32).contiguous()


def to_host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


class Model:
    """A workload's weights on host (for the oracle) and device (for the HIP path)."""

    def __init__(self, w, max_tokens=None, max_requests=None, max_steps=None, weights=None):
        t0 = time.time()
        self.w = w
        self.cfg = t2i.Config.from_shape(w, max_tokens, max_requests, max_steps)
        self.om = mmdit if w.arch == "mmdit" else dit   # the oracle module of this family
        table = t2i.weight_table(self.cfg)
        assert table == [(n, tuple(s)) for n, s in self.om.weight_layout(w)]
        self.host = weights if weights is not None else synth.weights(w, table)
        self.dev = [to_dev(a, w.dtype) for a in self.host]
        self.m = t2i.t2i_dit_init(self.cfg, self.dev)
        self._W = None
        say(f"model {w.name} ready in {time.time() - t0:.1f}s")

    @property
    def W(self):
        if self._W is None:
            self._W = self.om.as_dict(self.w, self.host)
        return self._W

    def latents_dev(self, lats):
        return torch.from_numpy(np.concatenate([np.ravel(l) for l in lats]).astype(np.float32)).to(DEV)

    def text_dev(self, texts):
        return to_dev(np.stack(texts), self.w.dtype)

    def split(self, flat, shapes):
        out, off = [], 0
        flat = np.asarray(flat)
        for s in shapes:
            n = int(np.prod(s))
            out.append(flat[off:off + n].reshape(s))
            off += n
        return out
