"""The handle without a caller workspace (t2i_dit_init_static: the library's
static device array) against a handle with one (t2i_dit_init), through the C
ABI: identical outputs, bitwise, on two calls in a row -- the second with a
smaller input, so that it runs on the array the first call left behind."""
import gc

import numpy as np
import pytest
import torch

import synth
import paper_2607_26566_amd as t2i
from gpu_common import DEV, say, to_dev

pytestmark = pytest.mark.gpu


def _step(m, w, lats, texts, hw, ts, tn):
    x = torch.from_numpy(np.concatenate([l.ravel() for l in lats]).astype(np.float32)).to(DEV)
    tx = to_dev(np.stack(texts), w.dtype)
    v = torch.zeros_like(x)
    rows = sum((h // w.patch) * (ww // w.patch) for h, ww in hw) * w.branches
    hid = torch.zeros((rows, w.hidden), dtype=torch.float32, device=DEV)
    t2i.t2i_dit_step(m, x, hw, ts, tx, guidance=w.guidance, t_next=tn, noise_pred=v,
                     hidden_out=hid)
    torch.cuda.synchronize()
    return [a.cpu().numpy() for a in (v, x, hid)]


@pytest.mark.parametrize("name,kw", [
    ("dit1024_cfg", dict(depth=2, requests=((32, 32), (16, 32)))),
    ("tiny_f32", dict(requests=((16, 16), (16, 8)))),
])
def test_static_workspace_handle_equals_allocated(name, kw):
    w = synth.reduced(synth.workload(name), **kw)
    cfg = t2i.Config.from_shape(w)
    table = t2i.weight_table(cfg)
    dev = t2i.upload(synth.weights(w, table), w.dtype)
    ref = t2i.t2i_dit_init(cfg, dev)
    sta = t2i.t2i_dit_init_static(cfg, dev)
    assert sta.workspace is None
    lats, texts = synth.latents(w), synth.texts(w)
    hw = list(w.requests)
    # call 1: every request; call 2: the smaller request alone
    for call, (idx, ts, tn) in enumerate((([0, 1], [0.9, 0.4], [0.85, 0.35]),
                                          ([1], [0.6], [0.55]))):
        args = ([lats[i] for i in idx], [texts[i] for i in idx], [hw[i] for i in idx], ts, tn)
        a = _step(ref, w, *args)
        b = _step(sta, w, *args)
        for x, y, what in zip(a, b, ("noise_pred", "latents", "hidden")):
            assert np.array_equal(x, y), (name, call, what)
        say(f"static workspace {name} call {call}: {len(idx)} request(s) bitwise equal")
    ref.close()
    sta.close()
    del ref, sta, dev
    gc.collect()
    torch.cuda.empty_cache()
