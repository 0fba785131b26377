"""Bitwise stability of every kernel family when its inputs are uploaded afresh before each call,
into device memory that other kernels have just used, with calls of the other families in
between (the n-gram weights at the 16-episode stress shape, the LoRA gradient at the Llama-8B
shape, the attention block's backward, the bf16 CE forward and backward, the serving forward).
Repeated calls on inputs that stay in place can hide a race whose outcome depends on where and
how recently data sat in the caches; these must give the first call's bits every time."""
import hashlib

import numpy as np
import pytest

from gpu_util import dev_dense, dev_f32, dev_i32, note
from workloads import Workload, random_dense

pytestmark = pytest.mark.gpu


def _bits(*ts):
    import torch
    h = hashlib.sha1()
    for t in ts:
        v = t.contiguous().view(torch.int16) if t.dtype == torch.bfloat16 else t.contiguous().view(torch.uint8)
        h.update(v.cpu().numpy().tobytes())
    return h.hexdigest()


def test_families_stable_under_recycled_memory(attt):
    import torch
    wl5 = Workload("c5")
    tok5, cfg5 = wl5.tokens(), wl5.cfg
    probs = Workload("c3").lora()
    att = [random_dense((2048, h, 128), s, True, 50 + i) for i, (h, s) in enumerate([(16, 1.0), (4, 1.0), (4, 1.0),
                                                                                    (16, 0.05)])]
    aoff = np.array([0, 700, 2048], np.int64)
    ce2 = Workload("c2").ce()
    cew = np.full(len(ce2["labels"]), 0.7, np.float32)
    sx = random_dense((2048, 4096), 1.0, True, 60)
    serve = [dict(y=random_dense((2048, o), 1.0, True, 61 + i), A=random_dense((16, 4096), 0.05, True, 70 + i),
                  B=random_dense((o, 16), 0.05, True, 80 + i)) for i, o in enumerate((4096, 1024, 1024))]

    def ngram():
        return _bits(*attt.ngram_weights(dev_i32(tok5["hist_flat"]), tok5["hist_off"], dev_i32(tok5["tok_flat"]),
                                         tok5["tok_off"], n=cfg5.n, w_min=cfg5.w_min))

    def lora():
        xs, dev = {}, []
        for p in probs:
            if id(p["x"]) not in xs:
                xs[id(p["x"])] = dev_dense(p["x"])
            r = p["rank"]
            dev.append(dict(x=xs[id(p["x"])], dy=dev_dense(p["dy"]), A=dev_dense(p["A"]), B=dev_dense(p["B"]),
                            scale=p["scale"], dA=torch.zeros(r, p["d_in"], dtype=torch.float32, device="cuda"),
                            dB=torch.zeros(p["d_out"], r, dtype=torch.float32, device="cuda")))
        attt.lora_grad(dev)
        return _bits(*[q["dA"] for q in dev], *[q["dB"] for q in dev])

    def attention():
        return _bits(*attt.attention_bwd(*[dev_dense(t) for t in att], row_offsets=aoff))

    def ce():
        return _bits(*attt.weighted_ce_fwd_bwd(dev_dense(ce2["h"]), dev_dense(ce2["W"]), dev_i32(ce2["labels"]),
                                               dev_f32(cew), row_offsets=ce2["row_offsets"]))

    def serving():
        x = dev_dense(sx)
        calls = [dict(x=x, y=dev_dense(p["y"]), A=dev_dense(p["A"]), B=dev_dense(p["B"]), scale=1.0) for p in serve]
        attt.lora_forward(calls)
        return _bits(*[c["y"] for c in calls])

    fams = [("ngram", ngram), ("lora", lora), ("attention", attention), ("ce", ce), ("serving", serving)]
    note("recycled-memory stability: 5 families x 40 calls, rotating order")
    first, bad = {}, []
    for it in range(40):
        for name, fn in fams[it % 5:] + fams[:it % 5]:
            h = fn()
            if name not in first:
                first[name] = h
            elif h != first[name]:
                bad.append((it, name))
    assert not bad, bad
