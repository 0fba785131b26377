"""The allocation-free n-gram entry point (static device scratch) against attt_ngram_weights
(caller workspace): two calls in a row on one GPU, the second with a smaller input, so counts
left in the shared scratch by the first call would show in the second. f and w must be
bit-identical to the workspace entry point's, and to the oracle's on the smaller input."""
import numpy as np
import pytest

from gpu_util import dev_i32, host, note
from oracle import ngram as ongram
from workloads import Workload

pytestmark = pytest.mark.gpu


def _both(attt, tok, n, w_min):
    args = (dev_i32(tok["hist_flat"]), tok["hist_off"], dev_i32(tok["tok_flat"]), tok["tok_off"])
    fw, ww = attt.ngram_weights(*args, n=n, w_min=w_min)
    fs, ws = attt.ngram_weights_noalloc(*args, n=n, w_min=w_min)
    return (host(fw).view(np.uint32), host(ww).view(np.uint32)), (host(fs).view(np.uint32), host(ws).view(np.uint32))


def test_noalloc_matches_workspace_entry_point_twice(attt):
    big, small = Workload("c5"), Workload("c2")
    for wl in (big, small):
        cfg = wl.cfg
        tok = wl.tokens()
        need = attt.ngram_workspace_size(tok["hist_off"], tok["tok_off"], cfg.n)
        note(f"noalloc ngram {cfg.key}: {cfg.episodes} episodes, {need} bytes of scratch")
        (fw, ww), (fs, ws) = _both(attt, tok, cfg.n, cfg.w_min)
        assert np.array_equal(fw, fs) and np.array_equal(ww, ws)
    fo, wo = ongram.ngram_weights(small.tokens()["history"], small.tokens()["updates"], small.cfg.n,
                                  small.cfg.w_min)
    assert np.array_equal(fs, fo) and np.array_equal(ws, wo.view(np.uint32))


def test_noalloc_rejects_beyond_scratch(attt):
    E = 64
    hoff = np.arange(E + 1, dtype=np.int64) * 3000
    toff = np.arange(E + 1, dtype=np.int64) * 40 * 4096
    import torch
    h = torch.zeros(int(hoff[-1]), dtype=torch.int32, device="cuda")
    x = torch.zeros(int(toff[-1]), dtype=torch.int32, device="cuda")
    with pytest.raises(attt.AtttError) as e:
        attt.ngram_weights_noalloc(h, hoff, x, toff, n=3)
    assert e.value.status == 3
