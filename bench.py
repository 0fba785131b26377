"""Throughput of the aTTT in-episode update step on one MI355X.

One step = the whole hot path over one batch of synthetic inputs resident in HBM:
  1. n-gram exposure and weights of the update tokens against the episode history (Eq. 8-9)
  2. token-weighted CE through the LM head, loss and dL/dh (Eq. 10)
  3. LoRA dA / dB of q, k, v, o; the o projection takes dL/dh as its upstream gradient
all through the C ABI on one stream. Default workload: the Llama-8B-shaped bf16 step
(8192 update tokens, 32 previous updates of 4096 tokens, n = 4, d = 4096, V = 128256,
rank-16 LoRA on q/k/v/o 4096x4096 / 4096x1024).

Prints one JSON line: update tokens/s, the roofline of the dominant kernel (per-launch
durations from HIP events recorded on the launch stream inside the timed region), and
the CPU oracle timed on a bounded sample on this host.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

METRIC = "aTTT update tokens/s (weights+weighted CE+LoRA grad); %MFMA and %HBM peak"
PEAK_BF16 = 2.5e15       # dense bf16 MFMA, FLOP/s
PEAK_F32_MFMA = 157.3e12
PEAK_HBM = 8.0e12        # bytes/s


# The paper's only timing figures are system-level wall clock of whole agent runs (Table
# "tab:throughput"): context for this step's cost, not a target, on hardware the paper does not
# name (its serving runs vLLM with runtime LoRA and trains on dedicated GPUs).
PAPER_CONTEXT = {
    "source": "Table tab:throughput (Sec. 4 and App. A)",
    "workload": "140 ALFWorld episodes, Qwen3.5-9B, 16 episodes concurrent",
    "no_ttt_min": 14.6, "concurrent_attt_min": 28.3, "sequential_attt_min": 186.0,
    "concurrent_attt_vs_no_ttt": 1.9, "hardware": "not stated", "precision": "not stated",
}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c3", help="workload key c1..c5 (default: Llama-8B shape)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=5120,
                    help="CE rows the oracle sample covers (about 10 s of float64 work at the Llama-8B shape)")
    ap.add_argument("--hbm-calibrate", action="store_true",
                    help="only run a plain 1 GiB device copy, 4 times: the reference for scaling "
                         "FETCH_SIZE / WRITE_SIZE counter readings to bytes")
    return ap.parse_args()


def hbm_calibrate():
    import torch
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration_copy_bytes": n, "copies": 4}), flush=True)


class Step:
    """Device-resident inputs, outputs and workspaces of one update step."""

    def __init__(self, wl, attt, torch):
        from gpu_util import dev_dense, dev_i32
        cfg = wl.cfg
        self.cfg, self.attt, self.torch = cfg, attt, torch
        t0 = time.time()
        tok, ce, probs = wl.tokens(), wl.ce(), wl.lora()
        log(f"inputs generated on host in {time.time() - t0:.1f}s")
        self.tok = tok
        self.hist = dev_i32(tok["hist_flat"])
        self.toks = dev_i32(tok["tok_flat"])
        self.h = dev_dense(ce["h"])
        self.W = dev_dense(ce["W"])
        self.labels = dev_i32(ce["labels"])
        self.row_off = ce["row_offsets"]
        T = int(tok["tok_off"][-1])
        dev = self.h.device
        self.f = torch.empty(T, dtype=torch.int32, device=dev)
        self.w = torch.empty(T, dtype=torch.float32, device=dev)
        E = cfg.episodes
        self.loss = torch.empty(E, dtype=torch.float32, device=dev)
        self.lse = torch.empty(T, dtype=torch.float32, device=dev)
        self.dH = torch.empty_like(self.h)
        xs = {}
        self.problems = []
        off = self.row_off
        for p in probs:
            key = id(p["x"])
            if key not in xs:
                xs[key] = dev_dense(p["x"])
            e = p["episode"]
            chained = p["name"].endswith(".o")
            dy = self.dH[int(off[e]):int(off[e + 1])] if chained else dev_dense(p["dy"])
            r = p["rank"]
            self.problems.append(dict(x=xs[key], dy=dy, A=dev_dense(p["A"]), B=dev_dense(p["B"]),
                                      scale=p["scale"],
                                      dA=torch.zeros(r, p["d_in"], dtype=torch.float32, device=dev),
                                      dB=torch.zeros(p["d_out"], r, dtype=torch.float32, device=dev)))
        self.probs_host = probs
        dt = attt.BF16 if cfg.dtype == "bf16" else attt.F32
        u8 = torch.uint8
        self.ws_ngram = torch.empty(attt.ngram_workspace_size(tok["hist_off"], tok["tok_off"], cfg.n), dtype=u8, device=dev)
        # The LM head is frozen (only the episode's adapter trains), so its transposed copy for
        # the bf16 backward is built once per model, outside the step (parts.head_transpose_once).
        self.W_t = None
        if dt == attt.BF16:
            self.W_t = attt.ce_head_transpose(self.W)
            torch.cuda.synchronize()
        self.ws_ce = torch.empty(attt.ce_workspace_size(T, cfg.d, cfg.vocab, dt, head_t=self.W_t is not None),
                                 dtype=u8, device=dev)
        self.ws_lora = torch.empty(attt.lora_workspace_size(self.problems, dt), dtype=u8, device=dev)
        log(f"workspaces: ngram {self.ws_ngram.numel() / 2**20:.1f} MiB, ce {self.ws_ce.numel() / 2**20:.1f} MiB, "
            f"lora {self.ws_lora.numel() / 2**20:.1f} MiB")

    def run(self):
        a, cfg = self.attt, self.cfg
        a.ngram_weights(self.hist, self.tok["hist_off"], self.toks, self.tok["tok_off"], n=cfg.n,
                        w_min=cfg.w_min, workspace=self.ws_ngram, out=(self.f, self.w))
        a.weighted_ce_fwd_bwd(self.h, self.W, self.labels, self.w, row_offsets=self.row_off,
                              workspace=self.ws_ce, out=(self.loss, self.lse, self.dH), lm_head_t=self.W_t)
        a.lora_grad(self.problems, workspace=self.ws_lora)


def algorithmic(cfg, tok, probs):
    """Algorithmic work per step of each part (what the method needs, not what a design
    executes): flops of the contractions and compulsory HBM bytes."""
    N, d, V = cfg.rows, cfg.d, cfg.vocab
    esz = 2 if cfg.dtype == "bf16" else 4
    H = int(tok["hist_off"][-1])
    ngram_bytes = 4 * H + 4 * N + 8 * N          # read history and tokens, write f and w
    lora_bytes, lora_flops, seen = 0, 0, set()
    for p in probs:
        if id(p["x"]) not in seen:
            seen.add(id(p["x"]))
            lora_bytes += p["x"].f32.size * esz
        r, di, do, rows = p["rank"], p["d_in"], p["d_out"], p["rows"]
        lora_bytes += rows * do * esz + (r * di + do * r) * esz + 2 * 4 * (r * di + do * r)
        lora_flops += 4 * rows * r * (di + do)
    return dict(ce_flops_fwd=2.0 * N * V * d, ce_flops_bwd=2.0 * N * V * d,
                ngram_bytes=float(ngram_bytes), lora_bytes=float(lora_bytes), lora_flops=float(lora_flops))


# the fused backward's label pass runs as ce_fused_bwd_kernel, or as its vocabulary-split form
# when d has fewer than 16 slices of 256
KERNEL_SYMBOL = {"ce_fwd_lse": ("attt::ce_fwd_",), "ce_bwd_dz": ("attt::ce_dz_",), "ce_bwd_dh": ("attt::ce_dh_",),
                 "ce_fused_bwd": ("attt::ce_fused_bwd_kernel<true>", "attt::ce_fused_bwd_split_kernel<true>")}


def counter_traffic(workload, kernel):
    """HBM bytes per dispatch of `kernel` from the committed rocprofv3 counter summary of this
    workload, or None when there is none or the kernel sources changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{workload}_kernels_hbm.md")
    if not os.path.exists(path):
        return None
    rec = None
    for line in open(path):
        if line.startswith("traffic-json: "):
            rec = json.loads(line[len("traffic-json: "):])
    if rec is None:
        return None
    for src, digest in rec["sources"].items():
        with open(os.path.join(ROOT, src), "rb") as fh:
            if hashlib.sha256(fh.read()).hexdigest()[:16] != digest:
                return None
    prefixes = KERNEL_SYMBOL.get(kernel, ())
    for name, b in rec["bytes_per_dispatch"].items():
        if any(name.removeprefix("void ").startswith(pre) for pre in prefixes):
            return b
    return None


def cpu_baseline(wl, rows):
    """The oracle as it stands on this host: full n-gram and LoRA parts, the CE part on the
    first `rows` update rows (rows are independent) scaled to all rows."""
    from oracle import ce as oce
    from oracle import lora as olora
    from oracle import ngram as ongram
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    cfg = wl.cfg
    tok, ce, probs = wl.tokens(), wl.ce(), wl.lora()
    N = cfg.rows
    t = time.perf_counter()
    f, w = ongram.ngram_weights(tok["history"], tok["updates"], cfg.n, cfg.w_min)
    t_ng = time.perf_counter() - t
    t = time.perf_counter()
    W64 = np.asarray(ce["W"].f32, np.float64)
    t_conv = time.perf_counter() - t
    rows = min(rows, N)
    t = time.perf_counter()
    oce.ce_rows(ce["h"].f32, W64, ce["labels"], w, ce["row_offsets"], np.arange(rows))
    t_rows = time.perf_counter() - t
    del W64
    t = time.perf_counter()
    for p in probs:
        olora.lora_grad(p["x"].f32, p["dy"].f32, p["A"].f32, p["B"].f32, p["scale"])
    t_lora = time.perf_counter() - t
    t_ce = t_conv + t_rows * N / rows
    total = t_ng + t_ce + t_lora
    return {"value": N / total, "unit": "update tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"float64 numpy oracle: n-gram weights and LoRA grads in full, CE fwd+bwd on "
                       f"{rows} of {N} rows scaled by {N / rows:.0f} (rows are independent); "
                       f"ngram {t_ng:.2f}s, ce {t_ce:.1f}s est, lora {t_lora:.2f}s")}


def ngram_set_part(wl, attt, torch, reps):
    """The persistent-set alternative for the n-gram rows (the history update of Algorithm 1),
    outside the timed step: per update, one append of that update's text to every episode's
    set (measured while the sets are built from the previous updates, one call per update)
    and one weights query of the new update (over `reps` calls). Times are the kernels' own,
    from the library's launch events; the calls are queued behind a GPU spin so that host call
    overhead between small calls is excluded."""
    from gpu_util import dev_i32
    cfg, tok = wl.cfg, wl.tokens()
    E = cfg.episodes
    capacity = int(max(np.diff(tok["hist_off"]))) + cfg.update_len
    nbytes = attt.ngram_set_size(capacity, cfg.n)
    sets = [torch.empty(nbytes, dtype=torch.uint8, device="cuda") for _ in range(E)]
    attt.ngram_set_init(sets, capacity, cfg.n)
    torch.cuda.synchronize()
    texts_per_update = []
    for i in range(cfg.prior_updates):
        texts = [h[i * cfg.prior_len:(i + 1) * cfg.prior_len] for h in tok["history"]]
        off = np.zeros(E + 1, np.int64)
        off[1:] = np.cumsum([len(t) for t in texts])
        texts_per_update.append((dev_i32(np.concatenate(texts)), off))
    attt.timing_enable(True)
    attt.timing_reset()
    gpu_hold(torch, len(texts_per_update))
    for flat, off in texts_per_update:
        attt.ngram_set_append(sets, flat, off, capacity, cfg.n)
    torch.cuda.synchronize()
    app_ms, app_n = attt.timing_read("ngram_set")
    toks = dev_i32(tok["tok_flat"])
    f = torch.empty(len(tok["tok_flat"]), dtype=torch.int32, device="cuda")
    w = torch.empty(len(tok["tok_flat"]), dtype=torch.float32, device="cuda")
    gpu_hold(torch, reps)
    for _ in range(reps):
        attt.ngram_set_weights(sets, toks, tok["tok_off"], capacity, cfg.n, cfg.w_min, out=(f, w))
    torch.cuda.synchronize()
    q_ms, q_n = attt.timing_read("ngram_set_weight")
    attt.timing_enable(False)
    append = app_ms / max(1, app_n)
    query = q_ms / max(1, q_n)
    return {"query_ms": query, "append_ms": append, "ms": query + append,
            "set_bytes_per_episode": nbytes, "capacity": capacity}


def repetition_part(wl, attt, torch, reps):
    """The paper's sequence-level baseline (Eq. 6-7, tau = 0.5), outside the timed step: rho, nu
    and the skip decision of every episode's update against each previous update of its history
    (token ids as word ids). Times are the kernels' own (launch events), queued behind a GPU
    spin; bytes are the words read once."""
    from gpu_util import dev_i32
    cfg, tok = wl.cfg, wl.tokens()
    texts = []
    for e in range(cfg.episodes):
        h = tok["history"][e]
        texts += [h[i * cfg.prior_len:(i + 1) * cfg.prior_len] for i in range(cfg.prior_updates)]
        texts.append(tok["updates"][e])
    toff = np.zeros(len(texts) + 1, np.int64)
    toff[1:] = np.cumsum([len(t) for t in texts])
    etx = np.arange(cfg.episodes + 1, dtype=np.int64) * (cfg.prior_updates + 1)
    words = dev_i32(np.concatenate(texts))
    toff_d = torch.from_numpy(toff).cuda()
    ws = torch.empty(attt.repetition_workspace_size(toff, etx), dtype=torch.uint8, device="cuda")
    attt.update_repetition(words, toff, etx, text_offsets_dev=toff_d, workspace=ws)
    torch.cuda.synchronize()
    attt.timing_enable(True)
    attt.timing_reset()
    gpu_hold(torch, reps)
    for _ in range(reps):
        rho, nu, skip, best, _ = attt.update_repetition(words, toff, etx, text_offsets_dev=toff_d, workspace=ws)
    torch.cuda.synchronize()
    c_ms, c_n = attt.timing_read("rep_count")
    r_ms, r_n = attt.timing_read("rep_reduce")
    attt.timing_enable(False)
    ms = c_ms / max(1, reps) + r_ms / max(1, reps)
    nbytes = 4.0 * float(toff[-1])
    return {"ms": ms, "count_ms": c_ms / max(1, reps), "reduce_ms": r_ms / max(1, reps),
            "texts": len(texts), "words": int(toff[-1]), "algorithmic_gbs": nbytes / (ms * 1e-3) / 1e9,
            "frac_of_hbm_peak": nbytes / (ms * 1e-3) / PEAK_HBM,
            "skipped_updates": int(skip.sum().item()), "mean_rho": float(rho.mean().item())}


def attention_part(wl, attt, torch, reps):
    """The adapted attention block's backward at the workload's shape (dY_q, dY_k, dY_v: the
    LoRA gradient's upstream gradients), outside the timed step: one call per episode batch
    of the update rows, heads = d / 128, key/value heads from the k projection. Synthetic bf16
    inputs. Algorithmic flops: the causal forward (QK^T and PV) plus the backward at 2.5x the
    forward, 7 N^2/2-sized products of 2 dh flops per (query, key, head)."""
    from workloads.gen import random_dense
    from gpu_util import dev_dense
    cfg = wl.cfg
    kproj = [p for p in cfg.projections if p.name == "k"]
    if not kproj or cfg.d % 128 or cfg.dtype != "bf16":
        return None
    H, Hkv = cfg.d // 128, kproj[0].d_out // 128
    N = cfg.rows
    off = np.arange(cfg.episodes + 1, dtype=np.int64) * cfg.update_len
    q = dev_dense(random_dense((N, H, 128), 1.0, True, 901))
    k = dev_dense(random_dense((N, Hkv, 128), 1.0, True, 902))
    v = dev_dense(random_dense((N, Hkv, 128), 1.0, True, 903))
    do = dev_dense(random_dense((N, H, 128), 0.05, True, 904))
    out = attt.attention_bwd(q, k, v, do, row_offsets=off)
    torch.cuda.synchronize()
    attt.timing_enable(True)
    attt.timing_reset()
    gpu_hold(torch, reps)
    for _ in range(reps):
        attt.attention_bwd(q, k, v, do, row_offsets=off, out=out)
    torch.cuda.synchronize()
    times = {n: attt.timing_read(n)[0] / reps for n in ("attn_fwd_stats", "attn_dkdv", "attn_dq")}
    attt.timing_enable(False)
    ms = sum(times.values())
    L = cfg.update_len
    pairs = cfg.episodes * L * (L + 1) / 2.0  # causal (query, key) pairs per head
    flops = 7.0 * 2.0 * 128 * pairs * H
    return {"ms": ms, **{k + "_ms": t for k, t in times.items()}, "heads": H, "kv_heads": Hkv,
            "algorithmic_tflops": flops / (ms * 1e-3) / 1e12, "frac_of_mfma_peak": flops / (ms * 1e-3) / PEAK_BF16}


def serve_part(wl, attt, torch, reps):
    """The serving side, outside the timed step, at the workload's projection shapes with 16
    concurrent episode adapters (the paper's concurrency): a decoding step (one token per
    episode through q, k, v, o), a prefill of the workload's update rows through the same
    adapters, and the hot swap of one whole adapter of a 32-layer model (float32 masters to
    bf16). Bytes: every input once and y read and written; for the swap 4 + 2 bytes per
    parameter."""
    cfg = wl.cfg
    if cfg.dtype != "bf16":
        return None
    E, r, s = 16, cfg.rank, cfg.scale
    projs = cfg.projections
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1100)

    def randn(shape, std):
        return (torch.randn(shape, generator=gen, device="cuda") * std).to(torch.bfloat16)
    adapters = [[(randn((r, p.d_in), 0.02), randn((p.d_out, r), 0.02)) for p in projs] for _ in range(E)]
    ad_bytes = sum(2.0 * (A.numel() + B.numel()) for ad in adapters for A, B in ad)

    def problems(rows_of):
        out, nbytes = [], ad_bytes
        for e in range(E):
            L = rows_of(e)
            xs = {}
            for i, p in enumerate(projs):
                if p.x_group not in xs:
                    xs[p.x_group] = randn((L, p.d_in), 1.0)
                    nbytes += 2.0 * L * p.d_in
                y = randn((L, p.d_out), 1.0)
                nbytes += 4.0 * L * p.d_out
                A, B = adapters[e][i]
                out.append(dict(x=xs[p.x_group], y=y, A=A, B=B, scale=s))
        return out, nbytes

    def timed(probs):
        attt.lora_forward(probs)
        torch.cuda.synchronize()
        attt.timing_enable(True)
        attt.timing_reset()
        gpu_hold(torch, reps)
        for _ in range(reps):
            attt.lora_forward(probs)
        torch.cuda.synchronize()
        ms, n = attt.timing_read("lora_fwd")
        attt.timing_enable(False)
        return ms / reps, n / reps

    dec, dec_bytes = problems(lambda e: 1)
    dec_ms, dec_l = timed(dec)
    rows_per = max(1, cfg.rows // E)
    pre, pre_bytes = problems(lambda e: rows_per)
    pre_ms, pre_l = timed(pre)
    del pre
    # hot swap: q, k, v, o adapters of 32 layers at this shape
    layer = [(r, p.d_in) for p in projs] + [(p.d_out, r) for p in projs]
    n_par = 32 * sum(a * b for a, b in layer)
    masters = torch.randn(n_par, generator=gen, dtype=torch.float32, device="cuda") * 0.02
    slot = torch.empty(n_par, dtype=torch.bfloat16, device="cuda")
    pairs, o = [], 0
    for _ in range(32):
        for a, b in layer:
            pairs.append((masters[o:o + a * b], slot[o:o + a * b]))
            o += a * b
    attt.lora_hot_swap(pairs)
    torch.cuda.synchronize()
    attt.timing_enable(True)
    attt.timing_reset()
    gpu_hold(torch, reps)
    for _ in range(reps):
        attt.lora_hot_swap(pairs)
    torch.cuda.synchronize()
    sw_ms, sw_n = attt.timing_read("lora_swap")
    attt.timing_enable(False)
    sw_ms /= reps
    return {"adapters": E, "rank": r,
            "decode": {"rows": E, "ms": dec_ms, "launches": dec_l, "bytes": dec_bytes,
                       "gbs": dec_bytes / (dec_ms * 1e-3) / 1e9},
            "prefill": {"rows": E * rows_per, "ms": pre_ms, "launches": pre_l, "bytes": pre_bytes,
                        "gbs": pre_bytes / (pre_ms * 1e-3) / 1e9,
                        "frac_of_hbm_peak": pre_bytes / (pre_ms * 1e-3) / PEAK_HBM},
            "hot_swap": {"layers": 32, "tensors": len(pairs), "params": n_par, "ms": sw_ms,
                         "launches": sw_n / reps, "gbs": 6.0 * n_par / (sw_ms * 1e-3) / 1e9}}


def gpu_hold(torch, calls):
    """Keep the GPU busy (torch.cuda._sleep, ~1 ms per 2e6 cycles) while `calls` small calls are
    queued behind it, so the launch events around each kernel measure the kernel and not the
    host between calls."""
    sleep = getattr(torch.cuda, "_sleep", None)
    if sleep is not None:
        sleep(int(max(2e7, 1e6 * calls)))


def lora_sgd_part(step, attt, torch, reps):
    """The adapter step of Eq. 2 for the step's adapters, outside the timed step: float32
    masters of every A and B updated by their gradients, bf16 operand copies written and the
    gradients reset (one grouped call, the kernel's own time over `reps` calls). Algorithm 1
    takes two such steps per update."""
    params, nbytes = [], 0
    for p in step.problems:
        for k, g in (("A", "dA"), ("B", "dB")):
            master = p[k].float().clone()
            params.append(dict(param=master, grad=p[g], param_bf16=torch.empty_like(p[k])
                               if p[k].dtype == torch.bfloat16 else None))
            nbytes += master.numel() * (4 + 4 + 4 + 4 + (2 if p[k].dtype == torch.bfloat16 else 0))
    attt.timing_enable(True)
    attt.timing_reset()
    gpu_hold(torch, reps)
    for _ in range(reps):
        attt.lora_sgd_step(params, 5e-4, zero_grad=True)
    torch.cuda.synchronize()
    ms, n = attt.timing_read("lora_sgd")
    attt.timing_enable(False)
    ms /= reps  # per call (one launch per 16 tensors)
    return {"ms": ms, "launches_per_call": n / reps, "bytes": nbytes, "gbs": nbytes / (ms * 1e-3) / 1e9,
            "lr": 5e-4}


def head_transpose_part(step, attt, torch, reps=5):
    """The once-per-model transpose of the frozen LM head (outside the step): kernel time from the
    library's launch events, and the bytes it moves (read W, write W^T)."""
    attt.timing_enable(True)
    attt.timing_reset()
    for _ in range(reps):
        attt.ce_head_transpose(step.W, out=step.W_t)
    torch.cuda.synchronize()
    ms, n = attt.timing_read("ce_head_transpose")
    attt.timing_enable(False)
    ms /= max(1, n)
    nbytes = step.W.numel() * 2 + step.W_t.numel()
    return {"ms": ms, "bytes": nbytes, "gbs": nbytes / (ms * 1e-3) / 1e9}


def main():
    args = parse()
    if args.hbm_calibrate:
        hbm_calibrate()
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the update step of one episode group runs on a single "
              "MI355X and this build has no multi-GPU path (--gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2607_03441_amd as attt
    from workloads import Workload

    attt.load()
    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    wl = Workload(args.config)
    cfg = wl.cfg
    step = Step(wl, attt, torch)
    for _ in range(args.warmup):
        step.run()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    attt.timing_enable(True)
    attt.timing_reset()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps - 1)]
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        step.run()
        if i + 1 < args.steps:
            marks[i].record()
    stop.record()
    torch.cuda.synchronize()
    attt.timing_enable(False)
    ms_step = start.elapsed_time(stop) / args.steps
    bounds = [start] + marks + [stop]
    per_step = np.array([bounds[i].elapsed_time(bounds[i + 1]) for i in range(args.steps)])
    kern = {}
    for name in attt.kernel_names():
        ms, n = attt.timing_read(name)
        if n:
            kern[name] = {"ms_per_step": ms / args.steps, "launches_per_step": n / args.steps,
                          "avg_launch_ms": ms / n}
    log("kernels: " + ", ".join(f"{k} {v['ms_per_step']:.3f}ms" for k, v in kern.items()))

    alg = algorithmic(cfg, wl.tokens(), wl.lora())
    bf16 = cfg.dtype == "bf16"
    peak = PEAK_BF16 if bf16 else PEAK_F32_MFMA
    ce_kernels = ("ce_fwd_lse", "ce_bwd_dz", "ce_bwd_dh", "ce_fused_bwd")
    dom = max(ce_kernels, key=lambda k: kern.get(k, {}).get("ms_per_step", 0.0))
    # the f32 GEMM kernels contract N x V x d once per step each; the fused bf16 backward does
    # both contractions (logits and dL/dh), 4 N V d
    per_step_flops = alg["ce_flops_fwd"] + (alg["ce_flops_bwd"] if dom == "ce_fused_bwd" else 0.0)
    k = kern[dom]
    per_launch = per_step_flops / k["launches_per_step"]
    achieved = per_launch / (k["avg_launch_ms"] * 1e-3)
    roofline = {"bound": "mfma", "kernel": dom, "achieved": achieved / 1e12, "peak": peak / 1e12,
                "unit": "TFLOP/s", "frac": achieved / peak,
                "traffic": counter_traffic(cfg.name, dom),
                "traffic_source": "rocprofv3 FETCH_SIZE/WRITE_SIZE summary committed under profiles/ "
                                  "(null unless the CE sources still hash to its recorded values)",
                "flops_per_launch": per_launch}
    ce_ms = sum(kern.get(n, {}).get("ms_per_step", 0.0) for n in
                ("ce_fwd_lse", "ce_label_logit", "ce_row_reduce", "ce_loss", "ce_head_transpose", "ce_fused_bwd",
                 "ce_bwd_dz", "ce_bwd_dh", "ce_overflow_guard"))
    ng_ms = sum(kern.get(n, {}).get("ms_per_step", 0.0) for n in ("ngram_table", "ngram_count", "ngram_weight"))
    lo_ms = sum(kern.get(n, {}).get("ms_per_step", 0.0) for n in ("lora_u_du", "lora_dadb", "lora_reduce"))
    parts = {
        "ce_pass": {"ms": ce_ms, "algorithmic_tflops": 4 * cfg.rows * cfg.vocab * cfg.d / (ce_ms * 1e-3) / 1e12,
                    "frac_of_mfma_peak": 4 * cfg.rows * cfg.vocab * cfg.d / (ce_ms * 1e-3) / peak},
        "ngram_pass": {"ms": ng_ms, "algorithmic_gbs": alg["ngram_bytes"] / (ng_ms * 1e-3) / 1e9,
                       "frac_of_hbm_peak": alg["ngram_bytes"] / (ng_ms * 1e-3) / PEAK_HBM},
        "lora_pass": {"ms": lo_ms, "algorithmic_gbs": alg["lora_bytes"] / (lo_ms * 1e-3) / 1e9,
                      "frac_of_hbm_peak": alg["lora_bytes"] / (lo_ms * 1e-3) / PEAK_HBM},
    }
    parts["lora_sgd_per_step"] = lora_sgd_part(step, attt, torch, max(args.steps, 10))
    if step.W_t is not None:
        parts["head_transpose_once"] = head_transpose_part(step, attt, torch)
    if cfg.prior_updates > 0:
        ns = ngram_set_part(wl, attt, torch, max(args.steps, 10))
        ns["streaming_ngram_pass_ms"] = ng_ms
        parts["ngram_set_per_update"] = ns
    parts["repetition_filter"] = repetition_part(wl, attt, torch, 10)
    ap = attention_part(wl, attt, torch, 5)
    if ap is not None:
        parts["attention_bwd"] = ap
    sp = serve_part(wl, attt, torch, 10)
    if sp is not None:
        parts["lora_serve"] = sp
    out = {
        "metric": METRIC, "value": cfg.rows / (ms_step * 1e-3), "unit": "update tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "step_ms_p10_p50_p90": [float(np.percentile(per_step, q)) for q in (10, 50, 90)],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype, "data": "synthetic (seeded; see workloads/gen.py)",
        "config": {"workload": cfg.name, "episodes": cfg.episodes, "update_tokens": cfg.rows,
                   "history_tokens": int(wl.tokens()["hist_off"][-1]), "n": cfg.n, "w_min": cfg.w_min,
                   "d": cfg.d, "V": cfg.vocab, "lora_rank": cfg.rank,
                   "lora_projections": [f"{p.name}:{p.d_in}x{p.d_out}" for p in cfg.projections]},
        "roofline": roofline, "parts": parts, "kernels": kern,
        "paper_context": PAPER_CONTEXT,
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle sample")
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_rows)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
