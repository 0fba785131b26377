"""Seeded input generator shared by the oracle tests, the GPU tests and the bench.

It produces token streams (the previous updates forming the history H^tok and the
new update x_k), LM-head inputs and LoRA inputs. Everything is drawn from numpy's
PCG64 generator seeded per configuration, so both sides of every parity check see
identical inputs. Nothing here computes any part of the method: no n-gram
counting, no softmax, no gradients.

Token streams (recipe):
  * Fresh tokens are uniform over [0, id_range) or Zipf(s) over ranks mapped to
    ids through a seeded permutation (inverse CDF over p_k proportional to k^-s).
  * Each update alternates a fresh gap and a copied span. Gap lengths are
    geometric with mean mu*(1-p)/p (mu = mean span length, p = copy fraction),
    so a fraction p of tokens is copied on average. A copied span has a length
    uniform in [lo, hi] and is taken from a uniformly chosen earlier update of the
    same episode at a uniform offset.
  * Previous update 0 is all fresh; previous update i copies from updates < i;
    the new update copies from all previous updates.

Dense inputs: hidden states ~ N(0,1), LM head ~ N(0, 0.02^2), LoRA A ~ N(0, 0.02^2),
B = 0 or ~ N(0, 0.02^2), LoRA inputs X ~ N(0,1), upstream gradients dY ~ N(0,1)/L.
bf16 configurations round every float input to bf16 (round to nearest even) and
hand both sides the same bf16 values: the oracle gets them widened exactly, the
GPU path gets the bit patterns.
"""
import numpy as np

from .configs import Config, get

_STREAM_IDS, _STREAM_H, _STREAM_W, _STREAM_X, _STREAM_A, _STREAM_B, _STREAM_DY, _STREAM_AUX = range(8)


def bf16_bits(a) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even. Inputs are finite."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounded = (u.astype(np.uint64) + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_to_f32(bits) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


class Dense:
    """A float input as exact float32 values plus, for bf16 configs, its bit patterns."""

    def __init__(self, values_f32, bf16):
        if bf16:
            self.bits = bf16_bits(values_f32)
            self.f32 = bf16_to_f32(self.bits)
        else:
            self.bits = None
            self.f32 = np.ascontiguousarray(values_f32, dtype=np.float32)

    @property
    def shape(self):
        return self.f32.shape

    def __array__(self, dtype=None, copy=None):
        return self.f32 if dtype is None else self.f32.astype(dtype)

    def __getitem__(self, idx):
        return self.f32[idx]


def _normal(rng, shape, std, bf16):
    a = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return Dense(a, bf16)


class _Fresh:
    def __init__(self, cfg: Config, rng):
        self.cfg = cfg
        if cfg.id_dist == "zipf":
            ranks = np.arange(1, cfg.id_range + 1, dtype=np.float64)
            p = ranks ** (-cfg.zipf_s)
            self.cdf = np.cumsum(p / p.sum())
            self.perm = rng.permutation(cfg.id_range).astype(np.int32)
        elif cfg.id_dist != "uniform":
            raise ValueError(cfg.id_dist)

    def draw(self, rng, count):
        if count <= 0:
            return np.empty(0, np.int32)
        if self.cfg.id_dist == "uniform":
            return rng.integers(0, self.cfg.id_range, count, dtype=np.int32)
        u = rng.random(count)
        idx = np.minimum(np.searchsorted(self.cdf, u, side="right"), self.cfg.id_range - 1)
        return self.perm[idx]


def _make_update(rng, fresh: _Fresh, length, sources, p, span):
    lo, hi = span
    mean_span = 0.5 * (lo + hi)
    out = []
    have = 0
    if not sources or p <= 0.0:
        return fresh.draw(rng, length)
    # P(gap = g) = q (1-q)^g, mean (1-q)/q = mean_span (1-p)/p
    q = p / (p + mean_span * (1.0 - p))
    while have < length:
        gap = int(rng.geometric(q)) - 1 if q < 1.0 else 0
        if gap:
            out.append(fresh.draw(rng, gap))
            have += gap
        if have >= length:
            break
        ell = int(rng.integers(lo, hi + 1))
        src = sources[int(rng.integers(0, len(sources)))]
        ell = min(ell, len(src))
        off = int(rng.integers(0, len(src) - ell + 1))
        out.append(src[off:off + ell])
        have += ell
    return np.concatenate(out)[:length].astype(np.int32)


class Workload:
    """All inputs of one configuration, generated lazily and cached."""

    def __init__(self, cfg, seed=None):
        self.cfg = get(cfg) if isinstance(cfg, str) else cfg
        ss = np.random.SeedSequence(self.cfg.seed if seed is None else seed)
        self._streams = ss.spawn(8)
        self._tokens = None
        self._ce = None
        self._lora = None

    def _rng(self, i):
        return np.random.Generator(np.random.PCG64(self._streams[i]))

    # ---- token streams ---------------------------------------------------------------
    def tokens(self):
        """Per-episode previous updates and new update, flattened with host offsets.

        Returns dict with history (list of int32 arrays: H^tok per episode, the
        concatenation of its previous updates), updates (list of int32 arrays:
        x_k per episode), hist_flat / hist_off and tok_flat / tok_off (int64 [E+1]).
        """
        if self._tokens is not None:
            return self._tokens
        cfg = self.cfg
        ep_seeds = self._streams[_STREAM_IDS].spawn(cfg.episodes + 1)
        fresh = _Fresh(cfg, np.random.Generator(np.random.PCG64(ep_seeds[-1])))
        histories, updates = [], []
        for e in range(cfg.episodes):
            rng = np.random.Generator(np.random.PCG64(ep_seeds[e]))
            prior = []
            for _ in range(cfg.prior_updates):
                prior.append(_make_update(rng, fresh, cfg.prior_len, prior, cfg.copy_frac, cfg.span))
            x = _make_update(rng, fresh, cfg.update_len, prior, cfg.copy_frac, cfg.span)
            histories.append(np.concatenate(prior).astype(np.int32) if prior else np.empty(0, np.int32))
            updates.append(x)
        self._tokens = pack_episodes(histories, updates)
        return self._tokens

    # ---- LM head inputs ---------------------------------------------------------------
    def ce(self):
        """h [N, d], W [V, d], labels [N] (= the update tokens), row_offsets [E+1]."""
        if self._ce is not None:
            return self._ce
        cfg = self.cfg
        bf16 = cfg.dtype == "bf16"
        tok = self.tokens()
        h = _normal(self._rng(_STREAM_H), (cfg.rows, cfg.d), 1.0, bf16)
        W = _normal(self._rng(_STREAM_W), (cfg.vocab, cfg.d), 0.02, bf16)
        labels = tok["tok_flat"].astype(np.int32)
        if labels.size and labels.max() >= cfg.vocab:
            raise ValueError("token ids exceed the LM-head vocabulary")
        self._ce = dict(h=h, W=W, labels=labels, row_offsets=tok["tok_off"].copy())
        return self._ce

    # ---- LoRA inputs ------------------------------------------------------------------
    def lora(self):
        """One problem per (episode, projection): x [L, d_in], dy [L, d_out], A [r, d_in],
        B [d_out, r], scale = alpha / r. Projections of one x_group share x."""
        if self._lora is not None:
            return self._lora
        cfg = self.cfg
        bf16 = cfg.dtype == "bf16"
        L = cfg.update_len
        rx, ra, rb, rdy = (self._rng(_STREAM_X), self._rng(_STREAM_A), self._rng(_STREAM_B),
                           self._rng(_STREAM_DY))
        problems = []
        for e in range(cfg.episodes):
            xs = {}
            for p in cfg.projections:
                if p.x_group not in xs:
                    xs[p.x_group] = _normal(rx, (L, p.d_in), 1.0, bf16)
                A = _normal(ra, (cfg.rank, p.d_in), 0.02, bf16)
                if cfg.lora_b_zero:
                    B = Dense(np.zeros((p.d_out, cfg.rank), np.float32), bf16)
                else:
                    B = _normal(rb, (p.d_out, cfg.rank), 0.02, bf16)
                dy = _normal(rdy, (L, p.d_out), 1.0 / L, bf16)
                problems.append(dict(name=f"e{e}.{p.name}", episode=e, x=xs[p.x_group], dy=dy,
                                     A=A, B=B, scale=cfg.scale, rank=cfg.rank,
                                     d_in=p.d_in, d_out=p.d_out, rows=L))
        self._lora = problems
        return problems


def pack_episodes(histories, updates):
    """Flatten per-episode token arrays into one array each plus int64 offsets [E+1]."""
    def flat(parts):
        off = np.zeros(len(parts) + 1, np.int64)
        off[1:] = np.cumsum([len(p) for p in parts])
        arr = np.concatenate(parts).astype(np.int32) if parts and off[-1] else np.empty(0, np.int32)
        return arr, off
    hf, ho = flat([np.asarray(h, np.int32) for h in histories])
    tf, to = flat([np.asarray(u, np.int32) for u in updates])
    return dict(history=[np.asarray(h, np.int32) for h in histories],
                updates=[np.asarray(u, np.int32) for u in updates],
                hist_flat=hf, hist_off=ho, tok_flat=tf, tok_off=to)


def random_dense(shape, std, bf16, seed):
    """A seeded dense input of arbitrary shape, for edge-case tests."""
    return _normal(np.random.Generator(np.random.PCG64(seed)), shape, std, bf16)
