"""Oracle: n-gram exposure f and token weights w of the aTTT update (Sec. 3.3, Eq. 8-9).

Test infrastructure only: the GPU library never imports this module.

Definitions followed (Sec. 3.3 "Repetition-Aware Token Reweighting", Algorithm 1):
  * The token history H^tok_k is the concatenation of all token sequences used in
    previous updates of the episode. It is taken literally as one flat sequence, so
    n-grams that straddle two previous updates are counted too.
  * count(g, H) is the number of start positions i with H[i:i+n] == g (sliding,
    overlapping occurrences).
  * Eq. 8: f_k(j) is the largest count(g, H^tok_k) over the n-grams g of x_k that
    contain position j; with no such n-gram (L < n) the maximum is taken as 0.
    Occurrences of g inside x_k itself are not counted.
  * Eq. 9: w_{k,j} = max(w_min, 1 / (1 + f_k(j))), evaluated in float32 with round to
    nearest even: the fp32 value of w_min against RN(1 / (1 + f)).
"""
from collections import Counter

import numpy as np


def ngram_counts(history, n):
    """count(g, H) for every n-gram g present in H (overlapping occurrences)."""
    h = [int(t) for t in history]
    m = len(h) - n + 1
    if m <= 0:
        return Counter()
    return Counter(zip(*[h[i:i + m] for i in range(n)]))


def exposure(history, tokens, n):
    """Eq. 8 for one episode: f[j] = max over n-grams of x covering j of their count in H."""
    x = [int(t) for t in tokens]
    L = len(x)
    cnt = ngram_counts(history, n)
    starts = L - n + 1
    c = [cnt.get(tuple(x[s:s + n]), 0) for s in range(max(starts, 0))]
    f = np.zeros(L, np.uint32)
    for j in range(L):
        lo = max(0, j - n + 1)
        hi = min(j, starts - 1)
        f[j] = max(c[lo:hi + 1], default=0)
    return f


def exposure_bruteforce(history, tokens, n):
    """Eq. 8 by direct scanning: every n-gram of x is compared with every window of H."""
    h = [int(t) for t in history]
    x = [int(t) for t in tokens]
    L = len(x)
    f = np.zeros(L, np.uint32)
    for j in range(L):
        best = 0
        for s in range(j - n + 1, j + 1):       # n-grams x[s:s+n] that contain position j
            if s < 0 or s + n > L:
                continue
            g = x[s:s + n]
            count = 0
            for i in range(len(h) - n + 1):
                if h[i:i + n] == g:
                    count += 1
            best = max(best, count)
        f[j] = best
    return f


def weights_from_exposure(f, w_min):
    """Eq. 9 in float32: max(w_min, RN(1 / (1 + f)))."""
    f32 = np.asarray(f, dtype=np.float32)
    one = np.float32(1.0)
    inv = one / (one + f32)
    return np.maximum(np.float32(w_min), inv).astype(np.float32)


def ngram_weights(histories, updates, n, w_min):
    """The weighting loop of Algorithm 1 for E episodes; returns concatenated (f uint32, w float32)."""
    fs = [exposure(h, x, n) for h, x in zip(histories, updates)]
    f = np.concatenate(fs) if fs else np.empty(0, np.uint32)
    return f.astype(np.uint32), weights_from_exposure(f, w_min)
