"""Oracle: update-text repetition rho, novelty nu and the sequence-level skip filter
(Sec. 3.2 "Update-Text Repetition", Eq. 6-7; the threshold tau = 0.5 of Appendix C).

Test infrastructure only: the GPU library never imports this module.

Definitions followed:
  * W(x) is the set of whitespace-separated words of an update text x. Texts are given as
    sequences of word ids (one id per whitespace word, equal words equal ids): the split and
    the mapping are host-side string work. `words_of_text` does both for literal strings.
  * J(A, B) = |A & B| / |A | B| (Jaccard similarity of two sets). Two empty sets have no
    union; J is taken as 0 there (reading: no overlap is evidenced).
  * Eq. 6: rho(x_k) = max over the previous update texts x' of the episode of J(W(x_k), W(x')),
    and rho = 0 for the first update (no previous text). Eq. 7: nu = 1 - rho.
  * The sequence-level baseline skips an update when nu < tau.
  * Arithmetic: J is exact (a fraction); the maximum is taken over exact fractions, the first
    previous text wins a tie. rho is the float64 nearest to the maximal fraction, nu the
    float64 nearest to 1 - rho, and the skip decision is nu < tau in float64.
"""
from fractions import Fraction


def words_of_text(text, vocab):
    """Whitespace split of a literal string, each word mapped to an id (new words get the
    next id of the shared dictionary `vocab`)."""
    ids = []
    for w in text.split():
        if w not in vocab:
            vocab[w] = len(vocab)
        ids.append(vocab[w])
    return ids


def jaccard(a_words, b_words):
    """J(W(a), W(b)) as an exact fraction, with (|A & B|, |A | B|)."""
    A, B = set(int(w) for w in a_words), set(int(w) for w in b_words)
    inter, union = len(A & B), len(A | B)
    return (Fraction(inter, union) if union else Fraction(0)), inter, union


def repetition(updates, tau=0.5):
    """One episode: `updates` are the word-id sequences of its update texts in order; the last
    is the candidate x_k, the others are the previous texts H_k.

    Returns dict(rho, nu, skip, best, pairs): best is the index of the previous text that
    attains the maximum (-1 for the first update), pairs the (|A & B|, |A | B|) of every
    previous text against the candidate."""
    cand = updates[-1]
    best, best_j, pairs = -1, Fraction(0), []
    for i, prev in enumerate(updates[:-1]):
        j, inter, union = jaccard(cand, prev)
        pairs.append((inter, union))
        if best < 0 or j > best_j:
            best, best_j = i, j
    rho = float(best_j)  # int / int in Python rounds to nearest
    nu = 1.0 - rho
    return dict(rho=rho, nu=nu, skip=bool(nu < tau), best=best, pairs=pairs)
