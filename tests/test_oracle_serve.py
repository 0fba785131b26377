"""Pins of the serving oracle (grouped multi-adapter forward and the adapter swap; Appendix A,
adapter of Sec. 3.1) against exact rational arithmetic with a hand-written round-to-nearest-
even, the zero adapter, a rank-one closed form, the merged-weight identity and worked
bfloat16 roundings."""
from fractions import Fraction

import numpy as np

from oracle import serve


def _bits(rng, shape, scale=1.0):
    v = (rng.standard_normal(shape) * scale).astype(np.float32)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def _frac_of_bits(b):
    return Fraction(float(serve.bf16_bits_to_f64(np.uint16(b))))


def _round_fraction_to_bf16(q):
    """Round a rational to bf16 by hand: find its binade, scale to an 8-bit significand,
    round half to even on the exact remainder."""
    if q == 0:
        return 0
    neg = q < 0
    a = -q if neg else q
    e = 0
    while a >= 2:
        a /= 2
        e += 1
    while a < 1:
        a *= 2
        e -= 1
    e = max(e, -126)                       # below the normal range the spacing stays 2^-133
    m = abs(q) / Fraction(2) ** (e - 7)    # significand scaled to [128, 256) (normal range)
    f = m.numerator // m.denominator
    r = m - f
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and f % 2 == 1):
        f += 1
    if f == 256:
        f, e = 128, e + 1
    val = Fraction(f) * Fraction(2) ** (e - 7)
    bits = int(np.float32(float(val)).view(np.uint32)) >> 16
    return bits | (0x8000 if neg else 0)


def test_forward_matches_exact_rationals():
    rng = np.random.default_rng(7)
    rows, d_in, d_out, r, s = 5, 6, 4, 3, 2.0
    x, y, A, B = _bits(rng, (rows, d_in)), _bits(rng, (rows, d_out)), _bits(rng, (r, d_in), 0.3), \
        _bits(rng, (d_out, r), 0.3)
    got = serve.lora_forward(x, y, A, B, s)
    for i in range(rows):
        for o in range(d_out):
            u = [sum(_frac_of_bits(x[i, k]) * _frac_of_bits(A[c, k]) for k in range(d_in)) for c in range(r)]
            exact = _frac_of_bits(y[i, o]) + Fraction(s) * sum(u[c] * _frac_of_bits(B[o, c]) for c in range(r))
            assert got[i, o] == _round_fraction_to_bf16(exact), (i, o)


def test_rounding_of_float64_by_hand():
    one = 1.0
    ulp = 2.0 ** -7
    cases = [(one, 0x3F80), (one + ulp / 2, 0x3F80), (one + 3 * ulp / 2, 0x3F82),
             (one + ulp / 2 + 2.0 ** -40, 0x3F81),      # just above the tie: float32 would lose it
             (-(one + ulp / 2 - 2.0 ** -40), 0xBF80), (0.0, 0x0000), (-0.0, 0x8000),
             (2.0 ** 128, 0x7F80), (3.4e38, 0x7F80), (-np.inf, 0xFF80), (2.0 ** -133, 0x0001),
             (1.5 * 2.0 ** -133, 0x0002), (2.0 ** -134, 0x0000)]
    got = serve.round_f64_to_bf16_bits(np.array([c[0] for c in cases]))
    assert got.tolist() == [c[1] for c in cases]
    assert (int(serve.round_f64_to_bf16_bits(np.array([np.nan]))[0]) & 0x7FC0) == 0x7FC0
    # agrees with exact rounding on random values across binades
    rng = np.random.default_rng(3)
    v = rng.standard_normal(300) * np.exp2(rng.integers(-40, 40, 300))
    got = serve.round_f64_to_bf16_bits(v)
    assert got.tolist() == [_round_fraction_to_bf16(Fraction(float(a))) for a in v]


def test_zero_adapter_keeps_y():
    rng = np.random.default_rng(1)
    x, y, A = _bits(rng, (9, 16)), _bits(rng, (9, 8)), _bits(rng, (4, 16))
    B = np.zeros((8, 4), np.uint16)
    assert np.array_equal(serve.lora_forward(x, y, A, B, 4.0), y)


def test_rank_one_closed_form():
    """A = a^T, B = b: the delta of row i, column o is s (x_i . a) b_o."""
    rng = np.random.default_rng(2)
    x, y = _bits(rng, (7, 12)), _bits(rng, (7, 5))
    a, b = _bits(rng, (1, 12), 0.5), _bits(rng, (5, 1), 0.5)
    xf, yf, af, bf = (serve.bf16_bits_to_f64(t) for t in (x, y, a, b))
    want = np.empty_like(yf)
    for i in range(7):
        dot = sum(xf[i, k] * af[0, k] for k in range(12))
        for o in range(5):
            want[i, o] = yf[i, o] + 2.0 * dot * bf[o, 0]
    assert np.array_equal(serve.lora_forward(x, y, a, b, 2.0), serve.round_f64_to_bf16_bits(want))


def test_merged_weight_identity():
    """Adding the adapter term equals multiplying by the merged weight s B A (small integers,
    so every product and sum is exact in float64)."""
    rng = np.random.default_rng(4)
    ints = lambda shape: (rng.integers(-3, 4, shape).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    x, y, A, B = ints((6, 10)), ints((6, 7)), ints((2, 10)), ints((7, 2))
    xf, yf, Af, Bf = (serve.bf16_bits_to_f64(t) for t in (x, y, A, B))
    merged = yf + xf @ (0.5 * (Bf @ Af)).T
    assert np.array_equal(serve.lora_forward(x, y, A, B, 0.5), serve.round_f64_to_bf16_bits(merged))


def test_grouped_problems_are_independent():
    rng = np.random.default_rng(5)
    probs = [dict(x=_bits(rng, (3, 8)), y=_bits(rng, (3, 8)), A=_bits(rng, (2, 8)), B=_bits(rng, (8, 2)),
                  scale=s) for s in (1.0, 2.0)]
    out = serve.grouped_lora_forward(probs)
    for p, o in zip(probs, out):
        assert np.array_equal(o, serve.lora_forward(p["x"], p["y"], p["A"], p["B"], p["scale"]))


def test_hot_swap_rounds_to_nearest_even():
    vals = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -1.0 - 2.0 ** -8 - 2.0 ** -20], np.float32)
    assert serve.hot_swap(vals).tolist() == [0x3F80, 0x3F80, 0x3F82, 0xBF81]
