"""GPU parity of the serving side (Appendix A; adapter of Sec. 3.1): the grouped multi-adapter
forward y <- RN_bf16(y + s (x A^T) B^T) and the adapter hot swap, through the C ABI, against
oracle/serve.py on the same seeded inputs.

Bar: the forward's y is bit-identical to the correctly rounded exact sum, except where a value
within the kernel's float32 error bound of that sum rounds differently (near a bf16 rounding
midpoint, or where y and the adapter term cancel): there the GPU's y must be the rounding of
some value within the bound. The bound is the standard a priori one,
(d_in + rank + 2) u (|y| + s sum_c |x||A_c| |B_c|) with u = 2^-24 (the kernel sums in float32,
the oracle exactly). Differences must also be rare. The swap is bit-exact."""
import numpy as np
import pytest

from gpu_util import note
from oracle import serve

pytestmark = pytest.mark.gpu


def _bits(rng, shape, scale=1.0):
    v = (rng.standard_normal(shape) * scale).astype(np.float32)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def _dev(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def _bits_of(t):
    import torch
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def _ordered(b):
    b = np.asarray(b, np.int64)
    return np.where(b & 0x8000, -(b & 0x7FFF), b)


def _check_forward(got, p):
    """got: the GPU's new y bits for problem p (dict of bit arrays and scale). Every element
    must equal the correctly rounded exact sum or, where the two differ, be the rounding of a
    value within the float32 error bound of the exact sum (RN is monotonic, so it lies between
    the roundings of exact -/+ bound). Returns the number of differing elements."""
    want = serve.lora_forward(p["x"], p["y"], p["A"], p["B"], p["scale"])
    diff = got != want
    if not diff.any():
        return 0
    x, y, A, B = (serve.bf16_bits_to_f64(p[k]) for k in ("x", "y", "A", "B"))
    s = float(p["scale"])
    exact = (y + s * ((x @ A.T) @ B.T))[diff]
    mag = (np.abs(y) + abs(s) * ((np.abs(x) @ np.abs(A).T) @ np.abs(B).T))[diff]
    bound = (x.shape[1] + A.shape[0] + 2) * 2.0 ** -24 * mag
    lo = _ordered(serve.round_f64_to_bf16_bits(exact - bound))
    hi = _ordered(serve.round_f64_to_bf16_bits(exact + bound))
    g = _ordered(got[diff])
    bad = (g < lo) | (g > hi)
    assert not bad.any(), (int(bad.sum()), np.argwhere(diff)[bad][:8].tolist())
    return int(diff.sum())


def _problem(rng, rows, d_in, d_out, rank, scale=2.0, x=None):
    return dict(x=_bits(rng, (rows, d_in)) if x is None else x, y=_bits(rng, (rows, d_out)),
                A=_bits(rng, (rank, d_in), 0.05), B=_bits(rng, (d_out, rank), 0.05), scale=scale)


def _run(attt, probs):
    dev = {}
    calls = []
    for p in probs:
        if id(p["x"]) not in dev:
            dev[id(p["x"])] = _dev(p["x"])
        calls.append(dict(x=dev[id(p["x"])], y=_dev(p["y"]), A=_dev(p["A"]), B=_dev(p["B"]), scale=p["scale"]))
    attt.lora_forward(calls)
    return [_bits_of(c["y"]) for c in calls]


@pytest.mark.parametrize("rows,d_in,d_out,rank", [(1, 64, 64, 8), (5, 136, 72, 3), (16, 256, 264, 16),
                                                  (17, 128, 64, 17), (64, 512, 520, 33), (65, 96, 8, 64),
                                                  (300, 1032, 1544, 16), (129, 4096, 1024, 8)])
def test_forward_shapes(attt, rows, d_in, d_out, rank):
    note(f"lora_forward rows={rows} d_in={d_in} d_out={d_out} rank={rank}")
    rng = np.random.default_rng(rows * 7919 + d_in + rank)
    p = _problem(rng, rows, d_in, d_out, rank)
    got, = _run(attt, [p])
    assert _check_forward(got, p) <= max(2, 2e-3 * got.size)


def test_forward_grouped_qkvo_ragged_episodes(attt):
    """Sixteen episodes with ragged row counts (0 to 200, decoding and prefill mixed), each with
    its own adapters on q, k, v (sharing x) and o, all in one call."""
    rng = np.random.default_rng(11)
    rows = [0, 1, 1, 2, 15, 16, 17, 31, 63, 64, 65, 100, 128, 129, 200, 3]
    d, kv, r = 512, 128, 8
    probs = []
    for L in rows:
        x = _bits(rng, (L, d))
        for d_out in (d, kv, kv):
            probs.append(_problem(rng, L, d, d_out, r, x=x))
        probs.append(_problem(rng, L, d, d, r))
    note(f"lora_forward grouped: {len(probs)} problems")
    outs = _run(attt, probs)
    near = sum(_check_forward(g, p) for g, p in zip(outs, probs))
    note(f"elements off the correctly rounded sum (within the float32 bound): {near} of {sum(g.size for g in outs)}")


def test_forward_mixed_ranks_share_x(attt):
    """Problems sharing x with ranks 16 + 33 + 15 (four 16-rank units together) and one more
    that does not fit the group."""
    rng = np.random.default_rng(12)
    x = _bits(rng, (77, 264))
    probs = [_problem(rng, 77, 264, o, r, scale=s, x=x) for o, r, s in ((64, 16, 1.0), (40, 33, 0.5), (8, 15, 4.0),
                                                                     (16, 2, 2.0))]
    outs = _run(attt, probs)
    for g, p in zip(outs, probs):
        _check_forward(g, p)


def test_forward_decode_16_adapters_llama_shape(attt):
    """The serving step the paper runs: 16 episodes, one new token each, adapters on q/k/v/o at
    d = 4096 (grouped-query k, v of 1024), rank 16."""
    rng = np.random.default_rng(13)
    probs = []
    for e in range(16):
        x = _bits(rng, (1, 4096))
        for d_out in (4096, 1024, 1024):
            probs.append(_problem(rng, 1, 4096, d_out, 16, scale=1.0, x=x))
        probs.append(_problem(rng, 1, 4096, 4096, 16, scale=1.0))
    outs = _run(attt, probs)
    for g, p in zip(outs, probs):
        _check_forward(g, p)


def test_forward_prefill_full_size(attt):
    """One episode's 8192 rows through q, k, v, o at the Llama-8B shape, every element."""
    rng = np.random.default_rng(14)
    x = _bits(rng, (8192, 4096))
    probs = [_problem(rng, 8192, 4096, o, 16, scale=1.0, x=x) for o in (4096, 1024, 1024)]
    probs.append(_problem(rng, 8192, 4096, 4096, 16, scale=1.0))
    note("lora_forward prefill 8192 x 4096, q/k/v/o")
    outs = _run(attt, probs)
    near = sum(_check_forward(g, p) for g, p in zip(outs, probs))
    total = sum(g.size for g in outs)
    note(f"elements off the correctly rounded sum (within the float32 bound): {near} of {total}")
    assert near <= 1e-3 * total


def test_forward_deterministic_and_zero_adapter(attt):
    import torch
    rng = np.random.default_rng(15)
    p = _problem(rng, 300, 1024, 512, 16)
    x, A, B = _dev(p["x"]), _dev(p["A"]), _dev(p["B"])
    y0 = _dev(p["y"])
    res = []
    for _ in range(3):
        y = y0.clone()
        attt.lora_forward([dict(x=x, y=y, A=A, B=B, scale=2.0)])
        res.append(_bits_of(y))
    assert all(np.array_equal(res[0], r) for r in res[1:])
    y = y0.clone()
    attt.lora_forward([dict(x=x, y=y, A=A, B=torch.zeros_like(B), scale=2.0)])
    assert np.array_equal(_bits_of(y), p["y"])


def _swap_values(rng, n):
    v = rng.standard_normal(n).astype(np.float32) * np.exp2(rng.integers(-30, 30, n)).astype(np.float32)
    special = np.array([np.inf, -np.inf, np.nan, 0.0, -0.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8,
                        3.4e38, 1e-40, -1e-45], np.float32)
    v[: min(n, special.size)] = special[: min(n, special.size)]
    return v


def test_hot_swap_bit_exact(attt):
    import torch
    rng = np.random.default_rng(16)
    sizes = [1, 7, 8, 9, 2047, 2048, 2049, 100003, 1 << 20]
    pairs, srcs = [], []
    for n in sizes:
        v = _swap_values(rng, n)
        srcs.append(v)
        pairs.append((torch.from_numpy(v).cuda(), torch.empty(n, dtype=torch.bfloat16, device="cuda")))
    # unaligned views take the element path
    base = torch.from_numpy(_swap_values(rng, 1001)).cuda()
    dst_base = torch.empty(1001, dtype=torch.bfloat16, device="cuda")
    pairs.append((base[1:], dst_base[1:]))
    srcs.append(base[1:].cpu().numpy())
    note(f"hot swap of {len(pairs)} tensors")
    attt.lora_hot_swap(pairs)
    for (_, dst), v in zip(pairs, srcs):
        got = _bits_of(dst)
        want = serve.hot_swap(v)
        nan = np.isnan(v)
        assert np.array_equal(got[~nan], want[~nan])
        assert np.all((got[nan] & 0x7F80) == 0x7F80) and np.all((got[nan] & 0x7F) != 0)


def test_swap_then_forward_on_one_stream(attt):
    """A forward launched after the swap on the same stream reads the swapped adapter."""
    import torch
    rng = np.random.default_rng(17)
    p = _problem(rng, 40, 256, 128, 8)
    A32 = (rng.standard_normal((8, 256)) * 0.05).astype(np.float32)
    B32 = (rng.standard_normal((128, 8)) * 0.05).astype(np.float32)
    A = _dev(p["A"])
    B = _dev(p["B"])
    y = _dev(p["y"])
    attt.lora_hot_swap([(torch.from_numpy(A32).cuda(), A.view(-1)), (torch.from_numpy(B32).cuda(), B.view(-1))])
    attt.lora_forward([dict(x=_dev(p["x"]), y=y, A=A, B=B, scale=2.0)])
    q = dict(p, A=serve.hot_swap(A32).reshape(8, 256), B=serve.hot_swap(B32).reshape(128, 8))
    _check_forward(_bits_of(y), q)
