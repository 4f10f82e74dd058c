"""The closed-loop replay divides with 32-bit multiply-highs whose constants
the library derives on the host (loop.hip: magic31, magic16, ceil_ms32).
These tests restate those derivations and check that each quotient is exact
over the whole range the kernel uses it on.

A multiplier m above 2^k / d gives floor(x * m / 2^k) >= floor(x / d) for
every x, and overshoots first just below a multiple of d: checking
x = k * d - 1 for every k (and the range's top value) covers every x."""
import numpy as np


def magic31(d):
    """(m, sh) with x // d == umulhi(x, m) >> sh for x < 2^31; sh = -1 for d = 1."""
    l = 0
    while (1 << l) < d:
        l += 1
    return (0 if l == 0 else ((1 << (31 + l)) + d - 1) // d), l - 1


def magic16(d):
    """m with x // d == umulhi(x, m) for x < 2^16 (m = 0: d = 1, x itself)."""
    if d == 1:
        return 0
    if d >= 65536:
        return 1
    return (1 << 32) // d + 1


def _umulhi(x, m):
    return (x.astype(np.uint64) * np.uint64(m)) >> np.uint64(32)


def _below_multiples(d, top):
    """x = k * d - 1 for every k with k * d - 1 <= top, and top itself."""
    k = np.arange(1, top // d + 2, dtype=np.uint64)
    x = k * np.uint64(d) - np.uint64(1)
    return np.concatenate([x[x <= top], np.array([top], np.uint64)])


def test_chunk_division_every_divisor():
    top = 65535
    for d in list(range(1, 65537)) + [65537, 100000, 1 << 20, (1 << 31) - 1]:
        m = magic16(d)
        x = _below_multiples(d, top) if d <= top else np.array([0, 1, top], np.uint64)
        q = x if m == 0 else _umulhi(x, m)
        assert np.array_equal(q, x // np.uint64(d)), d


def test_thousandth_every_32bit_dividend():
    # ceil(tokens * us / 1000) as umulhi(tokens * us + 999, ceil(2^38 / 1000)) >> 6
    m = 0x10624DD3
    assert m == -(-(1 << 38) // 1000)
    x = _below_multiples(1000, (1 << 32) - 1)
    assert np.array_equal(_umulhi(x, m) >> np.uint64(6), x // np.uint64(1000))


def test_window_division():
    top = (1 << 31) - 1
    rng = np.random.default_rng(31)
    divisors = list(range(1, 2049)) + [250, 1000, 86_400_000, top, top - 1]
    divisors += [(1 << e) + o for e in range(11, 31) for o in (-1, 0, 1)]
    divisors += [int(v) for v in rng.integers(2049, top, 300)]
    for d in divisors:
        m, sh = magic31(d)
        assert m < (1 << 32), d
        n = top // d + 1  # multiples k * d - 1 <= top for k = 1 .. n
        if n > 1 << 20:  # small divisors: the first and last 4096 multiples and a sample of the rest
            k = np.concatenate([np.arange(1, 4097), np.arange(n - 4095, n + 1), rng.integers(1, n + 1, 8192)])
        else:
            k = np.arange(1, n + 1)
        x = k.astype(np.uint64) * np.uint64(d) - np.uint64(1)
        x = np.concatenate([x[x <= top], np.array([top], np.uint64)])
        q = x if sh < 0 else _umulhi(x, m) >> np.uint64(sh)
        assert np.array_equal(q, x // np.uint64(d)), d
