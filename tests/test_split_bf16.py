"""The arithmetic of the c = 128 encode and decode kernels, which run their
fp32 contraction on bf16 MFMAs: each fp32 operand x is split into three
bf16 terms, x = h + m + l, each the rounding to nearest even of what the
earlier terms leave, and six of the nine term products are summed.  Here the
split is emulated bit by bit on the host and its claims are checked: the
split is exact, the terms shrink by 2^-8 each, every kept product is exact
in fp32, and the dropped products of a dot product sum to less than
2^-23 sum |a_k b_k| (two units of fp32 rounding).  The kernels themselves are
checked against the oracle on the GPU (dot-product bounds of the encode and
decode at c = 128)."""

import numpy as np


def bf16(x):
    """fp32 -> bf16 (round to nearest, ties to even) -> fp32, for finite x."""
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) & 0xFFFF0000
    return b.astype(np.uint32).view(np.float32)


def split3(x):
    x = np.asarray(x, dtype=np.float32)
    h = bf16(x)
    r = (x - h).astype(np.float32)
    m = bf16(r)
    l = bf16((r - m).astype(np.float32))
    return h, m, l


def significant_bits(v):
    """Bits between the leading and the trailing one of each fp32 significand."""
    b = np.asarray(v, dtype=np.float32).view(np.uint32)
    mant = (b & 0x7FFFFF) | np.where((b >> 23) & 0xFF, 0x800000, 0).astype(np.uint32)
    out = np.zeros(mant.shape, dtype=np.int64)
    nz = mant != 0
    mm = mant[nz].astype(np.int64)
    lead = np.floor(np.log2(mm)).astype(np.int64)
    trail = np.log2(mm & -mm).astype(np.int64)
    out[nz] = lead - trail + 1
    return out


def sample(rng, n):
    """fp32 values over 60 binades, both signs, with full 24-bit significands."""
    mant = rng.integers(1 << 23, 1 << 24, size=n).astype(np.float64)
    x = mant * 2.0 ** rng.integers(-53, 7, size=n) * rng.choice([-1.0, 1.0], size=n)
    return x.astype(np.float32)


def test_split_is_exact_and_each_term_is_a_bf16():
    rng = np.random.default_rng(1)
    x = np.concatenate([sample(rng, 200_000), np.float32([1.0, -1.0, 3.0, 1 + 2 ** -23, 2 ** -20, 65504.0])])
    h, m, l = split3(x)
    # each remainder is computed exactly in fp32
    assert np.array_equal((x.astype(np.float64) - h).astype(np.float32), (x - h).astype(np.float32))
    r = x.astype(np.float64) - h
    assert np.array_equal(r, (x - h).astype(np.float64))
    assert np.array_equal(r - m, ((x - h).astype(np.float32) - m).astype(np.float64))
    # the three terms add up to x exactly, and each holds at most 8 significant bits
    assert np.array_equal(h.astype(np.float64) + m + l, x.astype(np.float64))
    for t in (h, m, l):
        assert significant_bits(t).max() <= 8
        assert np.array_equal(bf16(t), t)
    ax = np.abs(x.astype(np.float64))
    assert np.all(np.abs(m) <= 2.0 ** -8 * (1 + 2.0 ** -8) * ax)
    assert np.all(np.abs(l) <= 2.0 ** -16 * ax)


def test_six_products_are_exact_and_the_dropped_three_are_below_two_units():
    rng = np.random.default_rng(2)
    for K in (4, 32, 128, 144):
        for _ in range(200):
            a, b = sample(rng, K), sample(rng, K)
            (ah, am, al), (bh, bm, bl) = split3(a), split3(b)
            kept = [(ah, bh), (ah, bm), (am, bh), (ah, bl), (am, bm), (al, bh)]
            for u, v in kept:                      # each kept product is exact in fp32
                prod = u.astype(np.float64) * v
                assert np.array_equal(prod.astype(np.float32).astype(np.float64), prod)
            approx = sum(np.sum(u.astype(np.float64) * v) for u, v in kept)
            exact = np.sum(a.astype(np.float64) * b)
            scale = np.sum(np.abs(a.astype(np.float64) * b))
            assert abs(approx - exact) <= 2.0 ** -23 * scale


def test_dropping_a_kept_product_breaks_the_bound():
    """The check above has teeth: without the m m product (or with only the
    three largest products) the error exceeds two units of fp32 rounding."""
    rng = np.random.default_rng(3)
    worst_five, worst_three = 0.0, 0.0
    for _ in range(200):
        a, b = sample(rng, 32), sample(rng, 32)
        (ah, am, al), (bh, bm, bl) = split3(a), split3(b)
        exact = np.sum(a.astype(np.float64) * b)
        scale = np.sum(np.abs(a.astype(np.float64) * b))
        five = [(ah, bh), (ah, bm), (am, bh), (ah, bl), (al, bh)]
        three = [(ah, bh), (ah, bm), (am, bh)]
        for prods, name in ((five, "five"), (three, "three")):
            err = abs(sum(np.sum(u.astype(np.float64) * v) for u, v in prods) - exact) / scale
            if name == "five":
                worst_five = max(worst_five, err)
            else:
                worst_three = max(worst_three, err)
    assert worst_five > 2.0 ** -23 and worst_three > 2.0 ** -23
