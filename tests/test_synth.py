"""The seeded input generators: the published splitmix64 sequence, the NumPy
path against the generator's definition in Python integers, the
distributions the workloads ask for, and the model shapes and bucket layout
of the synthetic gradients."""

import math

import numpy as np
import pytest

from paper_2609_23898_amd import synth


def test_splitmix64_matches_published_sequence():
    # splitmix64 from state 1234567: the first five outputs of the reference
    # generator (Steele, Lea & Flood 2014; Vigna's public-domain C version)
    x = 1234567
    got = []
    for _ in range(5):
        x = (x + synth._GOLDEN) & synth._MASK64
        got.append(synth._mix64_int(x))
    assert got == [6457827717110365317, 3203168211198807973, 9817491932198370423,
                   4593380528125082431, 16408922859458223821]


def _value_python(wl, worker, idx):
    """One entry from Python integers and floats alone: the definition of the
    generator written out, independent of the NumPy vectorisation."""
    import bisect
    if idx >= wl.d:
        return np.float32(0.0)
    key = wl.worker_key(worker)

    def bits(slot):
        return synth._mix64_int((key + (idx * 8 + slot + 1) * synth._GOLDEN) & synth._MASK64)

    # Box-Muller: u1 in (0, 1] and u2 in [0, 1) from the top 53 bits of slots 0 and 1
    u1 = float((bits(0) >> 11) + 1) * 2.0 ** -53
    i2 = bits(1) >> 11
    # ln u1 = e ln 2 + 2 atanh(t), u1 = m 2^e, m in [sqrt(1/2), sqrt(2)), t = (m - 1)/(m + 1)
    m, e = math.frexp(u1)
    if m < 0.707106781186547524401:
        m, e = m * 2.0, e - 1
    t = (m - 1.0) / (m + 1.0)
    acc = 1.0 / 21.0
    for k in range(9, -1, -1):
        acc = acc * (t * t) + 1.0 / float(2 * k + 1)
    ln_u1 = float(e) * 0.693147180559945309417 + 2.0 * (t * acc)
    # cos(2 pi u2) by octants: 2 pi u2 = (pi/4)(o + f)
    w8 = float(i2) * 2.0 ** -50
    o = i2 >> 50
    f = w8 - float(o)
    phi = (1.0 - f if o % 2 else f) * 0.785398163397448309616
    p2 = phi * phi

    def coef(first, k):
        fact = 1.0
        for i in range(2, first + 2 * k + 1):
            fact = fact * float(i)
        return (-1.0 if k % 2 else 1.0) / fact

    c = coef(0, 9)
    for k in range(8, -1, -1):
        c = c * p2 + coef(0, k)
    sn = coef(1, 8)
    for k in range(7, -1, -1):
        sn = sn * p2 + coef(1, k)
    sn = sn * phi
    cv = sn if o in (1, 2, 5, 6) else c
    if o in (2, 3, 4, 5):
        cv = -cv
    v = math.sqrt(-2.0 * ln_u1) * cv
    if wl.outlier_prob > 0 and (bits(6) & 0xFFFFFFFF) < wl.outlier_threshold:
        v = v * float(wl.outlier_factor)
    t = bisect.bisect_right(list(wl._offsets), idx) - 1
    return np.float32(v * float(wl.tensor_scales()[t]))


def test_numpy_path_matches_the_definition():
    """values_np (vectorised uint64 NumPy) against Python big integers, on
    every workload kind: tensor scales, i.i.d. scale, outliers, the pad."""
    rng = np.random.default_rng(0)
    for name in ("tiny-n4-c4", "iid-n8-c16-16m", "gpt2-small", "pythia-1.4b", "heavytail-n16-c128"):
        wl = synth.workload(name)
        idx = np.unique(np.concatenate([rng.integers(0, wl.d, 400), [0, wl.d - 1, wl.d, wl.d + 5]]))
        if wl.tensor_sizes is not None:           # both sides of every tensor boundary
            b = wl._offsets[1:-1]
            idx = np.unique(np.concatenate([idx, b, b - 1]))
        for w in (0, wl.N - 1):
            a = wl.values_np(w, idx)
            ref = np.array([_value_python(wl, w, int(i)) for i in idx], dtype=np.float32)
            assert a.dtype == np.float32
            np.testing.assert_array_equal(a.view(np.uint32), ref.view(np.uint32))
    wl = synth.workload("heavytail-n16-c128")
    assert np.abs(wl.values_np(1, np.arange(20000))).max() > 6      # outliers are in the check


def test_box_muller_normal_is_standard_normal():
    """The gradient entries' normal: moments, a Kolmogorov-Smirnov test and
    the tail beyond 4 sigma of N(0, 1), and its logarithm and cosine against
    the library functions to within a few units of double rounding."""
    from scipy import stats
    z = synth.gauss_np(synth.stream_key(1, 1), np.arange(2_000_000))
    assert abs(z.mean()) < 3e-3 and abs(z.var() - 1.0) < 3e-3
    assert abs(np.mean(z ** 4) - 3.0) < 0.03
    assert stats.kstest(z, "norm").pvalue > 0.01
    tail = np.mean(np.abs(z) > 4.0)                      # 6.33e-5 for N(0, 1)
    assert 3.5e-5 < tail < 9.5e-5 and np.abs(z).max() > 4.5
    rng = np.random.default_rng(7)
    u = (rng.integers(0, 1 << 53, 200_000) + 1).astype(np.float64) * 2.0 ** -53
    ln = synth._ln_unit_np(u)
    assert np.max(np.abs(ln - np.log(u)) / np.maximum(np.abs(np.log(u)), 1e-300)) < 4e-15
    i2 = rng.integers(0, 1 << 53, 200_000)
    w8 = i2.astype(np.float64) * 2.0 ** -50
    cos = synth._cos_2pi_np(w8, (i2 >> 50).astype(np.int64))
    assert np.max(np.abs(cos - np.cos(2.0 * np.pi * (i2.astype(np.float64) * 2.0 ** -53)))) < 4e-15


def test_irwin_hall_normal_moments():
    # Irwin-Hall(12) - 6 (plan-side numbers) has mean 0, variance exactly 1, support [-6, 6]
    x = synth.normal_np(synth.stream_key(1, 1), np.arange(1_000_000))
    assert abs(x.mean()) < 5e-3
    assert abs(x.var() - 1.0) < 5e-3
    assert x.min() >= -6 and x.max() <= 6
    # fourth moment of IH(12)-6: 3 - 1.2/12 = 2.9
    assert abs(np.mean(x ** 4) - 2.9) < 0.03


def test_workers_are_independent_streams():
    wl = synth.workload("iid-n8-c16-16m")
    idx = np.arange(200_000)
    a = wl.values_np(0, idx).astype(np.float64)
    b = wl.values_np(1, idx).astype(np.float64)
    assert abs(np.corrcoef(a, b)[0, 1]) < 0.01
    assert abs(a.std() - 1e-3) < 2e-5                  # N(0, 1e-6)


def test_outliers_are_one_percent_at_100x():
    wl = synth.workload("heavytail-n16-c128")
    idx = np.arange(400_000)
    key = wl.worker_key(3)
    hit = synth.uniform32_np(key, idx, 6) < wl.outlier_threshold
    assert abs(hit.mean() - 0.01) < 1e-3
    v = wl.values_np(3, idx).astype(np.float64)
    base = synth.gauss_np(key, idx)
    np.testing.assert_allclose(v[hit], (base[hit] * 100.0).astype(np.float32), rtol=0)
    np.testing.assert_allclose(v[~hit], base[~hit].astype(np.float32), rtol=0)


def test_model_shapes():
    g = synth.gpt2_small_tensor_sizes()
    assert len(g) == 148 and sum(g) == 124_439_808
    p = synth.pythia_1_4b_tensor_sizes()
    assert len(p) == 292 and sum(p) == 1_414_647_808
    assert synth.workload("pythia-1.4b").d == 1_414_647_808 and synth.workload("gpt2-small").d == 124_439_808


def test_per_tensor_scales_are_lognormal_and_shared():
    wl = synth.workload("pythia-1.4b")
    s = wl.tensor_scales().astype(np.float64)
    z = np.log(s)
    assert len(s) == 292
    assert abs(z.mean()) < 0.25 and abs(z.std() - 1.0) < 0.2
    # the scale applies to a whole tensor: the ratio value / normal is constant inside it
    off = np.concatenate([[0], np.cumsum(synth.pythia_1_4b_tensor_sizes())])
    t = 5
    idx = np.arange(off[t], off[t] + 1000)
    for w in (0, 7):
        ratio = wl.values_np(w, idx).astype(np.float64) / synth.gauss_np(wl.worker_key(w), idx)
        np.testing.assert_allclose(ratio, s[t], rtol=1e-6)


def test_ddp_buckets_cover_the_gradient():
    sizes = synth.gpt2_small_tensor_sizes()
    b = synth.ddp_buckets(sizes)
    assert len(b) == 17
    d = sum(sizes)
    pos = 0
    offsets = set(np.concatenate([[0], np.cumsum(sizes)]).tolist())
    for off, ln in b:
        assert off == pos and ln > 0
        assert off in offsets and off + ln in offsets      # buckets hold whole tensors
        pos += ln
        if ln > synth.DDP_BUCKET_FLOATS:                   # only a single oversize tensor
            assert ln in sizes
    assert pos == d
    assert synth.workload("gpt2-small").buckets == b


def test_base_matrix_is_seeded():
    a = synth.base_matrix(7, 8, 64)
    assert a.shape == (8, 64) and a.dtype == np.float64
    np.testing.assert_array_equal(a, synth.base_matrix(7, 8, 64))
    assert not np.array_equal(a, synth.base_matrix(8, 8, 64))
    assert math.isclose(float(np.std(synth.base_matrix(1, 64, 64))), 1.0, rel_tol=0.05)


def test_node_permutations():
    """Row 0 is the identity, every row is a permutation of 0..c-1, rows are
    distinct, and the table is a pure function of (seed, count, c)."""
    P = synth.node_permutations(3, 40, 16)
    assert P.shape == (40, 16) and P.dtype == np.int32
    np.testing.assert_array_equal(P[0], np.arange(16))
    for row in P:
        np.testing.assert_array_equal(np.sort(row), np.arange(16))
    assert len({tuple(r) for r in P}) == 40
    np.testing.assert_array_equal(P, synth.node_permutations(3, 40, 16))
    np.testing.assert_array_equal(P[:7], synth.node_permutations(3, 7, 16))
    assert not np.array_equal(P, synth.node_permutations(4, 40, 16))
