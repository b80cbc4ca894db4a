"""Pins of the oracle's protocol (oracle.ring) against facts the paper and the
mathematics fix: the worked example of Sec. II-A and Figure 1, the printed
M_0/M_1, brute-force sums, the textbook ring all-reduce special case, one-hot
inputs, linearity, the error bound (5), and the counted rounds and rates."""

import json
import os

import numpy as np
import pytest

from conftest import GOLDEN
from oracle import plan as P
from oracle import ring as RG


def tag_deltas(N, c):
    """delta_{w,j} = unit vector e_{w c + j - 1} of length N c: every message
    then shows, entry by entry, which delta terms it contains."""
    p = N * c
    return [np.eye(p)[:, w * c:(w + 1) * c] for w in range(N)]


def tag_vector(N, c, terms):
    v = np.zeros(N * c)
    for w, j in terms:
        v[w * c + j - 1] += 1.0
    return v


def random_plan(rng, N, c, eps=0.3):
    B = rng.standard_normal((N, c))
    H = np.diag(P.chebyshev_nodes(c))
    D = P.o_eps_perturbation(H, eps)
    U, R = P.mpc_plan(B, D)
    return U, R, D


# --- worked example (Sec. II-A, Figure 1) -----------------------------------

def test_worked_example_messages_and_states():
    fx = json.load(open(os.path.join(GOLDEN, "worked_example_n4_c5.json")))
    N, c, L = fx["N"], fx["c"], fx["L"]
    trace = []
    Y, stats = RG.run_protocol(tag_deltas(N, c), trace=trace)
    assert stats["rounds"] == L == len(trace)
    for key, terms in fx["messages"].items():
        if key == "comment":
            continue
        i, k = map(int, key.split(","))
        np.testing.assert_array_equal(trace[k - 1]["x"][i], tag_vector(N, c, terms))
    for key, val in fx["states"].items():
        if key == "comment":
            continue
        sender, k, w, j = val
        i, kk = map(int, key.split(","))
        assert kk == k
        expect = trace[k - 1]["x"][sender] - tag_vector(N, c, [(w, j)])
        np.testing.assert_array_equal(trace[k - 1]["sigma"][i], expect)
        assert expect.min() == 0.0          # the cancelled term was present
    # round 1: W_i receives delta_{i-1,1}; sigma_{i,1} = delta_{i-1,1}; stored as B_{i,1}
    for i in range(N):
        d = tag_vector(N, c, [((i - 1) % N, 1)])
        np.testing.assert_array_equal(trace[0]["sigma"][i], d)
        np.testing.assert_array_equal(Y[i][:, 0], d)
    # round 6 at W_0
    r6 = fx["round6_worker0"]
    np.testing.assert_array_equal(trace[5]["x"][3], tag_vector(N, c, r6["received"]))
    np.testing.assert_array_equal(trace[5]["sigma"][0], tag_vector(N, c, r6["kept"]))
    # stored observations of W_0
    ob = fx["observations_worker0"]
    np.testing.assert_array_equal(Y[0][:, 3], tag_vector(N, c, ob["y_0_4"]))
    np.testing.assert_array_equal(Y[0][:, 7], tag_vector(N, c, ob["y_0_8"]))
    # D_{i,1} holds x_{i-1,4} after round 4 and is not overwritten later
    for i in range(N):
        np.testing.assert_array_equal(Y[i][:, N - 1], trace[3]["x"][(i - 1) % N])


def test_printed_coefficient_maps_match_protocol():
    """The M_0, M_1 printed in Sec. II-A, the block-row formula (6), and M_i
    read off the protocol itself from one-hot gradients all agree."""
    fx = json.load(open(os.path.join(GOLDEN, "coefficient_maps_n4_c5.json")))
    N, c = fx["N"], fx["c"]
    rng = np.random.default_rng(5)
    U = rng.standard_normal((N, c, c))
    for name, rows in fx["block_rows"].items():
        if name == "comment":
            continue
        i = int(name.split("_")[1])
        M = P.coefficient_map(U, i)
        assert M.shape == (N * c, fx["columns"])
        for r, (lead, k, trail) in enumerate(rows):
            blk = M[r * c:(r + 1) * c]
            assert lead + c + trail == fx["columns"]
            np.testing.assert_array_equal(blk[:, :lead], 0.0)
            np.testing.assert_array_equal(blk[:, lead:lead + c], U[k])
            np.testing.assert_array_equal(blk[:, lead + c:], 0.0)
    # M_i from the protocol: gradient of worker w = e_l (p = 1, chunk l)
    for i in range(N):
        M_emp = np.zeros((N * c, c + N - 1))
        for w in range(N):
            for ell in range(c):
                G = [np.zeros((1, c)) for _ in range(N)]
                G[w][0, ell] = 1.0
                Y, _ = RG.run_protocol([RG.encode(G[v], U[v]) for v in range(N)])
                r = (w - i) % N
                M_emp[r * c + ell] = Y[i][0]
        np.testing.assert_allclose(M_emp, P.coefficient_map(U, i), rtol=0, atol=1e-12)


@pytest.mark.parametrize("N,c", [(2, 2), (2, 5), (3, 3), (3, 7), (4, 5), (5, 9), (8, 16)])
def test_three_routes_to_observations(N, c):
    """Algorithm 1 (copied messages) = unrolled update equations (2) = the
    coefficient map route Y_i = [G_i | .. | G_{i+N-1}] M_i."""
    rng = np.random.default_rng(N * 100 + c)
    U = rng.standard_normal((N, c, c))
    p = 11
    G = [rng.standard_normal((p, c)) for _ in range(N)]
    Delta = [RG.encode(G[i], U[i]) for i in range(N)]
    Y1, _ = RG.run_protocol(Delta)
    Y2 = RG.observations_closed_form(Delta)
    for i in range(N):
        calG = np.hstack([G[(i + r) % N] for r in range(N)])
        Y3 = calG @ P.coefficient_map(U, i)
        scale = np.abs(Y3).max()
        np.testing.assert_allclose(Y1[i], Y2[i], rtol=0, atol=1e-12 * scale)
        np.testing.assert_allclose(Y1[i], Y3, rtol=0, atol=1e-12 * scale)


# --- exact special cases ----------------------------------------------------

@pytest.mark.parametrize("N,d", [(2, 7), (3, 100), (4, 4097), (6, 60)])
def test_exact_case_c_equals_N_is_the_sum(N, d):
    """c = N with D = I is exact (Sec. II-B: plain ring all-reduce has zero
    error): brute-force sum over workers, any nonsingular B."""
    rng = np.random.default_rng(d)
    B = rng.standard_normal((N, N))
    U, R = P.mpc_plan(B, np.eye(N))
    assert P.phi(U, R) < 1e-20
    grads = rng.standard_normal((N, d)).astype(np.float32)
    brute = np.zeros(d)
    for w in range(N):
        for e in range(d):
            brute[e] += float(grads[w, e])
    out = RG.allreduce(grads, U, R)
    for i in range(N):
        np.testing.assert_allclose(out[i], brute, rtol=0, atol=1e-9 * np.abs(brute).max())


def test_textbook_ring_allreduce_schedule():
    """B = I_N, c = N, D = I: every U_k is a permutation, every message carries
    one chunk index only (reduce-scatter then all-gather), L = 2(N-1) and each
    worker sends 2(N-1) d/N floats (Sec. II, problem formulation)."""
    N = 5
    U, R = P.mpc_plan(np.eye(N), np.eye(N))
    for k in range(N):
        assert np.array_equal(np.sort(U[k].ravel())[-N:], np.ones(N))
        np.testing.assert_array_equal(U[k] @ U[k].T, np.eye(N))
    # tag inputs: gradient chunk l of worker w is the unit vector of (w, l)
    G = [np.eye(N * N)[:, w * N:(w + 1) * N] for w in range(N)]
    trace = []
    Y, stats = RG.run_protocol([RG.encode(G[w], U[w]) for w in range(N)], trace=trace)
    assert stats["rounds"] == 2 * (N - 1)
    d = N * N * N                                   # p = N^2 positions, c = N chunks
    assert all(s == 2 * (N - 1) * d // N for s in stats["sent_floats"])
    for rec in trace:
        for x in rec["x"]:
            chunks = {idx % N for idx in np.nonzero(x)[0]}
            assert len(chunks) == 1
    out = [RG.decode(Y[i], R[i]) for i in range(N)]
    S = sum(G)
    for i in range(N):
        np.testing.assert_allclose(out[i], S, atol=1e-12)


def test_mpc_output_matches_prop1_closed_form():
    """Encode + Algorithm 1 + decode with an MPC plan equals
    g_hat_i = sum_{w>=i} G_w + (sum_{w<i} G_w) D^{-1}; worker 0 is exact."""
    rng = np.random.default_rng(11)
    for N, c in [(2, 3), (3, 5), (4, 7), (5, 6)]:
        U, R, D = random_plan(rng, N, c, eps=0.2)
        G = [rng.standard_normal((13, c)) for _ in range(N)]
        out = RG.allreduce_chunks(G, U, R)
        ref = P.mpc_output_closed_form(G, D)
        for i in range(N):
            np.testing.assert_allclose(out[i], ref[i], rtol=0, atol=1e-9)
        np.testing.assert_allclose(out[0], sum(G), rtol=0, atol=1e-9)


def test_non_diagonal_perturbation_closed_form():
    rng = np.random.default_rng(12)
    N, c = 3, 5
    B = rng.standard_normal((N, c))
    D = np.eye(c) + 0.1 * rng.standard_normal((c, c))
    U, R = P.mpc_plan(B, D)
    G = [rng.standard_normal((4, c)) for _ in range(N)]
    out = RG.allreduce_chunks(G, U, R)
    ref = P.mpc_output_closed_form(G, D)
    for i in range(N):
        np.testing.assert_allclose(out[i], ref[i], atol=1e-9)


# --- one-hot, linearity, bound, counts --------------------------------------

def test_one_hot_gradient_gives_rows_of_MR():
    """g_w = 1 at (chunk l, position e), all else 0: worker i's output at e is
    row r c + l of M_i R_i with r = (w - i) mod N; every other position is 0."""
    rng = np.random.default_rng(3)
    N, c, p = 4, 6, 5
    U, R, _ = random_plan(rng, N, c)
    for w in range(N):
        for ell in range(c):
            e = (w + ell) % p
            G = [np.zeros((p, c)) for _ in range(N)]
            G[w][e, ell] = 1.0
            out = RG.allreduce_chunks(G, U, R)
            for i in range(N):
                r = (w - i) % N
                row = (P.coefficient_map(U, i) @ R[i])[r * c + ell]
                np.testing.assert_allclose(out[i][e], row, atol=1e-10)
                others = np.delete(out[i], e, axis=0)
                np.testing.assert_array_equal(others, 0.0)


def test_one_hot_observation_gives_rows_of_R():
    rng = np.random.default_rng(4)
    N, c = 3, 5
    _, R, _ = random_plan(rng, N, c)
    L = c + N - 2
    for i in range(N):
        for k in range(L + 1):
            Y = np.zeros((1, L + 1))
            Y[0, k] = 1.0
            np.testing.assert_array_equal(RG.decode(Y, R[i])[0], R[i][k])


def test_linearity():
    rng = np.random.default_rng(7)
    N, c, d = 4, 7, 123
    U, R, _ = random_plan(rng, N, c)
    g = rng.standard_normal((N, d))
    h = rng.standard_normal((N, d))
    a, b = 1.7, -0.3
    lhs = RG.allreduce(a * g + b * h, U, R)
    rhs = a * RG.allreduce(g, U, R) + b * RG.allreduce(h, U, R)
    np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-10 * np.abs(rhs).max())


def test_error_bound_eq5():
    """||g_hat_i - S||_2 <= ||[G_i | .. | G_{i+N-1}]||_2 ||M_i R_i - T||_F."""
    rng = np.random.default_rng(8)
    for N, c in [(3, 5), (4, 9), (2, 6)]:
        U, R, _ = random_plan(rng, N, c, eps=0.5)
        G = [rng.standard_normal((17, c)) for _ in range(N)]
        out = RG.allreduce_chunks(G, U, R)
        S = sum(G)
        for i in range(N):
            calG = np.hstack([G[(i + r) % N] for r in range(N)])
            bound = np.linalg.norm(calG, 2) * np.linalg.norm(P.residual(U, R, i), "fro")
            assert np.linalg.norm(out[i] - S) <= bound * (1 + 1e-12)
            assert np.linalg.norm(out[i] - S) > 0 or i == 0


@pytest.mark.parametrize("N,c,d", [(2, 2, 5), (4, 5, 101), (8, 16, 1000), (3, 10, 7)])
def test_counted_rounds_message_length_and_rates(N, c, d):
    rng = np.random.default_rng(d)
    U, R, _ = random_plan(rng, N, c)
    G = [RG.to_chunks(rng.standard_normal(d), c) for _ in range(N)]
    _, stats = RG.run_protocol([RG.encode(G[i], U[i]) for i in range(N)])
    p = -(-d // c)
    L = c + N - 2
    assert stats["rounds"] == L == P.num_rounds(N, c)
    assert stats["message_len"] == p
    assert all(s == L * p for s in stats["sent_floats"])
    assert stats["sent_floats"][0] / (c * p) == pytest.approx(1 + (N - 2) / c)
    assert stats["sent_floats"][0] / (c * p) == pytest.approx(P.communication_rate(N, c))
    assert stats["slots_per_worker"] * p / (c * p) == pytest.approx(1 + N / c)
    assert P.storage_rate(N, c) == pytest.approx(1 + N / c)


def test_chunking_and_padding():
    g = np.arange(1, 11, dtype=np.float64)       # d = 10, c = 4 -> p = 3, pad 2
    G = RG.to_chunks(g, 4)
    assert G.shape == (3, 4)
    np.testing.assert_array_equal(G[:, 0], [1, 2, 3])
    np.testing.assert_array_equal(G[:, 3], [10, 0, 0])
    np.testing.assert_array_equal(RG.from_chunks(G, 10), g)


def test_padded_chunk_length():
    """A longer chunk length is more zero padding (Sec. II): chunk l is still
    g[l p:(l+1) p], the tail is zero, and the exact plan still returns the
    exact sum; p = ceil(d/c) rounded up to the alignment."""
    g = np.arange(1, 11, dtype=np.float64)       # d = 10, c = 4: p = 3 -> 8 with align 8
    G = RG.to_chunks(g, 4, align=8)
    assert G.shape == (8, 4) and RG.chunk_len(10, 4, 8) == 8
    np.testing.assert_array_equal(G[:, 0], [1, 2, 3, 4, 5, 6, 7, 8])
    np.testing.assert_array_equal(G[:, 1], [9, 10, 0, 0, 0, 0, 0, 0])
    np.testing.assert_array_equal(G[:, 2:], 0)
    np.testing.assert_array_equal(RG.from_chunks(G, 10), g)
    for d, c, a in [(1, 4, 32), (100, 8, 32), (4096, 4, 32), (1001, 7, 32), (64 * 33 + 1, 64, 32)]:
        p = RG.chunk_len(d, c, a)
        assert p % a == 0 and c * p >= d and p - a < -(-d // c) <= p
    rng = np.random.default_rng(12)
    N = 4
    U, R = P.mpc_plan(np.eye(N), np.eye(N))       # exact plan (c = N)
    grads = rng.standard_normal((N, 301))
    for a in (1, 32):
        out = RG.allreduce(grads, U, R, align=a)
        np.testing.assert_allclose(out, np.broadcast_to(RG.exact_sum(grads), out.shape), atol=1e-12)


def test_d_smaller_than_c_and_N2():
    """Degenerate sizes: p = 1 with empty chunks, and the smallest ring."""
    rng = np.random.default_rng(9)
    N, c, d = 2, 5, 3
    D = P.o_eps_perturbation(np.diag(P.chebyshev_nodes(c)), 0.3)
    U, R = P.mpc_plan(rng.standard_normal((N, c)), D)
    grads = rng.standard_normal((N, d))
    out = RG.allreduce(grads, U, R)
    ref = P.mpc_output_closed_form([RG.to_chunks(g, c) for g in grads], D)
    for i in range(N):
        np.testing.assert_allclose(out[i], RG.from_chunks(ref[i], d), atol=1e-9)


def test_exact_sum_and_relative_error():
    grads = np.array([[1.0, 2.0], [3.0, -4.0]], dtype=np.float32)
    np.testing.assert_array_equal(RG.exact_sum(grads), [4.0, -2.0])
    assert RG.relative_error([3.0, 4.0], [0.0, 5.0]) == pytest.approx(np.sqrt(10) / 5)
