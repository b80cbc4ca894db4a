"""Pins of the oracle's plan constructions (oracle.plan): Propositions 1-2,
Theorem 1 and its appendix closed form, the O(eps) bound (14), Lemma 1,
Corollary 1's condition-number exponent, the finite-difference identity of
Appendix E (Example 1), the projection guarantee of Sec. II-D / Appendix G,
and optimality of the two least-squares half-steps."""

import json
import os

import numpy as np
import pytest

from conftest import GOLDEN
from oracle import plan as P
from oracle import ring as RG


def rand_base(rng, N, c):
    return rng.standard_normal((N, c))


# --- the a-sequence and its windows ------------------------------------------

def test_sequence_shift_for_all_integer_indices():
    """a_{l+N} = a_l D for every integer l (eq. (8)), negatives included."""
    rng = np.random.default_rng(1)
    N, c = 3, 5
    B = rand_base(rng, N, c)
    D = np.eye(c) + 0.2 * rng.standard_normal((c, c))
    for ell in range(-3 * N, 3 * N):
        np.testing.assert_allclose(P.mpc_row(B, D, ell + N), P.mpc_row(B, D, ell) @ D,
                                   rtol=1e-12, atol=1e-12)
    for r in range(N):
        np.testing.assert_array_equal(P.mpc_row(B, D, r), B[r])


def test_window_shift():
    """A_{l+N} = A_l D (Sec. II-B)."""
    rng = np.random.default_rng(2)
    N, c = 4, 6
    B = rand_base(rng, N, c)
    D = np.eye(c) + 0.1 * rng.standard_normal((c, c))
    for ell in range(-N, N):
        np.testing.assert_allclose(P.mpc_window(B, D, ell + N), P.mpc_window(B, D, ell) @ D,
                                   rtol=1e-12, atol=1e-12)


def test_finite_difference_example1():
    """F_3 [a; a D; a D^2] = diag(1, eps, eps^2) [a; a H; a H^2] (Appendix E,
    Example 1), with the rows a_l, a_{l+N}, a_{l+2N} of the sequence."""
    fx = json.load(open(os.path.join(GOLDEN, "finite_difference_F3.json")))
    F3 = np.array(fx["F3"], dtype=np.float64)
    assert round(np.linalg.det(F3)) == fx["det"]
    rng = np.random.default_rng(3)
    N, c, eps = 3, 4, 0.05
    B = rand_base(rng, N, c)
    H = rng.standard_normal((c, c))
    D = P.o_eps_perturbation(H, eps)
    for ell in (-4, 0, 2):
        a = P.mpc_row(B, D, ell)
        lhs = F3 @ np.vstack([P.mpc_row(B, D, ell + t * N) for t in range(3)])
        rhs = np.vstack([a, eps * a @ H, eps ** 2 * a @ H @ H])
        np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-12)


# --- Propositions 1 and 2 ------------------------------------------------------

@pytest.mark.parametrize("N,c,diag", [(2, 3, True), (3, 5, False), (4, 7, True), (5, 9, False)])
def test_prop1_block_identity(N, c, diag):
    """U_{i-1-s} W_s(R_i) = I_c if s >= i, else D^{-1}."""
    rng = np.random.default_rng(N * c)
    B = rand_base(rng, N, c)
    if diag:
        D = P.o_eps_perturbation(np.diag(P.chebyshev_nodes(c)), 0.3)
    else:
        D = np.eye(c) + 0.2 * rng.standard_normal((c, c))
    U, R = P.mpc_plan(B, D)
    Dinv = np.linalg.inv(D)
    for i in range(N):
        for s in range(N):
            blk = U[(i - 1 - s) % N] @ R[i][s:s + c]
            np.testing.assert_allclose(blk, np.eye(c) if s >= i else Dinv, atol=1e-9)


@pytest.mark.parametrize("N,c", [(2, 3), (3, 5), (4, 6), (4, 9), (6, 8)])
def test_prop2_phi_closed_form(N, c):
    rng = np.random.default_rng(10 * N + c)
    B = rand_base(rng, N, c)
    for D in (P.o_eps_perturbation(np.diag(P.chebyshev_nodes(c)), 0.2),
              np.eye(c) + 0.15 * rng.standard_normal((c, c))):
        U, R = P.mpc_plan(B, D)
        assert P.phi(U, R) == pytest.approx(P.phi_mpc_closed_form(N, D), rel=1e-8)


# --- Theorem 1 (Vandermonde) -------------------------------------------------

@pytest.mark.parametrize("N,c,tau", [(2, 3, 0.3), (3, 4, 0.2), (4, 5, 0.5), (4, 6, 0.1)])
def test_vandermonde_phi_matches_appendix_closed_form(N, c, tau):
    xi = P.chebyshev_nodes(c)
    B, D = P.vandermonde_base(N, tau, xi)
    U, R = P.mpc_plan(B, D)
    assert P.phi(U, R) == pytest.approx(P.phi_vandermonde_closed_form(N, tau, xi), rel=1e-6)


def test_vandermonde_leading_term_theorem1():
    """Phi = N^3 (N-1)/2 tau^2 sum xi^2 + O(tau^3): the relative gap to the
    leading term shrinks linearly in tau."""
    N, c = 4, 6
    xi = P.chebyshev_nodes(c)
    gaps = []
    for tau in (1e-1, 1e-2, 1e-3):
        exact = P.phi_vandermonde_closed_form(N, tau, xi)
        lead = P.phi_vandermonde_leading_term(N, tau, xi)
        gaps.append(abs(exact / lead - 1.0))
    assert gaps[1] < gaps[0] / 5 and gaps[2] < gaps[1] / 5
    assert gaps[2] < 1e-2


def test_vandermonde_error_shrinks_as_c_grows():
    """With tau_c = 1/c (so tau_c^2 sum xi_j^2 -> 0, Remark 1) the closed-form
    Phi falls monotonically toward 0; for c <= 8 the fp64 plan's numerical Phi
    agrees with it, and the all-reduce error on i.i.d. gradients also falls."""
    N = 4
    closed = [P.phi_vandermonde_closed_form(N, 1.0 / c, P.chebyshev_nodes(c))
              for c in range(N, 257)]
    assert all(b < a for a, b in zip(closed, closed[1:]))
    assert closed[-1] < closed[0] / 50
    rng = np.random.default_rng(0)
    errs = []
    for c in (4, 5, 6, 8):
        xi = P.chebyshev_nodes(c)
        U, R = P.mpc_plan(*P.vandermonde_base(N, 1.0 / c, xi))
        assert P.phi(U, R) == pytest.approx(P.phi_vandermonde_closed_form(N, 1.0 / c, xi), rel=1e-3)
        grads = rng.standard_normal((N, 240 * c))
        out = RG.allreduce(grads, U, R)
        S = RG.exact_sum(grads)
        errs.append(max(RG.relative_error(out[i], S) for i in range(N)))
    assert all(b < a for a, b in zip(errs, errs[1:]))


# --- O(eps) construction (Sec. II-C) ------------------------------------------

def test_o_eps_phi_bound_and_quadratic_scaling():
    rng = np.random.default_rng(4)
    N, c = 4, 9
    B = rand_base(rng, N, c)
    H = np.diag(P.chebyshev_nodes(c))
    phis = []
    for eps in (0.2, 0.1, 0.05, 0.025):
        U, R = P.mpc_plan(B, P.o_eps_perturbation(H, eps))
        ph = P.phi(U, R)
        assert ph <= P.phi_o_eps_bound(N, H, eps) * (1 + 1e-9)
        phis.append(ph / eps ** 2)
    assert max(phis) / min(phis) < 1.5


@pytest.mark.parametrize("N,c", [(2, 3), (3, 7), (4, 5), (8, 16)])
def test_lemma1_phi_positive_when_c_exceeds_N(N, c):
    rng = np.random.default_rng(N + c)
    B = rand_base(rng, N, c)
    H = np.diag(P.chebyshev_nodes(c))
    for eps in (0.5, 1e-2):
        U, R = P.mpc_plan(B, P.o_eps_perturbation(H, eps))
        assert P.phi(U, R) > 0
    U, R = P.kappa_design(B, H, 0.3, 1e3, 5)
    assert P.phi(U, R) > 0


def test_exact_plan_has_zero_phi():
    rng = np.random.default_rng(5)
    for N in (2, 4, 8):
        U, R = P.mpc_plan(rand_base(rng, N, N), np.eye(N))
        assert P.phi(U, R) < 1e-18


# --- Corollary 1: kappa_2(A_l(eps)) = Theta(eps^{-r_star}) -------------------

@pytest.mark.parametrize("N,c", [(4, 5), (3, 7), (2, 7), (4, 8)])
def test_corollary1_condition_number_exponent(N, c):
    rng = np.random.default_rng(100 + N * c)
    B = rand_base(rng, N, c)
    H = np.diag(P.chebyshev_nodes(c) + 1.5)      # nonsingular, distinct diagonal
    rs = P.r_star(N, c)
    e1, e2 = 1e-2, 1e-3
    for ell in range(N):
        k1 = P.kappa2(P.mpc_window(B, P.o_eps_perturbation(H, e1), ell))
        k2 = P.kappa2(P.mpc_window(B, P.o_eps_perturbation(H, e2), ell))
        slope = (np.log(k2) - np.log(k1)) / (np.log(e2) - np.log(e1))
        assert slope == pytest.approx(-rs, abs=0.15)
    U1, _ = P.mpc_plan(B, P.o_eps_perturbation(H, e1))
    U2, _ = P.mpc_plan(B, P.o_eps_perturbation(H, e2))
    for k in range(N):
        slope = (np.log(P.kappa2(U2[k])) - np.log(P.kappa2(U1[k]))) / (np.log(e2) - np.log(e1))
        assert slope == pytest.approx(-rs, abs=0.15)


def test_r_star_and_counts():
    assert P.r_star(8, 64) == 7 and P.r_star(16, 128) == 7 and P.r_star(8, 16) == 1
    assert P.r_star(4, 5) == 1 and P.r_star(4, 4) == 0 and P.r_star(8, 65) == 8
    assert P.num_rounds(4, 5) == 7 and P.num_rounds(8, 64) == 70


# --- constrained design (Sec. II-D) -------------------------------------------

def test_u_step_is_the_minimiser_over_U():
    """Phi(U + t E, R) >= Phi(u_step(R), R) for random directions E, and the
    directional derivative vanishes."""
    rng = np.random.default_rng(6)
    N, c = 3, 5
    B = rand_base(rng, N, c)
    _, R = P.mpc_plan(B, P.o_eps_perturbation(np.diag(P.chebyshev_nodes(c)), 0.3))
    R = R + 0.05 * rng.standard_normal(R.shape)
    U = P.u_step(R, N, c)
    base = P.phi(U, R)
    for _ in range(5):
        E = rng.standard_normal(U.shape)
        t = 1e-4
        up, dn = P.phi(U + t * E, R), P.phi(U - t * E, R)
        assert up >= base and dn >= base
        assert abs(up - dn) / (2 * t) < 1e-6 * max(1.0, base)


def test_r_step_is_the_minimiser_over_R():
    rng = np.random.default_rng(7)
    N, c = 3, 5
    U = rng.standard_normal((N, c, c))
    R = P.r_step(U)
    base = P.phi(U, R)
    for _ in range(5):
        E = rng.standard_normal(R.shape)
        assert P.phi(U, R + 1e-4 * E) >= base and P.phi(U, R - 1e-4 * E) >= base
    for i in range(N):                       # residual orthogonal to range(M_i)
        M = P.coefficient_map(U, i)
        g = M.T @ (M @ R[i] - P.target(N, c))
        assert np.abs(g).max() < 1e-9 * np.abs(M).max() ** 2


def test_projection_bounds_kappa_of_every_M():
    """After clipping every U_k's singular values to [a0, b0],
    kappa_2(M_i) <= sqrt(N) b0 / a0 = kappa_max (Appendix G)."""
    rng = np.random.default_rng(8)
    N, c = 4, 9
    B = rand_base(rng, N, c)
    U, _ = P.mpc_plan(B, P.o_eps_perturbation(np.diag(P.chebyshev_nodes(c)), 1e-3))
    assert P.max_kappa_M(U) > 1e3
    for kmax in (1e2, 1e3):
        Up, (a0, b0) = P.project_singular_values(U, kmax)
        assert np.sqrt(N) * b0 / a0 == pytest.approx(kmax)
        s = np.linalg.svd(Up, compute_uv=False)
        assert s.min() >= a0 * (1 - 1e-12) and s.max() <= b0 * (1 + 1e-12)
        assert P.max_kappa_M(Up) <= kmax * (1 + 1e-9)


@pytest.mark.parametrize("order", ["paper", "projected"])
def test_kappa_design_is_feasible_and_better_than_zero_plan(order):
    rng = np.random.default_rng(9)
    for N, c in [(4, 4), (4, 9), (8, 16)]:
        B = rand_base(rng, N, c)
        U, R = P.kappa_design(B, np.diag(P.chebyshev_nodes(c)), 0.3, 1e3, 30, order=order)
        assert P.max_kappa_M(U) <= 1e3 * (1 + 1e-9)
        # Phi of the trivial decoder R = 0 is ||T||^2 per worker = N * N c
        assert 0 < P.phi(U, R) < N * N * c
        # the returned decoders are the least-squares ones for the returned encoders
        np.testing.assert_allclose(R, P.r_step(U), atol=1e-10)
        # and the encoders lie in the projected set (Sec. II-D)
        s = np.linalg.svd(U, compute_uv=False)
        assert s.max() / s.min() <= 1e3 / np.sqrt(N) * (1 + 1e-9)


def test_kappa_design_orders_share_their_first_u_step():
    """Both orders start from the same O(eps0) plan and the same U-step; with
    one iteration they differ only in whether the R-step saw the projection,
    and the final R-step makes them identical."""
    rng = np.random.default_rng(10)
    B = rand_base(rng, 4, 9)
    H = np.diag(P.chebyshev_nodes(9))
    Ua, Ra = P.kappa_design(B, H, 0.3, 1e3, 1, order="paper")
    Ub, Rb = P.kappa_design(B, H, 0.3, 1e3, 1, order="projected")
    np.testing.assert_allclose(Ua, Ub, atol=1e-12)
    np.testing.assert_allclose(Ra, Rb, atol=1e-10)


def test_vandermonde_base_rows_are_node_powers():
    """b_l(tau) = [z_1^l .. z_c^l] for l = 0..N-1 with z_j = exp(tau xi_j), and
    D_tau = diag(z_j^N) (Sec. II-B).  A column scaling of B leaves Phi and the
    outputs unchanged, so this structural fact is pinned on its own."""
    N, c, tau = 4, 6, 0.3
    xi = P.chebyshev_nodes(c)
    B, D = P.vandermonde_base(N, tau, xi)
    np.testing.assert_array_equal(B[0], np.ones(c))
    np.testing.assert_allclose(B[1], np.exp(tau * xi), rtol=1e-15)
    for ell in range(1, N):
        np.testing.assert_allclose(B[ell] / B[ell - 1], np.exp(tau * xi), rtol=1e-14)
    np.testing.assert_allclose(np.diag(D), np.exp(N * tau * xi), rtol=1e-14)
    assert len(set(np.round(xi, 12))) == c and np.all(np.abs(xi) < 1)


# --- K^(l)(B, H) and gamma (Sec. II-C) -----------------------------------------

def _forward_differences(n):
    """F_n: row k takes the k-th forward difference of a sequence's first n terms."""
    from math import comb
    F = np.zeros((n, n))
    for k in range(n):
        for i in range(k + 1):
            F[k, i] = (-1) ** (k - i) * comb(k, i)
    return F


@pytest.mark.parametrize("N,c", [(2, 5), (3, 7), (4, 8), (4, 10), (5, 5)])
def test_k_matrix_is_the_limit_of_the_differenced_window(N, c):
    """Group the rows a_l .. a_{l+c-1} of A_l(eps) by remainder mod N, take
    forward differences within each class and divide the k-th by eps^k: the
    rows are exactly b_r D^m H^k (D = I + eps H commutes with H), and at
    eps = 0 they are K^(l)(B, H) up to row order (Sec. II-C, eq. (15)).  Also
    pins the class counts n_r(l) and first offsets m_r(l) stated there."""
    rng = np.random.default_rng(400 + N * c)
    B = rand_base(rng, N, c)
    H = np.diag(P.chebyshev_nodes(c)) + 0.2 * rng.standard_normal((c, c))   # D and H commute for any H
    beta, s = divmod(c, N)
    eps = 0.2
    D = P.o_eps_perturbation(H, eps)
    for ell in range(N):
        A = P.mpc_window(B, D, ell)
        E = {(ell + t) % N for t in range(s)}
        limit_rows = []
        for r in range(N):
            idx = [j for j in range(ell, ell + c) if j % N == r]
            assert len(idx) == (beta + 1 if r in E else beta)
            m = 0 if r >= ell else 1
            assert idx[0] == r + N * m
            diffs = _forward_differences(len(idx)) @ A[[j - ell for j in idx]]
            for k in range(len(idx)):
                expect = eps ** k * B[r] @ np.linalg.matrix_power(D, m) @ np.linalg.matrix_power(H, k)
                np.testing.assert_allclose(diffs[k], expect, rtol=0, atol=1e-11)
                limit_rows.append(B[r] @ np.linalg.matrix_power(H, k))
        Kref = np.vstack(limit_rows)
        K = P.k_matrix(B, H, ell)
        assert K.shape == (c, c)
        np.testing.assert_allclose(K.T @ K, Kref.T @ Kref, rtol=1e-12, atol=1e-12)


def test_gamma_special_cases():
    """gamma is homogeneous of degree 1 in B, does not depend on l when N | c,
    and vanishes when H = I makes the blocks of K repeat (beta >= 2)."""
    rng = np.random.default_rng(7)
    N, c = 4, 10
    B = rand_base(rng, N, c)
    H = np.diag(P.chebyshev_nodes(c))
    assert P.gamma(3.0 * B, H) == pytest.approx(3.0 * P.gamma(B, H), rel=1e-12)
    assert P.gamma(B, H) > 0
    assert P.gamma(B, np.eye(c)) < 1e-12
    B8 = rand_base(rng, 4, 8)
    H8 = np.diag(P.chebyshev_nodes(8))
    K0 = P.k_matrix(B8, H8, 0)
    for ell in range(1, 4):
        np.testing.assert_array_equal(P.k_matrix(B8, H8, ell), K0)


def test_node_permutation_keeps_phi_and_tracks_conditioning():
    """Permuting the nodes of a diagonal H leaves D's spectrum and so the
    Prop. 2 value of Phi unchanged, while gamma and the conditioning of the
    maps M_i change: the candidate with the largest gamma is better
    conditioned than the one with the smallest."""
    rng = np.random.default_rng(11)
    N, c, eps = 8, 16, 0.1
    B = rand_base(rng, N, c)
    nodes = P.chebyshev_nodes(c)
    perms = [np.arange(c)] + [rng.permutation(c) for _ in range(15)]
    gammas = [P.gamma(B, np.diag(nodes[p])) for p in perms]
    t, g = P.select_node_permutation(B, nodes, perms)
    assert g == max(gammas) and t == int(np.argmax(gammas))
    phis, kms = [], []
    for p in (perms[t], perms[int(np.argmin(gammas))]):
        D = P.o_eps_perturbation(np.diag(nodes[p]), eps)
        U, R = P.mpc_plan(B, D)
        phis.append(P.phi(U, R))
        kms.append(P.max_kappa_M(U))
    assert phis[0] == pytest.approx(phis[1], rel=1e-9)
    assert phis[0] == pytest.approx(P.phi_mpc_closed_form(N, P.o_eps_perturbation(np.diag(nodes), eps)), rel=1e-9)
    assert kms[0] < kms[1] / 3
