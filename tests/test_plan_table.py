"""The plan-quality table tool: every kappa-designed plan meets its bound,
the rates are the paper's, and in the O(eps) mode the chosen node
permutation never lowers gamma (the identity is a candidate) nor changes Phi
(a permutation of diagonal H leaves D's spectrum, Prop. 2)."""

import math

from paper_2609_23898_amd import plan_table as T


def test_kappa_rows_meet_their_bound():
    grid = [(4, 8, 1e2), (4, 10, 1e3), (8, 16, 1e3)]
    rows = list(T.rows(grid, iters=3, orders=(0, 1)))
    assert len(rows) == 2 * len(grid)
    for r in rows:
        assert r["kappa_M"] <= r["kappa_max"] * (1 + 1e-9), r
        assert math.isclose(r["comm_rate"], (r["c"] + r["N"] - 2) / r["c"], rel_tol=1e-12)
        assert r["phi"] > 0 and math.isfinite(r["phi_initial"])      # c > N: no exact plan (Lemma 1)


def test_o_eps_rows_choose_a_larger_gamma_with_the_same_phi():
    rows = list(T.o_eps_rows([(4, 8, 1e-1), (4, 10, 1e-1)], candidates=8))
    for r in rows:
        assert r["gamma"] >= r["gamma0"], r
        assert 0 <= r["choice"] < 8
        assert r["phi"] > 0
    a = T.C.Plan(4, 8, "o_eps", 1e-1, base=T.synth.base_matrix(1004, 4, 8))
    b = T.C.Plan(4, 8, "o_eps", 1e-1, base=T.synth.base_matrix(1004, 4, 8),
                 node_perms=T.synth.node_permutations(7, 8, 8))
    assert math.isclose(a.info()["phi"], b.info()["phi"], rel_tol=1e-9)
