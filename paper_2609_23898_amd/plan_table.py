"""Plan quality of the condition-number-constrained design (Sec. II-D) over a
grid of (N, c, kappa_max): Phi, the achieved max_i kappa_2(M_i), and the
relative error that Phi predicts for i.i.d. gradients.

For i.i.d. zero-mean gradients of equal variance, worker i's expected squared
error is ||M_i R_i - T||_F^2 times the variance, and the exact sum has
expected squared norm N c times the variance per position, so the mean over
workers of the squared relative error is Phi / (N * N c).

    python -m paper_2609_23898_amd.plan_table [--quick]
    python -m paper_2609_23898_amd.plan_table --o-eps [--candidates 64]

prints a Markdown table (plans are built by the library on the host, fp64).
With --o-eps it compares O(eps) plans with H = diag(nodes) against the H
chosen by gamma among node permutations (Sec. II-C assumption): same Phi,
different conditioning.
"""

import argparse
import math
import time

from . import cerar as C
from . import synth


def rows(grid, iters, orders):
    for N, c, kmax in grid:
        for order in orders:
            t = time.perf_counter()
            plan = C.Plan(N, c, "kappa", kmax, seed=1000 + N, eps0=0.3, als_iters=iters, als_order=order)
            info = plan.info()
            dt = time.perf_counter() - t
            yield {"N": N, "c": c, "kappa_max": kmax, "order": order, "phi": info["phi"],
                   "phi_initial": info["phi_initial"], "kappa_M": info["kappa_M"],
                   "rel_err": math.sqrt(info["phi"] / (N * N * c)), "comm_rate": info["comm_rate"],
                   "seconds": dt}
            plan.close()


def o_eps_rows(grid, candidates):
    for N, c, eps in grid:
        perms = synth.node_permutations(7, candidates, c)
        base = synth.base_matrix(1000 + N, N, c)
        t = time.perf_counter()
        a = C.Plan(N, c, "o_eps", eps, base=base)
        b = C.Plan(N, c, "o_eps", eps, base=base, node_perms=perms)
        ia, ib = a.info(), b.info()
        yield {"N": N, "c": c, "eps": eps, "phi": ib["phi"], "gamma0": ia["gamma"], "gamma": ib["gamma"],
               "kappa0": ia["kappa_M"], "kappa": ib["kappa_M"], "choice": ib["h_choice"],
               "seconds": time.perf_counter() - t}
        a.close()
        b.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--quick", action="store_true", help="N <= 8 only")
    ap.add_argument("--iters", type=int, default=100)
    ap.add_argument("--o-eps", action="store_true", help="O(eps) plans: H = diag(nodes) vs the largest-gamma H")
    ap.add_argument("--candidates", type=int, default=64)
    args = ap.parse_args()
    if args.o_eps:
        grid = [(N, c, eps) for N in ((4, 8) if args.quick else (4, 8, 16)) for c in (N * 2, N * 2 + N // 2, N * 4)
                for eps in (1e-2, 1e-1) if c <= 128]
        print("| N | c | eps | Phi | gamma, H = diag(nodes) | kappa_2(M_i) | gamma, chosen H | kappa_2(M_i) | candidate | s |")
        print("|---|---|---|---|---|---|---|---|---|---|")
        for r in o_eps_rows(grid, args.candidates):
            print(f"| {r['N']} | {r['c']} | {r['eps']:.0e} | {r['phi']:.4g} | {r['gamma0']:.3g} | {r['kappa0']:.3g} | "
                  f"{r['gamma']:.3g} | {r['kappa']:.3g} | {r['choice']} | {r['seconds']:.1f} |", flush=True)
        return
    Ns = (4, 8) if args.quick else (4, 8, 16)
    grid = []
    for N in Ns:
        for mult in (2, 4, 8):
            c = N * mult
            if c > 128:
                continue
            for kmax in (1e2, 1e3, 1e4):
                grid.append((N, c, kmax))
    print("| N | c | kappa_max | ALS order | comm rate | Phi (start) | Phi | max kappa_2(M_i) | rel. error (iid) | s |")
    print("|---|---|---|---|---|---|---|---|---|---|")
    for r in rows(grid, args.iters, (0, 1)):
        print(f"| {r['N']} | {r['c']} | {r['kappa_max']:.0e} | {r['order']} | {r['comm_rate']:.3f} | "
              f"{r['phi_initial']:.4g} | {r['phi']:.4g} | {r['kappa_M']:.3g} | {r['rel_err']:.3f} | "
              f"{r['seconds']:.1f} |", flush=True)


if __name__ == "__main__":
    main()
