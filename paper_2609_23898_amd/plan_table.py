"""Plan quality of the condition-number-constrained design (Sec. II-D) over a
grid of (N, c, kappa_max): Phi, the achieved max_i kappa_2(M_i), and the
relative error that Phi predicts for i.i.d. gradients.

For i.i.d. zero-mean gradients of equal variance, worker i's expected squared
error is ||M_i R_i - T||_F^2 times the variance, and the exact sum has
expected squared norm N c times the variance per position, so the mean over
workers of the squared relative error is Phi / (N * N c).

    python -m paper_2609_23898_amd.plan_table [--quick]

prints a Markdown table (plans are built by the library on the host, fp64).
"""

import argparse
import math
import time

from . import cerar as C


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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--quick", action="store_true", help="N <= 8 only")
    ap.add_argument("--iters", type=int, default=100)
    args = ap.parse_args()
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
