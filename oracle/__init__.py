"""Plain fp64 CPU oracle for CERAR, the coded approximate ring all-reduce.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or
links this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it.  It shares no code with the
HIP library (``paper_2609_23898_amd``) and imports nothing from it; both sides
receive their inputs as plain arrays.

Contents
--------
``oracle.plan``  the encoding/decoding matrices (U, R): the multiplicative
                 perturbation construction, the Vandermonde and O(eps) choices
                 of its base and perturbation, the coefficient maps M_i, the
                 least-squares objective Phi, condition numbers, and the
                 condition-number-constrained alternating least-squares design.
``oracle.ring``  the protocol itself: chunking, linear encode, Algorithm 1 run
                 in lock-step over N workers with copied messages, a second
                 closed-form route for the stored observations, the linear
                 decode and the error metrics.

Everything is float64, written for readability rather than speed; each
function cites the passage of the paper (Munim & Ramamoorthy, "Communication-
Efficient Distributed Training via Ring-Based Coded Approximate All-Reduce")
that it follows.

Parity status: every function is pinned by a ``-m "not gpu"`` test against a
fact the paper or the mathematics fixes (worked example of Sec. II-A, printed
M_0/M_1, Propositions 1-2, Theorem 1, eq. (14), Lemma 1, Corollary 1, the
exact c = N case, brute-force sums, one-hot inputs, linearity, counted rounds
and rates), except the quality of the alternating least-squares design (the
value of Phi it reaches), which is "parity unpinned": the paper prints no
fitted (U, R) or Phi; only its optimality conditions and the condition-number
guarantee are pinned.
"""
