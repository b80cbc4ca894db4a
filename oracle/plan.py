"""CERAR encoding/decoding matrices, plain fp64 NumPy.  Test infrastructure only.

Array conventions (0-based; the paper's objects in its own notation):

* ``U[k]`` (c x c) is the encoding matrix of worker W_k.  Column j is the
  paper's u_{k,j+1}; row l multiplies gradient chunk l (Sec. II,
  "Initialization": Delta_k = G_k U_k).
* ``R[i]`` ((L+1) x c) is the decoding matrix of W_i.  Row k multiplies the
  stored observation y_{i,k+1}; the paper numbers these rows 0..L (Sec. II-B).
* ``coefficient_map(U, i)`` is M_i (N c x (L+1)); its block row r is
  [0_{c x (N-1-r)}  U_{i+r}  0_{c x r}] with worker indices mod N (eq. (6)).

Readings where the paper leaves a choice open (each one is listed in the
design notes):

* Vandermonde nodes: the paper asks only for distinct reals xi_1..xi_c; the
  default here is the Chebyshev points of the first kind,
  xi_j = cos((2j-1) pi / (2c)), distinct and inside (-1, 1).
* O(eps) direction H: the appendix on the experiments says H is diagonal with
  small entries or derived from B; the default here is H = diag(xi) with the
  same Chebyshev nodes, so ||H||_2 <= 1 and D_eps = I + eps H.  The B-dependent
  choice taken here assigns the nodes to the columns of B: among given
  permutations it takes the one whose H = diag(xi[perm]) has the largest gamma,
  the smallest singular value over the limits K^(l)(B, H) (Sec. II-C
  assumption), so that the windows A_l(eps) and the maps M_i stay
  well-conditioned.
* Constrained design (Sec. II-D): one iteration is a U-step, an R-step, then
  the projection of every U_k's singular values into a common [a0, b0].  The
  interval is centred (geometrically) on the geometric mean s of all current
  singular values, with b0/a0 = kappa_max/sqrt(N), so that
  sqrt(N) b0/a0 = kappa_max.  After the last projection one more R-step makes
  R the least-squares decoder of the returned, feasible U.  The iteration count
  is fixed (no data-dependent stopping), so two implementations of the same
  steps can be compared iterate for iterate.
"""

import numpy as np


# --- counts (Sec. II and Sec. II-B) -----------------------------------------

def num_rounds(N, c):
    """L = c + N - 2 communication rounds (Sec. II)."""
    return c + N - 2


def r_star(N, c):
    """r_star = ceil(c/N) - 1 (Sec. II-C, Corollary 1)."""
    return -(-c // N) - 1


def communication_rate(N, c):
    """Normalised communication rate L/c = 1 + (N-2)/c (Sec. II-B)."""
    return num_rounds(N, c) / c


def storage_rate(N, c):
    """Normalised storage rate 1 + N/c: c encoded slots, N-1 receive slots and
    one rolling slot, each of length d/c (Sec. II-B)."""
    return (c + (N - 1) + 1) / c


def chebyshev_nodes(c):
    """Default distinct reals xi_1..xi_c in (-1, 1) (reading; see module doc)."""
    j = np.arange(1, c + 1, dtype=np.float64)
    return np.cos((2.0 * j - 1.0) * np.pi / (2.0 * c))


# --- multiplicative perturbation construction (Sec. II-B, eqs. (8)-(12)) ----

def mpc_row(B, D, idx):
    """a_idx = b_r D^m where idx = r + m N, 0 <= r < N, for any integer idx
    (eq. (8)); negative m uses powers of D^{-1}."""
    N = B.shape[0]
    m, r = divmod(idx, N)          # floor division: r in [0, N) for every idx
    return B[r] @ np.linalg.matrix_power(D, m)


def mpc_window(B, D, ell):
    """A_ell: the c consecutive rows a_ell .. a_{ell+c-1} (eq. (9))."""
    c = B.shape[1]
    return np.vstack([mpc_row(B, D, ell + t) for t in range(c)])


def mpc_plan(B, D):
    """Encoders and decoders of the multiplicative perturbation construction.

    V_{N-1-k} := A_k and U_k := V_k^{-1} (eq. (10)); R_i[l, :] = a_{l-i} for
    l = 0..L (eq. (11)).  B is the N x c base matrix, D the c x c perturbation.
    """
    B = np.asarray(B, dtype=np.float64)
    D = np.asarray(D, dtype=np.float64)
    N, c = B.shape
    L = num_rounds(N, c)
    U = np.empty((N, c, c))
    R = np.empty((N, L + 1, c))
    for k in range(N):
        V_k = mpc_window(B, D, N - 1 - k)          # V_k = A_{N-1-k}
        U[k] = np.linalg.inv(V_k)
    for i in range(N):
        for ell in range(L + 1):
            R[i, ell] = mpc_row(B, D, ell - i)
    return U, R


def vandermonde_base(N, tau, nodes):
    """Vandermonde choice of (B, D) (Sec. II-B, "A Vandermonde construction"):
    z_j = exp(tau xi_j), b_l = [z_1^l .. z_c^l] for l = 0..N-1, and
    D_tau = diag(z_1^N .. z_c^N)."""
    z = np.exp(tau * np.asarray(nodes, dtype=np.float64))
    B = np.vstack([z ** ell for ell in range(N)])
    D = np.diag(z ** N)
    return B, D


def o_eps_perturbation(H, eps):
    """D_eps = I + eps H (Sec. II-C)."""
    H = np.asarray(H, dtype=np.float64)
    return np.eye(H.shape[0]) + eps * H


# --- coefficient maps and the least-squares objective (Sec. II-B) -----------

def coefficient_map(U, i):
    """M_i(U): block row r is [0_{c x (N-1-r)}  U_{(i+r) mod N}  0_{c x r}]
    (eq. (6)); the printed M_0 and M_1 of Sec. II-A are its N=4, c=5 case."""
    N, c, _ = U.shape
    L = num_rounds(N, c)
    M = np.zeros((N * c, L + 1))
    for r in range(N):
        col0 = N - 1 - r
        M[r * c:(r + 1) * c, col0:col0 + c] = U[(i + r) % N]
    return M


def target(N, c):
    """T = 1_N (Kronecker) I_c (Sec. II-A)."""
    return np.kron(np.ones((N, 1)), np.eye(c))


def residual(U, R, i):
    """M_i R_i - T, the decoding residual of worker i (eq. (5))."""
    N, c, _ = U.shape
    return coefficient_map(U, i) @ R[i] - target(N, c)


def phi(U, R):
    """Phi(U, R) = sum_i ||M_i(U) R_i - T||_F^2 (eq. (7))."""
    return float(sum(np.linalg.norm(residual(U, R, i), "fro") ** 2
                     for i in range(U.shape[0])))


def phi_mpc_closed_form(N, D):
    """Phi of the construction = N(N-1)/2 ||D^{-1} - I_c||_F^2 (Prop. 2, eq. (13))."""
    D = np.asarray(D, dtype=np.float64)
    E = np.linalg.inv(D) - np.eye(D.shape[0])
    return N * (N - 1) / 2.0 * float(np.sum(E * E))


def phi_vandermonde_closed_form(N, tau, nodes):
    """N(N-1)/2 sum_j (exp(-N tau xi_j) - 1)^2 (Appendix C, eq. (19))."""
    xi = np.asarray(nodes, dtype=np.float64)
    return N * (N - 1) / 2.0 * float(np.sum((np.exp(-N * tau * xi) - 1.0) ** 2))


def phi_vandermonde_leading_term(N, tau, nodes):
    """Leading term N^3 (N-1)/2 tau^2 sum_j xi_j^2 of Theorem 1."""
    xi = np.asarray(nodes, dtype=np.float64)
    return N ** 3 * (N - 1) / 2.0 * tau ** 2 * float(np.sum(xi * xi))


def phi_o_eps_bound(N, H, eps):
    """Upper bound N(N-1)/2 eps^2 ||H||_F^2 / (1 - eps ||H||_2)^2 (eq. (14))."""
    H = np.asarray(H, dtype=np.float64)
    h2 = np.linalg.norm(H, 2)
    hf = np.linalg.norm(H, "fro")
    return N * (N - 1) / 2.0 * eps ** 2 * hf ** 2 / (1.0 - eps * h2) ** 2


def kappa2(X):
    """2-norm condition number sigma_max / sigma_min (Sec. II-B, Remark 2)."""
    s = np.linalg.svd(np.asarray(X, dtype=np.float64), compute_uv=False)
    return float(s[0] / s[-1])


def max_kappa_M(U):
    """max_i kappa_2(M_i(U)), the quantity bounded in eq. (16)."""
    return max(kappa2(coefficient_map(U, i)) for i in range(U.shape[0]))


# --- conditioning of the O(eps) windows (Sec. II-C) ---------------------------

def k_matrix(B, H, ell):
    """K^(l)(B, H): B, BH, ..., BH^(beta-1), then (if s > 0) the rows
    r in E_l = {l, ..., l+s-1} (mod N) of BH^beta, where c = beta N + s
    (Sec. II-C; the eps -> 0 limit of the rescaled window rows)."""
    B = np.asarray(B, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    N, c = B.shape
    beta, s = divmod(c, N)
    blocks = [B @ np.linalg.matrix_power(H, j) for j in range(beta)]
    if s:
        E = [(ell + t) % N for t in range(s)]
        blocks.append((B @ np.linalg.matrix_power(H, beta))[E])
    return np.vstack(blocks)


def gamma(B, H):
    """min over l = 0..N-1 of sigma_min(K^(l)(B, H)): the constant of the
    Sec. II-C assumption."""
    N = np.asarray(B).shape[0]
    return min(float(np.linalg.svd(k_matrix(B, H, ell), compute_uv=False)[-1]) for ell in range(N))


def select_node_permutation(B, nodes, perms):
    """Index and gamma of the candidate H_t = diag(nodes[perm_t]) with the
    largest gamma (the first one on ties)."""
    nodes = np.asarray(nodes, dtype=np.float64)
    best, best_t = -1.0, -1
    for t, perm in enumerate(perms):
        g = gamma(B, np.diag(nodes[np.asarray(perm)]))
        if g > best:
            best, best_t = g, t
    return best_t, best


# --- condition-number-constrained design (Sec. II-D, eq. (16)) --------------

def u_step(R, N, c):
    """Minimise Phi over U with R fixed.

    Block row r of M_i R_i is U_{i+r} W_{N-1-r}(R_i) (proof of Lemma 1), so the
    terms that hold U_k are sum_r ||U_k W_r - I_c||_F^2 with
    W_r = W_{N-1-r}(R_{k-r}) (c-row window, Sec. II-B).  Setting the gradient to
    zero gives the normal equations U_k (sum_r W_r W_r^T) = sum_r W_r^T.
    """
    U = np.empty((N, c, c))
    for k in range(N):
        gram = np.zeros((c, c))
        rhs = np.zeros((c, c))
        for r in range(N):
            s = N - 1 - r
            W = R[(k - r) % N][s:s + c, :]
            gram += W @ W.T
            rhs += W.T
        # U_k gram = rhs  <=>  gram^T U_k^T = rhs^T
        U[k] = np.linalg.solve(gram.T, rhs.T).T
    return U


def r_step(U):
    """Minimise Phi over R with U fixed: R_i = argmin ||M_i R - T||_F, an
    ordinary least-squares problem per worker (M_i is N c x (L+1), tall)."""
    N, c, _ = U.shape
    T = target(N, c)
    return np.stack([np.linalg.lstsq(coefficient_map(U, i), T, rcond=None)[0]
                     for i in range(N)])


def projection_interval(U, kappa_max):
    """[a0, b0] with b0/a0 = kappa_max/sqrt(N), geometrically centred on the
    geometric mean of all singular values of U_0..U_{N-1} (reading)."""
    N = U.shape[0]
    s = np.linalg.svd(U, compute_uv=False)
    centre = float(np.exp(np.mean(np.log(s))))
    half = np.sqrt(kappa_max / np.sqrt(N))
    return centre / half, centre * half


def project_singular_values(U, kappa_max):
    """Replace each U_k = P diag(s) Q^T by P diag(clip(s, a0, b0)) Q^T
    (Sec. II-D); then kappa_2(M_i) <= sqrt(N) b0/a0 = kappa_max (Appendix G)."""
    a0, b0 = projection_interval(U, kappa_max)
    P, s, QT = np.linalg.svd(U)
    s = np.clip(s, a0, b0)
    return P @ (s[:, :, None] * QT), (a0, b0)


def kappa_design(B, H, eps0, kappa_max, iters, order="paper"):
    """Alternating least squares for eq. (16), started from the O(eps) plan
    with D = I + eps0 H (Sec. II-D).  Returns (U, R).

    order "paper": each iteration minimises Phi over U (R fixed), then over R
    (U fixed), then projects the singular values of every U_k, as Sec. II-D
    states; a last R-step fits the decoders to the projected encoders.
    order "projected": U-step, projection, R-step, so that every R-step fits
    projected encoders (a variant, not the paper's stated order)."""
    B = np.asarray(B, dtype=np.float64)
    N, c = B.shape
    U, R = mpc_plan(B, o_eps_perturbation(H, eps0))
    for _ in range(iters):
        U = u_step(R, N, c)
        if order == "paper":
            R = r_step(U)
            U, _ = project_singular_values(U, kappa_max)
        else:
            U, _ = project_singular_values(U, kappa_max)
            R = r_step(U)
    if order == "paper":
        R = r_step(U)
    return U, R


def mpc_output_closed_form(G_list, D):
    """Output of an MPC plan in exact arithmetic, from Prop. 1: block r of
    M_i R_i is I_c for workers w = i..N-1 and D^{-1} for w = 0..i-1, hence
    g_hat_i = sum_{w >= i} G_w + (sum_{w < i} G_w) D^{-1}.  Needs no inverse of
    any A_ell, so it stays trustworthy when the plan is ill-conditioned."""
    N = len(G_list)
    Dinv = np.linalg.inv(np.asarray(D, dtype=np.float64))
    out = []
    for i in range(N):
        upper = sum(np.asarray(G_list[w], dtype=np.float64) for w in range(i, N))
        if i > 0:
            lower = sum(np.asarray(G_list[w], dtype=np.float64) for w in range(i))
            upper = upper + lower @ Dinv
        out.append(upper)
    return out
