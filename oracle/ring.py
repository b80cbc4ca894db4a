"""The CERAR protocol in plain fp64 NumPy.  Test infrastructure only.

A worker's gradient is a length-d vector; ``to_chunks`` turns it into
G_i (p x c, column l = chunk l).  Encoded vectors Delta_i = G_i U_i are kept
as p x c arrays whose column j is the paper's delta_{i,j+1}.  Stored
observations Y_i are p x (L+1) arrays whose column k is y_{i,k+1}.

Every operation acts on each position e in [0, p) separately, so the same
functions also run on any subset of positions: pass the rows of G_i for those
positions only.
"""

import numpy as np


def chunk_len(d, c, align=1):
    """Chunk (message) length p.  The gradient is zero-padded until it splits
    into c chunks of p entries (Sec. II); the padding only has to make
    c p >= d, so p = ceil(d / c) is the least choice (align = 1) and any larger
    p works the same way.  With align > 1, p is ceil(d / c) rounded up to a
    multiple of align."""
    p = -(-d // c)
    return -(-p // align) * align


def exact_sum(grads):
    """The target of the all-reduce, S = sum_w g_w, in fp64 (Sec. I and
    eq. (1); the 1/N~ scaling is already inside each worker's gradient)."""
    return np.sum(np.asarray(grads, dtype=np.float64), axis=0)


def to_chunks(g, c, align=1):
    """G_i = [g[0] .. g[c-1]] in R^{p x c}, column l = g[l p:(l+1) p], with the
    tail beyond d set to zero (Sec. II); p = chunk_len(d, c, align)."""
    g = np.asarray(g, dtype=np.float64).ravel()
    d = g.size
    p = chunk_len(d, c, align)
    padded = np.zeros(c * p)
    padded[:d] = g
    return padded.reshape(c, p).T


def from_chunks(G, d):
    """Inverse of ``to_chunks``: concatenate the c columns and drop the pad."""
    return np.asarray(G).T.reshape(-1)[:d]


def encode(G, U):
    """Delta_i = G_i U_i, i.e. delta_{i,j} = sum_l U_i[l, j] g_i[l] (Sec. II)."""
    return np.asarray(G, dtype=np.float64) @ np.asarray(U, dtype=np.float64)


def run_protocol(Delta, trace=None):
    """Algorithm 1 at every worker, all N workers in lock-step (Sec. II).

    ``Delta`` is a list of N arrays (p x c).  Messages are copied from sender
    to receiver.  Returns (Y, stats): Y[i] is the p x (L+1) matrix
    [B_{i,1} .. B_{i,N-1} | D_{i,1} .. D_{i,c}] and stats counts rounds and the
    floats each worker sent.  If ``trace`` is a list, one dict per round is
    appended with the transmitted x_{i,k}, the rolling states sigma_{i,k} and
    copies of the D and B buffers after the round.
    """
    N = len(Delta)
    p, c = np.asarray(Delta[0]).shape
    L = c + N - 2
    # initialisation: D_{i,j} <- delta_{i,j}; C_i <- sigma_{i,0} = 0
    D = [[np.array(Delta[i][:, j], dtype=np.float64) for j in range(c)]
         for i in range(N)]
    Bstore = [[None] * (N - 1) for _ in range(N)]
    C = [np.zeros(p) for _ in range(N)]
    sent_floats = [0] * N
    for k in range(1, L + 1):
        # Step 1: accumulate and transmit
        sent = []
        for i in range(N):
            if k <= c:
                C[i] = C[i] + D[i][k - 1]
            sent.append(C[i].copy())
            sent_floats[i] += p
        # Step 2: receive, store, update
        for i in range(N):
            C[i] = sent[(i - 1) % N].copy()
            if k <= N - 1:
                Bstore[i][k - 1] = C[i].copy()
            else:
                j = k - N + 1
                C[i] = C[i] - D[i][j - 1]        # cancel the returning own term
                D[i][j - 1] = D[i][j - 1] + C[i]  # D_{i,j} now holds x_{i-1,k}
        if trace is not None:
            trace.append({"k": k,
                          "x": [s.copy() for s in sent],
                          "sigma": [ci.copy() for ci in C],
                          "D": [[v.copy() for v in D[i]] for i in range(N)],
                          "B": [[None if v is None else v.copy() for v in Bstore[i]]
                                for i in range(N)]})
    Y = [np.column_stack(Bstore[i] + D[i]) for i in range(N)]
    stats = {"rounds": L, "message_len": p, "sent_floats": sent_floats,
             "slots_per_worker": c + (N - 1) + 1}
    return Y, stats


def observations_closed_form(Delta):
    """Second route to Y_i, from unrolling the update equations (eq. (2)):
    y_{i,k} = sum_{t=0}^{N-1} delta_{i-1-t, k-t} for k = 1..L+1, with
    delta_{w,j} = 0 for j outside 1..c.  Column k of M_i (eq. (6)) says the same."""
    N = len(Delta)
    p, c = np.asarray(Delta[0]).shape
    L = c + N - 2
    Y = []
    for i in range(N):
        cols = []
        for k in range(1, L + 2):
            y = np.zeros(p)
            for t in range(N):
                j = k - t
                if 1 <= j <= c:
                    y = y + np.asarray(Delta[(i - 1 - t) % N][:, j - 1], dtype=np.float64)
            cols.append(y)
        Y.append(np.column_stack(cols))
    return Y


def decode(Y, R):
    """g_hat_i = Y_i R_i (Sec. II-A): column m approximates chunk m of the sum."""
    return np.asarray(Y, dtype=np.float64) @ np.asarray(R, dtype=np.float64)


def allreduce_chunks(G_list, U, R):
    """Encode, Algorithm 1 and decode for chunked inputs (list of p x c).
    Returns the list of g_hat_i as p x c arrays."""
    Delta = [encode(G_list[i], U[i]) for i in range(len(G_list))]
    Y, _ = run_protocol(Delta)
    return [decode(Y[i], R[i]) for i in range(len(G_list))]


def allreduce(grads, U, R, align=1):
    """Full pipeline on length-d gradients (N x d); returns g_hat (N x d).
    `align` sets the chunk length (chunk_len)."""
    grads = np.asarray(grads)
    N, d = grads.shape
    c = U.shape[1]
    G_list = [to_chunks(grads[i], c, align) for i in range(N)]
    ghat = allreduce_chunks(G_list, U, R)
    return np.stack([from_chunks(ghat[i], d) for i in range(N)])


def relative_error(approx, exact):
    """||approx - exact||_2 / ||exact||_2, the metric of Table 3 (per worker;
    the paper reports its maximum over workers)."""
    approx = np.asarray(approx, dtype=np.float64)
    exact = np.asarray(exact, dtype=np.float64)
    return float(np.linalg.norm(approx - exact) / np.linalg.norm(exact))
