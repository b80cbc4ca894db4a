"""Where the fp32 error of the path comes from, at the top of the gated range
(kappa_2(M) = 953: N = 2, c = 64, kappa_max = 1e3 design).

The path is simulated on the CPU in fp64 with chosen roundings to fp32, and
each variant is compared with the plain fp64 oracle (Sec. II: encode,
Algorithm 1, decode).  The check pins the reading behind the 1e-4 gate:
rounding the coefficients and the stored encoded chunks costs little, the
messages of the rounds set the error (a message keeps the rounding of every
earlier round; the returning own term cancels, its rounding does not), and
one rounding per round instead of two lowers it.  The encode and decode
accumulation orders barely matter."""

import numpy as np

from oracle import plan as OP
from oracle import ring as OR
from paper_2609_23898_amd import synth

from gpu_util import host_grads, oracle_chunks

U32 = 2.0 ** -24


def f32(x):
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def observations(Delta, one_rounding):
    """Y_i for all workers with fp32 messages: x_{i,k+1} = recv + delta_{i,k+1}
    (k < N), recv - delta_{i,j} (+ delta_{i,k+1}) otherwise, rounded once per
    round or once per operation."""
    N = len(Delta)
    p, c = Delta[0].shape
    L = c + N - 2
    x = [f32(Delta[i][:, 0]) for i in range(N)]
    Y = [[None] * (L + 1) for _ in range(N)]
    for k in range(1, L + 1):
        recv = [x[(i - 1) % N] for i in range(N)]
        nxt = []
        for i in range(N):
            if k <= N - 1:
                Y[i][k - 1] = recv[i]
                v = f32(recv[i] + Delta[i][:, k])
            else:
                j = k - N + 1
                Y[i][N - 2 + j] = recv[i]
                if k + 1 <= c:
                    v = recv[i] - Delta[i][:, j - 1] + Delta[i][:, k]
                    v = f32(v) if one_rounding else f32(f32(recv[i] - Delta[i][:, j - 1]) + Delta[i][:, k])
                else:
                    v = f32(recv[i] - Delta[i][:, j - 1])
            nxt.append(v)
        x = nxt
    for i in range(N):
        Y[i][L] = Delta[i][:, c - 1]           # D_{i,c} keeps delta_{i,c}
    return [np.column_stack(Y[i]) for i in range(N)]


def test_message_roundings_set_the_error_at_kappa_1e3():
    N, c, d = 2, 64, 64 * 256
    B = synth.base_matrix(N * 1000 + c, N, c)
    U, R = OP.kappa_design(B, np.diag(OP.chebyshev_nodes(c)), 0.3, 1e3, 20)
    kappa = OP.max_kappa_M(U)
    assert 900 <= kappa <= 1e3
    g = host_grads(N, d, seed=N + c)
    G = [oracle_chunks(g[i], c) for i in range(N)]
    ref = OR.allreduce_chunks(G, U, R)
    Uf, Rf = f32(U), f32(R)

    def parity(out):
        return max(np.linalg.norm(out[i] - ref[i]) / np.linalg.norm(ref[i]) for i in range(N)) / (kappa * U32)

    # coefficients in fp32, everything else exact
    coef = parity([OR.decode(OR.observations_closed_form([G[i] @ Uf[i] for i in range(N)])[i], Rf[i])
                   for i in range(N)])
    # + encoded chunks stored in fp32
    Dst = [f32(G[i] @ Uf[i]) for i in range(N)]
    store = parity([OR.decode(OR.observations_closed_form(Dst)[i], Rf[i]) for i in range(N)])
    # + fp32 messages, two roundings per round N <= k < c, and one
    two = parity([observations(Dst, False)[i] @ Rf[i] for i in range(N)])
    one = parity([observations(Dst, True)[i] @ Rf[i] for i in range(N)])
    # + the decode accumulated in fp32, four observations per step
    Y1 = observations(Dst, True)

    def dec32(Y, Rm):
        acc = np.zeros((Y.shape[0], Rm.shape[1]), dtype=np.float32)
        for k0 in range(0, Y.shape[1], 4):
            acc = (acc.astype(np.float64) + Y[:, k0:k0 + 4] @ Rm[k0:k0 + 4]).astype(np.float32)
        return acc.astype(np.float64)

    acc = parity([dec32(Y1[i], Rf[i]) for i in range(N)])
    print(f"kappa={kappa:.4g}; parity / (kappa u): coefficients {coef:.3f}, + stored chunks {store:.3f}, "
          f"+ messages two roundings {two:.3f}, one rounding {one:.3f}, + fp32 decode accumulation {acc:.3f}")
    assert coef < 0.2 and store < 0.3              # rounding the coefficients and the chunks: small
    assert two > 1.3 and two > 5 * store           # the messages set the error
    assert one < 0.9 * two                         # one rounding per round lowers it
    assert abs(acc - one) < 0.15 * one             # the decode's accumulation order barely matters
    assert one * kappa * U32 < 1e-4                # and the gate holds with room
