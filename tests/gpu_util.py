"""Shared helpers of the GPU parity tests: device buffers, slot reads, and the
oracle run on the same seeded inputs."""

import numpy as np

from oracle import plan as OP
from oracle import ring as OR
from paper_2609_23898_amd import cerar as C
from paper_2609_23898_amd import synth

U32 = 2.0 ** -24
CHUNK_ALIGN = 32          # the library pads chunks to multiples of 32 floats (cerar_chunk_len)


def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    return torch, "cuda:0"


def host_grads(N, d, seed, scale=1.0, outlier_prob=0.0):
    w = synth.Workload("test", N, N, d, seed=seed, scale=scale, outlier_prob=outlier_prob,
                       outlier_factor=100.0)
    return np.stack([w.values_np(i, np.arange(d)) for i in range(N)])


def to_device(a, ld=None, align_elems=0):
    """(N, d) float32 array -> (N, ld) device tensor view (row stride ld)."""
    torch, dev = torch_dev()
    N, d = a.shape
    ld = ld or d
    buf = torch.zeros(N * ld + align_elems, dtype=torch.float32, device=dev)
    t = buf[align_elems:].view(N, ld)
    t[:, :d] = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
    return t


def buffers(plan, d, ld_work=None, ld_out=None, work_offset=0, out_offset=0, ws_offset=0):
    torch, dev = torch_dev()
    p, stride = plan.chunk_len(d)
    ld_work = ld_work or plan.c * p
    ld_out = ld_out or d
    work = torch.full((plan.N * ld_work + work_offset,), float("nan"), dtype=torch.float32,
                      device=dev)[work_offset:].view(plan.N, ld_work)
    nbytes = plan.workspace_bytes(d)
    ws = torch.zeros(nbytes + 4 * ws_offset, dtype=torch.uint8, device=dev)[4 * ws_offset:]
    out = torch.full((plan.N * ld_out + out_offset,), float("nan"), dtype=torch.float32,
                     device=dev)[out_offset:].view(plan.N, ld_out)
    return work, ws, out


def read_slot(plan, d, work, ws, s):
    """Host copy of the p floats of slot s."""
    torch, _ = torch_dev()
    p, stride = plan.chunk_len(d)
    Nc = plan.N * plan.c
    if s < Nc:
        w, l = divmod(s, plan.c)
        return work[w, l * p:(l + 1) * p].double().cpu().numpy()
    wsf = ws.view(torch.float32)
    q = s - Nc
    return wsf[q * stride:q * stride + p].double().cpu().numpy()


def oracle_allreduce(grads, U, R):
    """The oracle with the library's chunk length."""
    return OR.allreduce(grads, U, R, align=CHUNK_ALIGN)


def oracle_chunks(g, c):
    return OR.to_chunks(g, c, align=CHUNK_ALIGN)


def rel_l2(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / nb) if nb > 0 else float(np.linalg.norm(a - b))


def max_rel_l2(gpu, ref):
    return max(rel_l2(gpu[i], ref[i]) for i in range(len(ref)))


def orthogonal_plan(N, c, seed):
    """A well-conditioned explicit plan: random orthogonal U_k and the
    least-squares decoders R_i for them (oracle r_step)."""
    rng = np.random.default_rng(seed)
    U = np.stack([np.linalg.qr(rng.standard_normal((c, c)))[0] for _ in range(N)])
    R = OP.r_step(U)
    return U, R


def mpc_plan(N, c, eps, seed):
    B = synth.base_matrix(seed, N, c)
    D = OP.o_eps_perturbation(np.diag(OP.chebyshev_nodes(c)), eps)
    return OP.mpc_plan(B, D)


def gate(kappa_M):
    """Parity bar: relative l2 <= 1e-4 for plans with kappa_2(M) <= 1e3;
    larger condition numbers are reported against a looser bound that grows
    with kappa (fp32 rounding amplified by the decode)."""
    if kappa_M <= 1e3:
        return 1e-4
    return max(1e-4, 64 * kappa_M * U32)


def f32(x):
    """Round to fp32 and back to fp64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def fp32_observations(Delta, one_rounding=True):
    """Y_i of Algorithm 1 with every message held in fp32 (the wire format):
    x_{i,k+1} = recv + delta_{i,k+1} for k < N, recv - delta_{i,j}
    (+ delta_{i,k+1}) for k >= N, rounded once per round (or once per
    operation), all other arithmetic exact.  Delta: N arrays (p, c)."""
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


def fp32_protocol_floor(g, U, R):
    """Relative l2 error, against the fp64 oracle, of the protocol itself run
    with fp32 coefficients, fp32-stored encoded chunks and fp32 messages
    (one rounding per round), encode and decode otherwise exact: what any
    implementation with fp32 messages carries.  g: (N, d) host gradients."""
    N = g.shape[0]
    c = U.shape[1]
    G = [oracle_chunks(g[i], c) for i in range(N)]
    ref = OR.allreduce_chunks(G, U, R)
    Uf, Rf = f32(U), f32(R)
    Y = fp32_observations([f32(G[i] @ Uf[i]) for i in range(N)], True)
    return max(np.linalg.norm(Y[i] @ Rf[i] - ref[i]) / np.linalg.norm(ref[i]) for i in range(N))
