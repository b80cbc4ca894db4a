"""Parity of the HIP path (through the C ABI) with the fp64 oracle on the same
seeded inputs: each kernel step, the per-round buffer state, and the whole
all-reduce, over vector and scalar layouts, ragged tails, in-place encode,
N = 2 and c = N edge cases, error norms, buckets and the copy kernel."""

import numpy as np
import pytest

from oracle import plan as OP
from oracle import ring as OR
from paper_2609_23898_amd import cerar as C

from gpu_util import (U32, buffers, gate, host_grads, max_rel_l2, mpc_plan, oracle_allreduce, oracle_chunks,
                      orthogonal_plan, read_slot,
                      rel_l2, to_device, torch_dev)

pytestmark = pytest.mark.gpu


def sync():
    torch, _ = torch_dev()
    torch.cuda.synchronize()


# --- K1 encode -------------------------------------------------------------------

@pytest.mark.parametrize("N,c,d", [(4, 4, 4096), (3, 7, 1001), (8, 16, 16 * 777), (2, 64, 64 * 300 + 5),
                                   (4, 128, 128 * 64 + 3)])
def test_encode_with_permutations_is_exact(N, c, d):
    """U_k = permutation matrices: every delta is one input chunk, so the MFMA
    tiles must reproduce the inputs bit for bit (checks the lane layout)."""
    rng = np.random.default_rng(c)
    U = np.stack([np.eye(c)[rng.permutation(c)] for _ in range(N)])
    R = np.zeros((N, c + N - 1, c))
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=1)
    grads = to_device(g)
    work, ws, _ = buffers(plan, d)
    C.encode_round(plan, 0, d, grads, work, ws)
    sync()
    p, _ = plan.chunk_len(d)
    for i in range(N):
        G = oracle_chunks(g[i], c).astype(np.float32)
        expect = G @ U[i].astype(np.float32)
        got = work[i, :c * p].cpu().numpy().reshape(c, p).T
        np.testing.assert_array_equal(got, expect)
        x1 = read_slot(plan, d, work, ws, plan.slot_map(0)[i, c + N - 1])
        np.testing.assert_array_equal(x1, expect[:, 0])


@pytest.mark.parametrize("N,c,d,misalign", [(4, 4, 4096, 0), (3, 7, 1001, 0), (8, 64, 64 * 500 + 7, 0),
                                            (8, 16, 16 * 1024, 1), (2, 128, 128 * 70, 0), (5, 9, 9 * 64, 0),
                                            (2, 128, 128 * 640 - 17, 0)])
def test_encode_matches_oracle_within_dot_product_bound(N, c, d, misalign):
    """|delta_gpu - delta| <= (c + 4) u32 (|G| |U|) elementwise: fp32-rounded
    coefficients, fp32 products and any summation order fit this bound, and
    so do the c = 128 interior blocks, whose products are split into three
    bf16 terms each (the last case: interior blocks and a ragged tail)."""
    U, R = orthogonal_plan(N, c, seed=N + c)
    U = U * np.random.default_rng(1).uniform(0.5, 2.0, size=(N, 1, c))   # not orthogonal any more
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=2)
    grads = to_device(g, align_elems=misalign)
    work, ws, _ = buffers(plan, d, work_offset=misalign)
    C.encode_round(plan, 0, d, grads, work, ws)
    sync()
    p, _ = plan.chunk_len(d)
    for i in range(N):
        G = oracle_chunks(g[i], c)
        exact = OR.encode(G, U[i])
        bound = (c + 4) * U32 * (np.abs(G) @ np.abs(U[i])) + 1e-38
        got = work[i, :c * p].double().cpu().numpy().reshape(c, p).T
        assert np.all(np.abs(got - exact) <= bound)


@pytest.mark.parametrize("N,c,d", [(4, 16, 16 * 1024), (3, 64, 64 * 500 + 7), (4, 128, 128 * 640 - 17),
                                   (2, 128, 128 * 70), (18, 128, 128 * 128)])
def test_decode_matches_oracle_within_dot_product_bound(N, c, d):
    """The decode applied to the device's own observations after round L,
    against the oracle's decode of those observations (Sec. II-A):
    |err| <= (K + 4) u32 (|Y| |R|), K = L + 1.  Covers the c = 128 interior
    kernel on split bf16 operands (K <= 144), its ragged tail, the generic
    kernel alone, and c = 128 with K = 145 (the fp32 wide kernel)."""
    U, R = orthogonal_plan(N, c, seed=N + c + 1)
    R = R * np.random.default_rng(2).uniform(0.5, 2.0, size=(N, R.shape[1], 1))
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=4)
    grads = to_device(g)
    work, ws, out = buffers(plan, d)
    for k in range(plan.L + 1):
        C.encode_round(plan, k, d, grads, work, ws)
    C.decode(plan, d, work, ws, out)
    sync()
    sm = plan.slot_map(plan.L)
    K = plan.L + 1
    got_all = out.double().cpu().numpy()
    for i in range(N):
        cols = [sm[i, c + j] for j in range(N - 1)] + [sm[i, j] for j in range(c)]   # [B_1..B_{N-1} | D_1..D_c]
        Y = np.column_stack([read_slot(plan, d, work, ws, s) for s in cols])
        exact = OR.decode(Y, R[i]).T.reshape(-1)[:d]
        bound = ((K + 4) * U32 * (np.abs(Y) @ np.abs(R[i]))).T.reshape(-1)[:d] + 1e-38
        assert np.all(np.abs(got_all[i] - exact) <= bound), i


# --- K2/K3 rounds: per-round buffer state ---------------------------------------------

@pytest.mark.parametrize("N,c,d", [(4, 5, 5 * 300), (2, 2, 2 * 64), (3, 3, 3 * 101), (8, 16, 16 * 256 + 3),
                                   (4, 9, 9 * 128)])
def test_each_round_matches_algorithm1_state(N, c, d):
    """After step k, the slots the ownership table names for D_{i,j}, B_{i,j}
    and the next message x_{i,k+1} hold the oracle's Algorithm 1 values."""
    U, R = orthogonal_plan(N, c, seed=3)
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=3)
    grads = to_device(g)
    work, ws, out = buffers(plan, d)
    Delta = [OR.encode(oracle_chunks(g[i], c), U[i]) for i in range(N)]
    trace = []
    Y, _ = OR.run_protocol(Delta, trace=trace)
    L = c + N - 2
    for k in range(0, L + 1):
        C.encode_round(plan, k, d, grads, work, ws)
        sync()
        sm = plan.slot_map(k)
        for i in range(N):
            for j in range(c):
                ref = Delta[i][:, j] if k == 0 else trace[k - 1]["D"][i][j]
                assert rel_l2(read_slot(plan, d, work, ws, sm[i, j]), ref) < 1e-5, (k, i, j)
            for j in range(min(k, N - 1)):
                ref = trace[k - 1]["B"][i][j]
                assert rel_l2(read_slot(plan, d, work, ws, sm[i, c + j]), ref) < 1e-5, (k, i, "B", j)
            if k < L:
                ref = trace[k]["x"][i]                                   # x_{i,k+1}
                assert rel_l2(read_slot(plan, d, work, ws, sm[i, c + N - 1]), ref) < 1e-5, (k, i, "x")
    C.decode(plan, d, work, ws, out)
    sync()
    ref = np.stack([OR.from_chunks(OR.decode(Y[i], R[i]), d) for i in range(N)])
    assert max_rel_l2(out.double().cpu().numpy(), ref) < 1e-5


# --- whole ring: gate ---------------------------------------------------------------

CASES = [
    # name, N, c, d, plan kind, param
    ("cfg1-vandermonde", 4, 4, 4096, "vandermonde", 0.5),
    ("cfg1-o_eps", 4, 4, 4096, "o_eps", 1e-3),
    ("cfg1-exact", 4, 4, 4096, "o_eps", 0.0),
    ("N2-c5-ragged", 2, 5, 5 * 333 + 2, "o_eps", 0.2),
    ("N3-c7-odd-p", 3, 7, 7 * 101 + 3, "o_eps", 0.3),
    ("N8-c16-tail", 8, 16, 16 * 4096 + 9, "o_eps", 0.3),
    ("N8-c32", 8, 32, 32 * 2048, "kappa", 1e3),
    ("N8-c64-ragged", 8, 64, 64 * 1536 + 61, "kappa", 1e3),
    ("N13-c64", 13, 64, 64 * 900 + 29, "kappa", 1e3),      # K = 76: the 20-K-step decode
    ("N2-c64", 2, 64, 64 * 700, "kappa", 1e3),             # K = 65: 17 K-steps padded to 18; kappa_M = 953,
                                                           # the top of the gated range
    ("N2-c64-k500", 2, 64, 64 * 700 + 19, "kappa", 5e2),
    ("N16-c128", 16, 128, 128 * 320, "kappa", 1e3),
]


def case_plan(N, c, kind, param):
    if kind == "vandermonde":
        B, D = OP.vandermonde_base(N, param, OP.chebyshev_nodes(c))
        return OP.mpc_plan(B, D)
    if kind == "o_eps":
        return mpc_plan(N, c, param, seed=N * 1000 + c)
    from paper_2609_23898_amd import synth
    B = synth.base_matrix(N * 1000 + c, N, c)
    return OP.kappa_design(B, np.diag(OP.chebyshev_nodes(c)), 0.3, param, 20 if c <= 64 else 4)


@pytest.mark.parametrize("name,N,c,d,kind,param", CASES, ids=[x[0] for x in CASES])
def test_ring_simulate_parity(name, N, c, d, kind, param):
    U, R = case_plan(N, c, kind, param)
    kappa = OP.max_kappa_M(U)
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=N + c)
    grads = to_device(g)
    work, ws, out = buffers(plan, d)
    C.ring_simulate(plan, d, grads, work, ws, out)
    sync()
    gpu = out.double().cpu().numpy()
    ref = oracle_allreduce(g, U, R)
    S = OR.exact_sum(g)
    parity = max_rel_l2(gpu, ref)
    # diagnostic: the oracle on the fp32-rounded coefficients the kernels use,
    # which leaves only the kernels' own arithmetic in the difference
    U32c, R32c = U.astype(np.float32).astype(np.float64), R.astype(np.float32).astype(np.float64)
    parity32 = max_rel_l2(gpu, oracle_allreduce(g, U32c, R32c))
    err_gpu = max(rel_l2(gpu[i], S) for i in range(N))
    err_orc = max(rel_l2(ref[i], S) for i in range(N))
    print(f"{name}: kappa_M={kappa:.3g} parity={parity:.3g} parity_vs_fp32_coefficients={parity32:.3g} "
          f"err_gpu={err_gpu:.4g} err_oracle={err_orc:.4g}")
    assert np.all(np.isfinite(gpu))
    assert parity <= gate(kappa)
    assert parity32 <= gate(kappa)
    if kappa <= 1e3:
        assert abs(err_gpu - err_orc) <= 1e-4
    if kind == "o_eps" and param == 0.0:
        assert err_orc < 1e-12 and err_gpu < 1e-5        # exact ring all-reduce (c = N)


def _random_shapes(count, seed):
    """Seeded (N, c, d) shapes: c = 128 with every decode kernel (K = c + N - 1
    up to 144 on the split-operand kernel, above it on the fp32 one),
    multiples of 16 and odd c, d with and without interior blocks."""
    rng = np.random.default_rng(seed)
    shapes = []
    for t in range(count):
        N = int(rng.integers(2, 19))
        c = 128 if t % 3 == 0 else (16 * int(rng.integers(1, 9)) if t % 3 == 1 else int(rng.integers(N, 100)))
        c = max(c, N)
        p = 64 * int(rng.integers(1, 7)) + (int(rng.integers(0, 64)) if t % 2 else 0)
        d = max(1, c * p - int(rng.integers(0, 3 * p if t % 4 == 3 else 64)))
        shapes.append((N, c, d))
    return shapes


@pytest.mark.parametrize("N,c,d", _random_shapes(24, 2609))
def test_random_shapes_match_oracle(N, c, d):
    """The whole ring on a well-conditioned plan (orthogonal U_k, least-squares
    R_i) over seeded random shapes, gated like the named cases."""
    U, R = orthogonal_plan(N, c, seed=N * 7 + c)
    kappa = OP.max_kappa_M(U)
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=d % 1000)
    grads = to_device(g)
    work, ws, out = buffers(plan, d)
    C.ring_simulate(plan, d, grads, work, ws, out)
    sync()
    gpu = out.double().cpu().numpy()
    assert np.all(np.isfinite(gpu))
    assert max_rel_l2(gpu, oracle_allreduce(g, U, R)) <= gate(kappa), (N, c, d, kappa)


EDGE = [
    # name, N, c, d: degenerate and extreme shapes
    ("d1", 4, 8, 1),                       # p = 1: seven chunks are pure padding
    ("d-below-c", 4, 8, 7),
    ("N2-c2-exact", 2, 2, 2 * 1000 + 1),   # c = N, the textbook ring
    ("N2-c128", 2, 128, 128 * 70 + 5),     # largest c, smallest N
    ("N64-c64-exact", 64, 64, 64 * 80),    # largest N
    ("N64-c65", 64, 65, 65 * 64 + 1),
    ("N64-c128", 64, 128, 128 * 640 - 3),  # largest N and c: L = 190, the 48-K-step wide decode
    ("p-63", 4, 16, 16 * 63),              # one partial 64-position block
    ("p-64", 4, 16, 16 * 64),              # exactly one block
    ("p-65", 4, 16, 16 * 65),
]


@pytest.mark.parametrize("name,N,c,d", EDGE, ids=[e[0] for e in EDGE])
def test_edge_shapes(name, N, c, d):
    """Well-conditioned explicit plans (orthogonal encoders, least-squares
    decoders; for c = N the exact plan with B = I) on degenerate shapes."""
    if c == N:
        U, R = OP.mpc_plan(np.eye(N), np.eye(N))       # B = I: the textbook ring schedule
    else:
        U, R = orthogonal_plan(N, c, seed=N + c)
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=c + d)
    grads = to_device(g)
    work, ws, out = buffers(plan, d)
    C.ring_simulate(plan, d, grads, work, ws, out)
    sync()
    gpu = out.double().cpu().numpy()
    ref = oracle_allreduce(g, U, R)
    assert np.all(np.isfinite(gpu))
    assert max_rel_l2(gpu, ref) <= 1e-4, name
    if c == N:
        S = OR.exact_sum(g)
        assert max(rel_l2(gpu[i], S) for i in range(N)) < 1e-5


def test_side_stream_and_step_calls_match_single_call():
    """The step-wise calls on a non-default stream give the same bits as the
    single call on the current stream (same kernels, ordered by the stream)."""
    torch, dev = torch_dev()
    N, c, d = 8, 64, 64 * 700 + 13
    U, R = orthogonal_plan(N, c, seed=21)
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=21)
    grads = to_device(g)
    work, ws, out = buffers(plan, d)
    C.ring_simulate(plan, d, grads, work, ws, out)
    sync()
    side = torch.cuda.Stream()
    work2, ws2, out2 = buffers(plan, d)
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for k in range(plan.L + 1):
            C.encode_round(plan, k, d, grads, work2, ws2, stream=side)
        C.decode(plan, d, work2, ws2, out2, stream=side)
    side.synchronize()
    assert bool(torch.equal(out, out2))


def test_two_streams_share_one_plan():
    """One plan, two independent all-reduces enqueued step by step on two
    streams, interleaved call by call from the host, so their kernels may
    overlap on the device: each gives the bits of the same call made alone,
    and each workspace's step cursor follows its own stream's calls."""
    torch, dev = torch_dev()
    N, c, d = 8, 32, 32 * 3000 + 5
    U, R = orthogonal_plan(N, c, seed=41)
    plan = C.Plan.explicit(U, R)
    ga, gb = to_device(host_grads(N, d, seed=41)), to_device(host_grads(N, d, seed=42))
    ref = []
    for g in (ga, gb):
        work, ws, out = buffers(plan, d)
        C.ring_simulate(plan, d, g, work, ws, out)
        sync()
        ref.append(out.clone())
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    bufs = [buffers(plan, d), buffers(plan, d)]
    for s in (sa, sb):
        s.wait_stream(torch.cuda.current_stream())
    for k in range(plan.L + 1):
        for g, s, (work, ws, _) in ((ga, sa, bufs[0]), (gb, sb, bufs[1])):
            C.encode_round(plan, k, d, g, work, ws, stream=s)
    for s, (work, ws, out) in ((sa, bufs[0]), (sb, bufs[1])):
        C.decode(plan, d, work, ws, out, stream=s)
    sa.synchronize()
    sb.synchronize()
    assert bool(torch.equal(bufs[0][2], ref[0]))
    assert bool(torch.equal(bufs[1][2], ref[1]))


def test_binding_checks_dtype_layout_and_extent():
    """Tensors the kernels would read or write out of range, or in the wrong
    element type, are refused by the binding before any launch."""
    torch, dev = torch_dev()
    N, c, d = 4, 8, 8 * 300 + 3
    U, R = orthogonal_plan(N, c, seed=5)
    plan = C.Plan.explicit(U, R)
    grads = to_device(host_grads(N, d, seed=5))
    work, ws, out = buffers(plan, d)
    bad = [
        ("grads must be float32", lambda: C.ring_simulate(plan, d, grads.double(), work, ws, out)),
        ("grads has shape", lambda: C.ring_simulate(plan, d, grads[:N - 1], work, ws, out)),
        ("grads has shape", lambda: C.ring_simulate(plan, d + 1, grads, work, ws, out)),
        ("work has shape", lambda: C.encode_round(plan, 0, d, grads, work[:, :-1], ws)),
        ("ws holds", lambda: C.ring_simulate(plan, d, grads, work, ws[:-4], out)),
        ("ws must be contiguous", lambda: C.ring_simulate(plan, d, grads, work, ws.view(2, -1).t(), out)),
        ("out has shape", lambda: C.decode(plan, d, work, ws, out[:, :d - 1])),
        ("row-major", lambda: C.ring_simulate(plan, d, grads, work, ws, out.t().contiguous().t())),
        ("out has shape", lambda: C.ring_simulate_fused(plan, d, grads, out[1:])),
        ("norms must be", lambda: C.error_norms(N, d, grads, out, torch.zeros(N, dtype=torch.float64, device=dev))),
        ("dst has", lambda: C.copy_f32(out.view(-1)[:-1], grads.view(-1))),
    ]
    before = out.clone()
    for what, call in bad:
        with pytest.raises(ValueError, match=what):
            call()
    sync()
    assert bool(torch.equal(out.isnan(), before.isnan()))


def test_host_threads_share_one_fresh_plan():
    """Four host threads make their first calls on one plan at the same time
    (the one-time device upload and the per-workspace step records are
    shared state), each stepping its own all-reduce on its own stream; each
    result equals the single call made afterwards on the same inputs."""
    import threading
    torch, dev = torch_dev()
    N, c, d = 4, 16, 16 * 2000 + 3
    U, R = orthogonal_plan(N, c, seed=51)
    plan = C.Plan.explicit(U, R)                   # not yet on the device
    inputs = [to_device(host_grads(N, d, seed=510 + t)) for t in range(4)]
    bufs = [buffers(plan, d) for _ in range(4)]
    streams = [torch.cuda.Stream() for _ in range(4)]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    start, errors = threading.Barrier(4), []

    def worker(t):
        try:
            work, ws, out = bufs[t]
            start.wait()
            for k in range(plan.L + 1):
                C.encode_round(plan, k, d, inputs[t], work, ws, stream=streams[t])
            C.decode(plan, d, work, ws, out, stream=streams[t])
            streams[t].synchronize()
        except Exception as e:                     # reported below
            errors.append((t, repr(e)))

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(4)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not errors, errors
    for t in range(4):
        work, ws, out = buffers(plan, d)
        C.ring_simulate(plan, d, inputs[t], work, ws, out)
        sync()
        assert bool(torch.equal(bufs[t][2], out)), t


IN_PLACE = [
    # name, N, c, d, extra floats of row stride (odd: the scalar layout)
    ("c16", 4, 16, 16 * 1000, 0),              # the pipelined encode
    ("c5-ragged", 3, 5, 5 * 333 + 2, 0),       # c not a multiple of 16: the masked kernels
    ("c64-ragged", 8, 64, 64 * 1536 + 61, 0),  # the double-buffered c = 64 encode, then the tail
    ("c128-ragged", 4, 128, 128 * 320 + 7, 0), # the wide c = 128 encode, then the generic tail
    ("c64-scalar", 4, 64, 64 * 500 + 3, 1),    # misaligned rows: the scalar layout
]


@pytest.mark.parametrize("name,N,c,d,extra", IN_PLACE, ids=[x[0] for x in IN_PLACE])
def test_in_place_encode_matches_out_of_place(name, N, c, d, extra):
    """work == grads (the storage rule of Sec. II: Delta_i overwrites G_i):
    every kernel family reads a block's c input rows before it writes any of
    them, so the result is bit-identical to the out-of-place encode."""
    U, R = mpc_plan(N, c, 0.3, seed=9) if c <= 16 else orthogonal_plan(N, c, seed=9)
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=9)
    p, _ = plan.chunk_len(d)
    torch, dev = torch_dev()
    ld = c * p + extra
    a = to_device(np.pad(g, ((0, 0), (0, c * p - d))), ld=ld)      # grads with room for c*p
    work, ws, out = buffers(plan, d, ld_work=ld)
    C.ring_simulate(plan, d, a, work, ws, out)
    ws2 = torch.zeros_like(ws)
    out2 = torch.empty_like(out)
    C.ring_simulate(plan, d, a, a, ws2, out2)                        # encode in place
    sync()
    np.testing.assert_array_equal(out.cpu().numpy(), out2.cpu().numpy())
    # the rows now hold the encoded chunks: the same bits as the separate work buffer
    np.testing.assert_array_equal(a[:, :c * p].cpu().numpy(), work[:, :c * p].cpu().numpy())
    ref = oracle_allreduce(g, U, R)
    assert max_rel_l2(out2.double().cpu().numpy(), ref) <= gate(OP.max_kappa_M(U))


def test_scalar_layout_matches_vector_layout():
    """Misaligned strides force the scalar kernels; same values as vector ones."""
    N, c, d = 4, 8, 8 * 512
    U, R = mpc_plan(N, c, 0.3, seed=10)
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=10)
    p, _ = plan.chunk_len(d)
    work, ws, out = buffers(plan, d)
    C.ring_simulate(plan, d, to_device(g), work, ws, out)
    work2, ws2, out2 = buffers(plan, d, ld_work=c * p + 1, ld_out=d + 3, out_offset=1)
    C.ring_simulate(plan, d, to_device(g, ld=d + 1), work2, ws2, out2)
    sync()
    a, b = out.double().cpu().numpy(), out2[:, :d].double().cpu().numpy()
    assert max_rel_l2(b, a) < 1e-6
    ref = oracle_allreduce(g, U, R)
    assert max_rel_l2(b, ref) < 1e-4


def test_decode_never_writes_beyond_d():
    N, c, d = 3, 5, 5 * 64 + 2
    U, R = mpc_plan(N, c, 0.3, seed=11)
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=11)
    work, ws, out = buffers(plan, d, ld_out=d + 64)
    C.ring_simulate(plan, d, to_device(g), work, ws, out)
    sync()
    o = out.cpu().numpy()
    assert np.all(np.isnan(o[:, d:]))
    assert np.all(np.isfinite(o[:, :d]))


def test_rerun_on_same_buffers_is_deterministic():
    N, c, d = 8, 32, 32 * 999
    U, R = mpc_plan(N, c, 0.3, seed=12)
    plan = C.Plan.explicit(U, R)
    grads = to_device(host_grads(N, d, seed=12))
    work, ws, out = buffers(plan, d)
    C.ring_simulate(plan, d, grads, work, ws, out)
    first = out.clone()
    C.ring_simulate(plan, d, grads, work, ws, out)
    sync()
    assert bool((first == out).all())


def test_step_order_enforced_on_device_buffers():
    N, c, d = 4, 5, 500
    U, R = mpc_plan(N, c, 0.3, seed=13)
    plan = C.Plan.explicit(U, R)
    grads = to_device(host_grads(N, d, seed=13))
    work, ws, out = buffers(plan, d)
    C.encode_round(plan, 0, d, grads, work, ws)
    with pytest.raises(C.CerarError) as ei:
        C.encode_round(plan, 2, d, grads, work, ws)
    assert ei.value.status == -6
    with pytest.raises(C.CerarError):
        C.decode(plan, d, work, ws, out)
    with pytest.raises(C.CerarError) as ei:                # a round with another length
        C.encode_round(plan, 1, d - 5, grads, work, ws)
    assert ei.value.status == -6
    for k in range(1, c + N - 1):
        C.encode_round(plan, k, d, grads, work, ws)
    with pytest.raises(C.CerarError) as ei:                # a decode with another length
        C.decode(plan, d - 5, work, ws, out)
    assert ei.value.status == -6
    C.decode(plan, d, work, ws, out)
    sync()


# --- K5 error norms, buckets, copy -------------------------------------------------------

def test_error_norms_kernel():
    torch, dev = torch_dev()
    N, d = 5, 100_003
    g = host_grads(N, d, seed=14)
    o = host_grads(N, d, seed=15)
    norms = torch.empty(N + 1, dtype=torch.float64, device=dev)
    C.error_norms(N, d, to_device(g), to_device(o), norms)
    sync()
    S = OR.exact_sum(g)
    ref = [np.sum((o[i].astype(np.float64) - S) ** 2) for i in range(N)] + [np.sum(S * S)]
    np.testing.assert_allclose(norms.cpu().numpy(), ref, rtol=1e-12)
    N = 17
    g = host_grads(N, 4097, seed=16)
    norms = torch.empty(N + 1, dtype=torch.float64, device=dev)
    C.error_norms(N, 4097, to_device(g), to_device(g), norms)
    sync()
    S = OR.exact_sum(g)
    ref = [np.sum((g[i].astype(np.float64) - S) ** 2) for i in range(N)] + [np.sum(S * S)]
    np.testing.assert_allclose(norms.cpu().numpy(), ref, rtol=1e-12)


def test_sampled_norms_kernel():
    """K5's parity term: squared differences against reference values at
    sampled flat indices, and squared references, per worker in fp64; an
    index outside [0, d) makes the sums NaN instead of reading out of range."""
    torch, dev = torch_dev()
    N, d, count = 5, 100_003, 5000
    rng = np.random.default_rng(18)
    o = host_grads(N, d, seed=18)
    idx = rng.integers(0, d, size=count).astype(np.int64)
    ref = rng.standard_normal((N, count))
    norms = torch.empty(2 * N, dtype=torch.float64, device=dev)
    out = to_device(o, ld=d + 3)
    C.sampled_norms(N, d, torch.from_numpy(idx).to(dev), torch.from_numpy(ref).to(dev), out, norms)
    sync()
    got = norms.cpu().numpy()
    for i in range(N):
        g = o[i][idx].astype(np.float64)
        np.testing.assert_allclose(got[2 * i], np.sum((g - ref[i]) ** 2), rtol=1e-12)
        np.testing.assert_allclose(got[2 * i + 1], np.sum(ref[i] ** 2), rtol=1e-12)
    idx[17] = d                                     # one index past the end
    C.sampled_norms(N, d, torch.from_numpy(idx).to(dev), torch.from_numpy(ref).to(dev), out, norms)
    sync()
    got = norms.cpu().numpy()
    assert np.all(np.isnan(got[0::2])) and np.all(np.isfinite(got[1::2]))


def test_bucketed_matches_independent_instances():
    torch, dev = torch_dev()
    N, c = 4, 8
    buckets = [(0, 8 * 300), (8 * 300, 1001), (8 * 300 + 1001, 8 * 64), (8 * 364 + 1001, 13)]
    d = buckets[-1][0] + buckets[-1][1]
    U, R = mpc_plan(N, c, 0.3, seed=17)
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=17)
    work_floats, ws_bytes = plan.bucketed_sizes([b[1] for b in buckets])
    work = torch.empty((N, work_floats), dtype=torch.float32, device=dev)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device=dev)
    out = torch.full((N, d), float("nan"), dtype=torch.float32, device=dev)
    C.ring_simulate_bucketed(plan, buckets, to_device(g), work, ws, out)
    sync()
    gpu = out.double().cpu().numpy()
    for off, ln in buckets:
        ref = oracle_allreduce(g[:, off:off + ln], U, R)
        assert max_rel_l2(gpu[:, off:off + ln], ref) < 1e-4


def _bucket_list(rng, nb, c):
    """nb buckets, back to back, 16-byte aligned: c*32*k - 4*j floats, so
    that most have interior blocks and a ragged last chunk row."""
    lens = [int(c * 32 * rng.integers(1, 40) - 4 * rng.integers(0, 8)) for _ in range(nb)]
    offs = np.concatenate([[0], np.cumsum(lens)[:-1]]).tolist()
    return [(int(o), int(n)) for o, n in zip(offs, lens)]


@pytest.mark.parametrize("N,c,nb,kind", [(8, 16, 40, "o_eps"), (4, 64, 5, "kappa"), (3, 20, 6, "o_eps"),
                                         (8, 32, 33, "kappa")])
def test_bucketed_batched_encode_and_decode(N, c, nb, kind):
    """16-byte aligned buckets take the batched encode/decode (up to 32 buckets
    per launch, interior blocks then tails); every bucket must match its own
    oracle instance."""
    torch, dev = torch_dev()
    rng = np.random.default_rng(N * 100 + c)
    buckets = _bucket_list(rng, nb, c)
    buckets.append((buckets[-1][0] + buckets[-1][1], 4))          # a bucket of one position per chunk row
    d = buckets[-1][0] + buckets[-1][1]
    U, R = case_plan(N, c, kind, 0.3 if kind == "o_eps" else 1e3)
    kappa = OP.max_kappa_M(U)
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=N + c + nb)
    work_floats, ws_bytes = plan.bucketed_sizes([b[1] for b in buckets])
    work = torch.empty((N, work_floats), dtype=torch.float32, device=dev)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device=dev)
    out = torch.full((N, d), float("nan"), dtype=torch.float32, device=dev)
    C.ring_simulate_bucketed(plan, buckets, to_device(g), work, ws, out)
    sync()
    gpu = out.double().cpu().numpy()
    assert np.all(np.isfinite(gpu))
    for off, ln in buckets:
        ref = oracle_allreduce(g[:, off:off + ln], U, R)
        assert max_rel_l2(gpu[:, off:off + ln], ref) <= gate(kappa), (off, ln)


def test_c128_at_the_top_of_the_kappa_range_stays_at_the_fp32_message_floor():
    """N = 4, c = 128 on a kappa_max = 1e3 design (kappa_2(M) ~ 850), through
    the single call (split-operand interior kernels and the tail) and the
    bucketed call (batched fp32 kernels).  Here the protocol with fp32
    messages is itself above 1e-4 (about 2.1 kappa u), so the bar is that
    floor, computed on the host for the same plan and inputs: the kernels may
    add at most 15 % to it (they round each message once, as the floor
    does, and accumulate the contractions in fp32)."""
    torch, dev = torch_dev()
    from gpu_util import fp32_protocol_floor
    N, c = 4, 128
    U, R = case_plan(N, c, "kappa", 1e3)
    kappa = OP.max_kappa_M(U)
    plan = C.Plan.explicit(U, R)
    d = 128 * 640 - 37
    g = host_grads(N, d, seed=41)
    work, ws, out = buffers(plan, d)
    C.ring_simulate(plan, d, to_device(g), work, ws, out)
    sync()
    gpu = out.double().cpu().numpy()
    parity = max_rel_l2(gpu, oracle_allreduce(g, U, R))
    floor = fp32_protocol_floor(g, U, R)
    print(f"N4-c128 kappa_M={kappa:.4g}: parity {parity:.3g}, fp32-message floor {floor:.3g}")
    assert parity <= max(gate(kappa), 1.15 * floor)
    rng = np.random.default_rng(43)
    buckets = _bucket_list(rng, 4, c)
    db = buckets[-1][0] + buckets[-1][1]
    gb = host_grads(N, db, seed=44)
    work_floats, ws_bytes = plan.bucketed_sizes([b[1] for b in buckets])
    bwork = torch.empty((N, work_floats), dtype=torch.float32, device=dev)
    bws = torch.zeros(ws_bytes, dtype=torch.uint8, device=dev)
    bout = torch.full((N, db), float("nan"), dtype=torch.float32, device=dev)
    C.ring_simulate_bucketed(plan, buckets, to_device(gb), bwork, bws, bout)
    sync()
    bgpu = bout.double().cpu().numpy()
    for off, ln in buckets:
        part = gb[:, off:off + ln]
        par = max_rel_l2(bgpu[:, off:off + ln], oracle_allreduce(part, U, R))
        fl = fp32_protocol_floor(part, U, R)
        assert par <= max(gate(kappa), 1.15 * fl), (off, ln, par, fl)


def test_copy_kernel():
    torch, dev = torch_dev()
    for n in (1, 7, 4096, 1_000_003):
        src = torch.randn(n + 1, device=dev)[1:] if n % 2 else torch.randn(n, device=dev)
        dst = torch.empty_like(src)
        C.copy_f32(dst, src)
        sync()
        assert bool((dst == src).all())


# --- single-GPU fused variant (reported, not the counted path) ------------------------

FUSED = [
    # name, N, c, d
    ("N8-c64-ragged", 8, 64, 64 * 1536 + 61),
    ("N4-c16", 4, 16, 16 * 4096),
    ("N8-c32-tail", 8, 32, 32 * 777 + 5),
    ("N16-c32", 16, 32, 32 * 640),
    ("N2-c48", 2, 48, 48 * 300 + 7),
    ("N8-c64-d1", 8, 64, 1),
    # N not in {2, 4, 8}: the one-barrier-per-round kernel
    ("N3-c16", 3, 16, 16 * 500 + 3),
    ("N6-c64", 6, 64, 64 * 700 + 9),
    ("N5-c48-tail", 5, 48, 48 * 129 + 47),
]


@pytest.mark.parametrize("name,N,c,d", FUSED, ids=[x[0] for x in FUSED])
def test_fused_variant_matches_oracle_and_ring(name, N, c, d):
    torch, dev = torch_dev()
    U, R = orthogonal_plan(N, c, seed=N * 7 + c) if N < c else OP.mpc_plan(np.eye(N), np.eye(N))
    U = U * np.random.default_rng(c).uniform(0.5, 2.0, size=(N, 1, c))   # not orthogonal any more
    R = OP.r_step(U)
    plan = C.Plan.explicit(U, R)
    g = host_grads(N, d, seed=N + c + d)
    ld = (d + 3) // 4 * 4                            # the fused variant needs 16-byte aligned rows
    grads = to_device(g, ld=ld)
    out = torch.full((N, ld), float("nan"), dtype=torch.float32, device=dev)
    C.ring_simulate_fused(plan, d, grads, out)
    work, ws, out_ring = buffers(plan, d)
    C.ring_simulate(plan, d, grads, work, ws, out_ring)
    sync()
    assert bool(torch.isnan(out[:, d:]).all())       # nothing written beyond d
    fused = out[:, :d].double().cpu().numpy()
    ring = out_ring.double().cpu().numpy()
    ref = oracle_allreduce(g, U, R)
    kappa = OP.max_kappa_M(U)
    parity = max_rel_l2(fused, ref)
    print(f"fused {name}: kappa_M={kappa:.3g} parity={parity:.3g} max|fused - ring|={np.abs(fused - ring).max():.3g}")
    assert np.all(np.isfinite(fused))
    assert parity <= gate(kappa)
    # the fused kernels apply the ring's fp32 operations in the ring's order
    # (MFMA K-steps in order, (recv - delta) + delta in the rounds), so the
    # results are bit-identical, not just close
    np.testing.assert_array_equal(fused, ring)


def test_fused_variant_rejects_unsupported_shapes():
    torch, dev = torch_dev()
    for N, c in ((4, 128), (16, 64), (4, 20)):
        U, R = orthogonal_plan(N, c, seed=1)
        plan = C.Plan.explicit(U, R)
        d = c * 64
        g = to_device(host_grads(N, d, seed=1))
        out = torch.empty((N, d), dtype=torch.float32, device=dev)
        with pytest.raises(C.CerarError) as ei:
            C.ring_simulate_fused(plan, d, g, out)
        assert ei.value.status == -1
