"""Every kernel writes only inside the buffers it owns: the encode into the c*p
slot area of each work row and the workers' first pool slots, the rounds into
work and workspace slots, the decode into the first d floats of each out row.

One device allocation holds guard zones filled with a sentinel before, between
and after grads, work, ws and out, and the row gaps of strided buffers are
sentinel-filled too; after a full run (both the single call and the step-wise
calls) every guard is intact and grads are unchanged.  Covers c below, at and
above one 16-row MFMA tile, c not a multiple of 4, ragged d and odd strides."""

import numpy as np
import pytest

from paper_2609_23898_amd import cerar as C

from gpu_util import host_grads, mpc_plan, torch_dev

pytestmark = pytest.mark.gpu

SENTINEL = np.float32(-7.25e29)
GUARD = 4096            # floats (16 KiB) around every region


class Arena:
    """Regions carved from one allocation, separated by sentinel guards."""

    def __init__(self, sizes):
        torch, dev = torch_dev()
        total = GUARD + sum(n + GUARD for n in sizes)
        self.buf = torch.full((total,), float(SENTINEL), dtype=torch.float32, device=dev)
        self.offsets = []
        off = GUARD
        for n in sizes:
            self.offsets.append(off)
            off += n + GUARD

    def region(self, i, n):
        return self.buf[self.offsets[i]:self.offsets[i] + n]


CASES = [
    # N, c, d, extra ld floats for grads / work / out
    (4, 4, 4096, 0, 0, 0),
    (4, 4, 4096, 3, 5, 7),
    (3, 8, 8 * 257 + 3, 0, 4, 8),
    (4, 12, 12 * 300, 0, 0, 0),
    (2, 20, 20 * 64 + 19, 1, 1, 1),
    (8, 16, 16 * 1024, 0, 0, 0),
    (8, 64, 64 * 700 + 33, 0, 64, 64),
    (8, 64, 64 * 1024, 0, 0, 0),
    (4, 128, 128 * 130, 0, 0, 4),
    (2, 128, 128 * 640, 0, 0, 0),        # c = 128 interior blocks: the wide MFMA kernels
    (3, 128, 128 * 640 - 17, 0, 4, 4),   # ... plus a ragged tail on the generic ones
    (16, 32, 32 * 96 + 5, 4, 8, 12),
    (64, 128, 128 * 640 - 3, 0, 4, 4),   # largest N and c
]


@pytest.mark.parametrize("N,c,d,eg,ew,eo", CASES)
def test_kernels_stay_inside_their_buffers(N, c, d, eg, ew, eo):
    run_bounds(N, c, d, eg, ew, eo, in_place=False)


IN_PLACE_CASES = [
    # N, c, d, extra ld floats (grads = work, so one stride)
    (4, 5, 5 * 300 + 2, 0),
    (8, 16, 16 * 1024 + 9, 4),
    (8, 64, 64 * 700 + 33, 0),
    (4, 64, 64 * 300 + 5, 1),            # odd stride: the scalar layout
    (3, 128, 128 * 640 - 17, 4),         # the wide c = 128 encode and its tail
]


@pytest.mark.parametrize("N,c,d,extra", IN_PLACE_CASES)
def test_in_place_encode_stays_inside_its_buffers(N, c, d, extra):
    """work == grads: the encode writes the c*p slot area of each row in
    place (the zero pad of the last chunk included) and nothing else."""
    run_bounds(N, c, d, 0, extra, 0, in_place=True)


def run_bounds(N, c, d, eg, ew, eo, in_place):
    torch, dev = torch_dev()
    U, R = mpc_plan(N, c, 0.3, seed=N * 100 + c)
    plan = C.Plan.explicit(U, R)
    p, _ = plan.chunk_len(d)
    ldg, ldw, ldo = d + eg, c * p + ew, d + eo
    if in_place:
        ldg = ldw
    ws_floats = plan.workspace_bytes(d) // 4
    arena = Arena([N * ldg, N * ldw, ws_floats, N * ldo])
    g = host_grads(N, d, seed=c)
    grads = arena.region(0, N * ldg).view(N, ldg)
    grads[:, :d] = torch.from_numpy(g).to(dev)
    if in_place:
        grads[:, d:c * p] = 0.0                    # the zero pad of the last chunk
    work = grads if in_place else arena.region(1, N * ldw).view(N, ldw)
    ws = arena.region(2, ws_floats)
    out = arena.region(3, N * ldo).view(N, ldo)
    ws.zero_()
    before = arena.buf.clone()
    wsb = ws.view(torch.uint8)
    C.ring_simulate(plan, d, grads, work, wsb, out)
    if not in_place:                               # in place, the single call consumed the gradients
        for k in range(plan.L + 1):
            C.encode_round(plan, k, d, grads, work, wsb)
        C.decode(plan, d, work, wsb, out)
    torch.cuda.synchronize()
    after = arena.buf
    # guards untouched
    edges = [0] + [x for o, n in zip(arena.offsets, [N * ldg, N * ldw, ws_floats, N * ldo])
                   for x in (o, o + n)] + [after.numel()]
    for lo, hi in zip(edges[0::2], edges[1::2]):
        assert bool((after[lo:hi] == before[lo:hi]).all()), f"guard [{lo}, {hi}) overwritten"
    # grads unchanged (out-of-place encode), row gaps of work and out untouched
    if in_place:
        assert bool((after[arena.offsets[1]:arena.offsets[1] + N * ldw] == SENTINEL).all())  # unused region
        assert bool(torch.isfinite(work[:, :c * p]).all())
    else:
        assert bool((grads == before[arena.offsets[0]:arena.offsets[0] + N * ldg].view(N, ldg)).all())
    assert bool((work[:, c * p:] == SENTINEL).all())
    assert bool((out[:, d:] == SENTINEL).all())
    assert bool(torch.isfinite(out[:, :d]).all())
