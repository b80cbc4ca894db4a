"""K6, the device generator of the synthetic gradients (cerar_synth_fill),
against the host generator the oracle's inputs come from: identical bits on
every workload kind (log-normal tensor scales with their boundaries, an
i.i.d. scale, 1 % outliers), across the end of the gradient (the zero pad),
at unaligned starts and lengths, and on misaligned output (the scalar
stores)."""

import numpy as np
import pytest

from paper_2609_23898_amd import cerar as C
from paper_2609_23898_amd import synth

from gpu_util import torch_dev

pytestmark = pytest.mark.gpu


def _check(wl, worker, start, n, misalign=0):
    torch, dev = torch_dev()
    buf = torch.full((n + misalign,), float("nan"), dtype=torch.float32, device=dev)
    out = buf[misalign:]
    C.synth_fill(out, wl, worker, start=start)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ref = wl.values_np(worker, np.arange(start, start + n, dtype=np.int64))
    np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("name", synth.WORKLOADS)
def test_device_generator_matches_host_generator(name):
    wl = synth.workload(name)
    rng = np.random.default_rng(len(name))
    for worker in (0, wl.N - 1):
        _check(wl, worker, 0, 1 << 16)
        _check(wl, worker, int(rng.integers(0, wl.d)), 65537, misalign=1)
        _check(wl, worker, max(0, wl.d - 40001), 40001 + 4099)          # across d: the pad reads 0
    if wl.tensor_sizes is not None:                                      # every tensor boundary
        for b in wl._offsets[1:-1][:: max(1, len(wl._offsets) // 40)]:
            _check(wl, 1, int(b) - 3, 10)


def test_device_generator_whole_gradient_sampled():
    """One worker's whole GPT-2-small gradient in one launch, sampled."""
    torch, dev = torch_dev()
    wl = synth.workload("gpt2-small")
    out = torch.empty(wl.d, dtype=torch.float32, device=dev)
    C.synth_fill(out, wl, 3)
    idx = np.unique(np.random.default_rng(5).integers(0, wl.d, 200_000))
    got = out[torch.from_numpy(idx).to(dev)].cpu().numpy()
    np.testing.assert_array_equal(got.view(np.uint32), wl.values_np(3, idx).view(np.uint32))
    assert bool(torch.isfinite(out).all())


def test_device_generator_rejects_bad_tables():
    torch, dev = torch_dev()
    out = torch.empty(16, dtype=torch.float32, device=dev)
    lib = C.lib()
    assert lib.cerar_synth_fill(C._ptr(out), 16, 0, 16, 1, None, None, 1, 0, 1.0, None) == -1
    offs = torch.zeros(2, dtype=torch.int64, device=dev)
    sc = torch.ones(1, dtype=torch.float32, device=dev)
    assert lib.cerar_synth_fill(C._ptr(out), 16, 0, 16, 1, C._ptr(offs), C._ptr(sc), 0, 0, 1.0, None) == -1
    assert lib.cerar_synth_fill(C._ptr(out), 0, 0, 16, 1, None, None, 0, 0, 1.0, None) == 0
