"""Python binding of libcerar (ctypes).  Argument marshalling only: every
step of the all-reduce runs in the library's HIP kernels; torch supplies
device memory and the stream.

The in-tree ``libcerar.so`` is required: importing this module raises if it
has not been built (``__graft_entry__.build()``), and there is no fallback.
"""

import ctypes
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcerar.so")

VANDERMONDE, O_EPS, KAPPA, EXPLICIT = 0, 1, 2, 3
_KINDS = {"vandermonde": VANDERMONDE, "o_eps": O_EPS, "kappa": KAPPA, "explicit": EXPLICIT}

STATUS = {0: "OK", -1: "E_INVAL", -2: "E_NOMEM", -3: "E_SINGULAR", -4: "E_NOCONV",
          -5: "E_DEVICE", -6: "E_STATE"}


class CerarError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class PlanDesc(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int), ("c", ctypes.c_int), ("kind", ctypes.c_int),
                ("param", ctypes.c_double), ("seed", ctypes.c_uint64),
                ("base", ctypes.POINTER(ctypes.c_double)),
                ("perturb", ctypes.POINTER(ctypes.c_double)),
                ("nodes", ctypes.POINTER(ctypes.c_double)),
                ("eps0", ctypes.c_double), ("als_iters", ctypes.c_int), ("als_order", ctypes.c_int),
                ("node_perms", ctypes.POINTER(ctypes.c_int)), ("n_node_perms", ctypes.c_int),
                ("svd_sweeps", ctypes.c_int), ("als_restarts", ctypes.c_int)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int), ("c", ctypes.c_int), ("L", ctypes.c_int), ("r_star", ctypes.c_int),
                ("kind", ctypes.c_int), ("param", ctypes.c_double),
                ("phi", ctypes.c_double), ("phi_closed_form", ctypes.c_double),
                ("phi_initial", ctypes.c_double), ("kappa_M", ctypes.c_double),
                ("kappa_U", ctypes.c_double), ("kappa_R", ctypes.c_double),
                ("amplification", ctypes.c_double), ("comm_rate", ctypes.c_double),
                ("storage_rate", ctypes.c_double), ("proj_a0", ctypes.c_double),
                ("proj_b0", ctypes.c_double), ("fp64_reliable", ctypes.c_int),
                ("seed_used", ctypes.c_uint64), ("gamma", ctypes.c_double), ("h_choice", ctypes.c_int),
                ("svd_converged", ctypes.c_int), ("restart_used", ctypes.c_int)]


_P = ctypes.c_void_p
_SZ = ctypes.c_size_t
_I = ctypes.c_int

# name -> (restype, argtypes); mirrors include/cerar.h
SIGNATURES = {
    "cerar_plan_create": (_I, [_I, _I, _I, ctypes.c_double, ctypes.c_uint64, ctypes.POINTER(_P)]),
    "cerar_plan_create_desc": (_I, [ctypes.POINTER(PlanDesc), ctypes.POINTER(_P)]),
    "cerar_plan_create_explicit": (_I, [_I, _I, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_P)]),
    "cerar_plan_destroy": (None, [_P]),
    "cerar_plan_prepare_device": (_I, [_P]),
    "cerar_plan_get_info": (_I, [_P, ctypes.POINTER(PlanInfo)]),
    "cerar_plan_get_matrices": (_I, [_P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    "cerar_chunk_len": (_I, [_P, _SZ, ctypes.POINTER(_SZ), ctypes.POINTER(_SZ)]),
    "cerar_workspace_bytes": (_I, [_P, _SZ, ctypes.POINTER(_SZ)]),
    "cerar_slot_map": (_I, [_P, _I, ctypes.POINTER(_I)]),
    "cerar_encode_round": (_I, [_P, _I, _SZ, _P, _SZ, _P, _SZ, _P, _P]),
    "cerar_decode": (_I, [_P, _SZ, _P, _SZ, _P, _P, _SZ, _P]),
    "cerar_ring_simulate": (_I, [_P, _SZ, _P, _SZ, _P, _SZ, _P, _P, _SZ, _P]),
    "cerar_ring_simulate_fused": (_I, [_P, _SZ, _P, _SZ, _P, _SZ, _P]),
    "cerar_ring_simulate_noalloc": (_I, [_P, _SZ, _P, _SZ, _P, _SZ, _P, _SZ, _P]),
    "cerar_bucketed_workspace_bytes": (_I, [_P, ctypes.POINTER(_SZ), _I, ctypes.POINTER(_SZ), ctypes.POINTER(_SZ)]),
    "cerar_ring_simulate_bucketed": (_I, [_P, _I, ctypes.POINTER(_SZ), ctypes.POINTER(_SZ), _P, _SZ, _P, _SZ,
                                          _P, _P, _SZ, _P]),
    "cerar_error_norms": (_I, [_I, _SZ, _P, _SZ, _P, _SZ, _P, _P]),
    "cerar_sampled_norms": (_I, [_I, _SZ, _SZ, _P, _P, _P, _SZ, _P, _P]),
    "cerar_copy_f32": (_I, [_P, _P, _SZ, _P]),
    "cerar_synth_fill": (_I, [_P, _SZ, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64, _P, _P, _I,
                              ctypes.c_uint32, ctypes.c_double, _P]),
    "cerar_last_error": (ctypes.c_char_p, []),
}

_lib = None


def _hip_runtimes():
    """Distinct HIP runtime files mapped into this process."""
    found = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                path = line.split()[-1]
                if "libamdhip64" in os.path.basename(path):
                    found.add(os.path.realpath(path))
    except OSError:
        pass
    return found


def lib():
    """The loaded in-tree libcerar.so (raises if it was not built).

    torch is imported first: libcerar needs the HIP runtime by its soname
    (libamdhip64.so.7), and once torch has loaded its runtime the dynamic
    loader binds that soname to torch's copy, so device pointers and streams
    from torch are valid in the library.  Two runtimes in one process would
    not share them, so that case raises."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        import torch  # noqa: F401  (loads the HIP runtime libcerar must share)
        handle = ctypes.CDLL(LIB_PATH)
        runtimes = _hip_runtimes()
        if len(runtimes) > 1:
            raise ImportError(f"two HIP runtimes are loaded ({sorted(runtimes)}); libcerar must share torch's")
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def _check(status):
    if status != 0:
        raise CerarError(status, lib().cerar_last_error().decode())


def _dptr(a):
    return None if a is None else ctypes.cast(a, ctypes.POINTER(ctypes.c_double))


class Plan:
    """Encoding/decoding plan (host fp64), see cerar_plan_create_desc."""

    def __init__(self, N, c, kind, param=0.0, seed=0, base=None, perturb=None, nodes=None,
                 eps0=0.0, als_iters=0, als_order=0, node_perms=None, svd_sweeps=0, als_restarts=0,
                 _handle=None):
        L = lib()
        self._h = _P()
        if _handle is not None:
            self._h = _handle
        else:
            keep = []

            def arr(x, n):
                if x is None:
                    return None
                a = np.ascontiguousarray(x, dtype=np.float64).ravel()
                assert a.size == n, (a.size, n)
                keep.append(a)
                return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))

            kind = _KINDS[kind] if isinstance(kind, str) else int(kind)
            perms, nperm = None, 0
            if node_perms is not None:
                pa = np.ascontiguousarray(node_perms, dtype=np.int32)
                assert pa.ndim == 2 and pa.shape[1] == c, pa.shape
                keep.append(pa)
                perms, nperm = pa.ctypes.data_as(ctypes.POINTER(ctypes.c_int)), pa.shape[0]
            desc = PlanDesc(N, c, kind, float(param), int(seed), arr(base, N * c),
                            arr(perturb, c * c), arr(nodes, c), float(eps0), int(als_iters),
                            int(als_order), perms, nperm, int(svd_sweeps), int(als_restarts))
            _check(L.cerar_plan_create_desc(ctypes.byref(desc), ctypes.byref(self._h)))
        info = self.info()
        self.N, self.c, self.L = info["N"], info["c"], info["L"]

    @classmethod
    def explicit(cls, U, R):
        U = np.ascontiguousarray(U, dtype=np.float64)
        R = np.ascontiguousarray(R, dtype=np.float64)
        N, c, _ = U.shape
        h = _P()
        _check(lib().cerar_plan_create_explicit(N, c, _dptr(U.ctypes.data), _dptr(R.ctypes.data),
                                                ctypes.byref(h)))
        return cls(N, c, EXPLICIT, _handle=h)

    @property
    def handle(self):
        return self._h

    def info(self):
        inf = PlanInfo()
        _check(lib().cerar_plan_get_info(self._h, ctypes.byref(inf)))
        return {name: getattr(inf, name) for name, _ in PlanInfo._fields_}

    def matrices(self):
        U = np.empty((self.N, self.c, self.c))
        R = np.empty((self.N, self.L + 1, self.c))
        _check(lib().cerar_plan_get_matrices(self._h, _dptr(U.ctypes.data), _dptr(R.ctypes.data)))
        return U, R

    def prepare_device(self):
        """Upload the plan to the current device now (cerar_plan_prepare_device),
        so that the enqueueing calls can be captured into a HIP graph."""
        _check(lib().cerar_plan_prepare_device(self._h))

    def chunk_len(self, d):
        p, s = _SZ(), _SZ()
        _check(lib().cerar_chunk_len(self._h, d, ctypes.byref(p), ctypes.byref(s)))
        return p.value, s.value

    def workspace_bytes(self, d):
        b = _SZ()
        _check(lib().cerar_workspace_bytes(self._h, d, ctypes.byref(b)))
        return b.value

    def slot_map(self, step):
        out = np.empty(self.N * (self.c + self.N), dtype=np.int32)
        _check(lib().cerar_slot_map(self._h, step, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int))))
        return out.reshape(self.N, self.c + self.N)

    def bucketed_sizes(self, bucket_len):
        lens = (_SZ * len(bucket_len))(*bucket_len)
        wf, wb = _SZ(), _SZ()
        _check(lib().cerar_bucketed_workspace_bytes(self._h, lens, len(bucket_len),
                                                    ctypes.byref(wf), ctypes.byref(wb)))
        return wf.value, wb.value

    def save(self, path):
        """Write the plan's fp64 matrices to an .npz file (plans are built
        offline once; Plan.load rebuilds the same plan as an explicit one)."""
        U, R = self.matrices()
        info = self.info()
        np.savez(path, U=U, R=R, kind=np.int32(info["kind"]), param=np.float64(info["param"]),
                 seed_used=np.uint64(info["seed_used"]))

    @classmethod
    def load(cls, path):
        """Plan from a file written by save()."""
        with np.load(path, allow_pickle=False) as z:
            return cls.explicit(z["U"], z["R"])

    def close(self):
        if self._h:
            lib().cerar_plan_destroy(self._h)
            self._h = _P()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# --- device calls (torch tensors) ----------------------------------------------

def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def _ld(t):
    return t.stride(0)


def _on_device(t, name):
    """t must be a tensor in device memory of the current device: the kernels
    read and write it directly."""
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a tensor on the GPU")
    if t.device.index != torch.cuda.current_device():
        raise ValueError(f"{name} is on cuda:{t.device.index}, the current device is "
                         f"cuda:{torch.cuda.current_device()}")


def _rows(t, name, rows, cols, dtype="float32"):
    """t must be an (at least rows x cols) row-major tensor of `dtype`, so
    that every element the kernels touch through (pointer, row stride) lies
    inside it."""
    _on_device(t, name)
    if str(t.dtype) != "torch." + dtype:
        raise ValueError(f"{name} must be {dtype}, not {t.dtype}")
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError(f"{name} must be a 2-D row-major tensor (unit column stride)")
    if t.shape[0] < rows or t.shape[1] < cols:
        raise ValueError(f"{name} has shape {tuple(t.shape)}; at least ({rows}, {cols}) is needed")


def _bytes(t, name, nbytes):
    """t must be a contiguous device tensor of at least nbytes bytes."""
    _on_device(t, name)
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() * t.element_size() < nbytes:
        raise ValueError(f"{name} holds {t.numel() * t.element_size()} bytes; {nbytes} are needed")


def allocate(plan, d, device="cuda", work_like_grads=False):
    """Device buffers for one all-reduce of length-d gradients: work (N, c*p),
    ws (workspace bytes) and out (N, d)."""
    import torch
    p, _ = plan.chunk_len(d)
    work = torch.empty((plan.N, plan.c * p), dtype=torch.float32, device=device)
    ws = torch.empty(plan.workspace_bytes(d), dtype=torch.uint8, device=device)
    out = torch.empty((plan.N, d), dtype=torch.float32, device=device)
    return work, ws, out


def _step_buffers(plan, d, grads=None, work=None, ws=None, out=None):
    p, _ = plan.chunk_len(d)
    if grads is not None:
        _rows(grads, "grads", plan.N, d)
    if work is not None:
        _rows(work, "work", plan.N, plan.c * p)
    if ws is not None:
        _bytes(ws, "ws", plan.workspace_bytes(d))
    if out is not None:
        _rows(out, "out", plan.N, d)


def encode_round(plan, step, d, grads, work, ws, stream=None):
    _step_buffers(plan, d, grads, work, ws)
    _check(lib().cerar_encode_round(plan.handle, step, d, _ptr(grads), _ld(grads), _ptr(work), _ld(work),
                                    _ptr(ws), _stream(stream)))


def decode(plan, d, work, ws, out, stream=None):
    _step_buffers(plan, d, None, work, ws, out)
    _check(lib().cerar_decode(plan.handle, d, _ptr(work), _ld(work), _ptr(ws), _ptr(out), _ld(out),
                              _stream(stream)))


def ring_simulate(plan, d, grads, work, ws, out, stream=None):
    _step_buffers(plan, d, grads, work, ws, out)
    _check(lib().cerar_ring_simulate(plan.handle, d, _ptr(grads), _ld(grads), _ptr(work), _ld(work),
                                     _ptr(ws), _ptr(out), _ld(out), _stream(stream)))


NOALLOC_SCRATCH_BYTES = 64 << 20          # CERAR_NOALLOC_SCRATCH_BYTES


def ring_simulate_noalloc(plan, d, grads, work, out, stream=None):
    """cerar_ring_simulate_noalloc: the whole all-reduce with the message pool
    in the library's static device array (no workspace, no allocation); the
    plan must have been prepared on the device (Plan.prepare_device)."""
    _step_buffers(plan, d, grads, work, None, out)
    _check(lib().cerar_ring_simulate_noalloc(plan.handle, d, _ptr(grads), _ld(grads), _ptr(work), _ld(work),
                                             _ptr(out), _ld(out), _stream(stream)))


def ring_simulate_fused(plan, d, grads, out, stream=None):
    """The single-GPU fused variant (cerar_ring_simulate_fused)."""
    _rows(grads, "grads", plan.N, d)
    _rows(out, "out", plan.N, d)
    _check(lib().cerar_ring_simulate_fused(plan.handle, d, _ptr(grads), _ld(grads), _ptr(out), _ld(out),
                                           _stream(stream)))


def ring_simulate_bucketed(plan, buckets, grads, work, ws, out, stream=None):
    span = max((b[0] + b[1] for b in buckets), default=0)
    work_floats, ws_bytes = plan.bucketed_sizes([b[1] for b in buckets])
    _rows(grads, "grads", plan.N, span)
    _rows(work, "work", plan.N, work_floats)
    _bytes(ws, "ws", ws_bytes)
    _rows(out, "out", plan.N, span)
    offs = (_SZ * len(buckets))(*[b[0] for b in buckets])
    lens = (_SZ * len(buckets))(*[b[1] for b in buckets])
    _check(lib().cerar_ring_simulate_bucketed(plan.handle, len(buckets), offs, lens, _ptr(grads), _ld(grads),
                                              _ptr(work), _ld(work), _ptr(ws), _ptr(out), _ld(out),
                                              _stream(stream)))


def error_norms(N, d, grads, out, norms, stream=None):
    _rows(grads, "grads", N, d)
    _rows(out, "out", N, d)
    _on_device(norms, "norms")
    if str(norms.dtype) != "torch.float64" or not norms.is_contiguous() or norms.numel() < N + 1:
        raise ValueError(f"norms must be a contiguous float64 tensor of at least {N + 1} entries")
    _check(lib().cerar_error_norms(N, d, _ptr(grads), _ld(grads), _ptr(out), _ld(out), _ptr(norms),
                                   _stream(stream)))


def sampled_norms(N, d, idx, ref, out, norms, stream=None):
    """K5's parity term (cerar_sampled_norms): idx an int64 device tensor of
    flat output indices, ref an (N, len(idx)) float64 device tensor, norms a
    float64 device tensor of 2N entries."""
    _rows(out, "out", N, d)
    _on_device(idx, "idx")
    _on_device(ref, "ref")
    _on_device(norms, "norms")
    if str(idx.dtype) != "torch.int64" or idx.dim() != 1 or not idx.is_contiguous() or idx.numel() == 0:
        raise ValueError("idx must be a non-empty contiguous 1-D int64 tensor")
    if str(ref.dtype) != "torch.float64" or not ref.is_contiguous() or tuple(ref.shape) != (N, idx.numel()):
        raise ValueError(f"ref must be a contiguous float64 tensor of shape ({N}, {idx.numel()})")
    if str(norms.dtype) != "torch.float64" or not norms.is_contiguous() or norms.numel() < 2 * N:
        raise ValueError(f"norms must be a contiguous float64 tensor of at least {2 * N} entries")
    _check(lib().cerar_sampled_norms(N, idx.numel(), d, _ptr(idx), _ptr(ref), _ptr(out), _ld(out), _ptr(norms),
                                     _stream(stream)))


def copy_f32(dst, src, stream=None):
    for t, name in ((dst, "dst"), (src, "src")):
        _on_device(t, name)
        if str(t.dtype) != "torch.float32" or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 tensor")
    if dst.numel() != src.numel():
        raise ValueError(f"dst has {dst.numel()} elements, src {src.numel()}")
    _check(lib().cerar_copy_f32(_ptr(dst), _ptr(src), dst.numel(), _stream(stream)))


_SYNTH_TABLES = {}


def _synth_tables(wl, device):
    """Device copies of a workload's tensor offsets and scales (cached)."""
    import torch
    k = (id(wl), str(device))
    if k not in _SYNTH_TABLES:
        offs = torch.as_tensor(np.ascontiguousarray(wl._offsets, dtype=np.int64), device=device)
        scales = torch.as_tensor(np.ascontiguousarray(wl._scales, dtype=np.float32), device=device)
        _SYNTH_TABLES[k] = (wl, offs, scales)
    return _SYNTH_TABLES[k][1:]


def synth_fill(out, wl, worker, start=0, stream=None):
    """Entries [start, start + out.numel()) of the workload's gradient of
    `worker` into the contiguous float32 device tensor `out`, generated by
    the library's K6 kernel (cerar_synth_fill); the same bits as
    wl.values_np(worker, indices)."""
    _on_device(out, "out")
    if str(out.dtype) != "torch.float32" or not out.is_contiguous():
        raise ValueError("out must be a contiguous float32 tensor")
    offs, scales = _synth_tables(wl, out.device)
    thr = wl.outlier_threshold if wl.outlier_prob > 0 else 0
    _check(lib().cerar_synth_fill(_ptr(out), out.numel(), int(start), int(wl.d), int(wl.worker_key(worker)),
                                  _ptr(offs), _ptr(scales), int(scales.numel()), int(thr),
                                  float(wl.outlier_factor), _stream(stream)))
    return out


def algorithmic_bytes_per_worker(N, c, p):
    """Bytes one worker must move under handoff sends: encode (2c+1)p,
    rounds (4c+2N-9)p, decode (2c+N-1)p, all fp32."""
    return (8 * c + 3 * N - 9) * p * 4


def phase_bytes_per_worker(N, c, p):
    """Per-launch algorithmic fp32 bytes of each phase for one worker."""
    L = c + N - 2
    rounds = {}
    for k in range(1, L + 1):
        if k <= N - 1:
            rounds[k] = 3 * p * 4
        elif k < L:
            rounds[k] = (4 if k + 1 <= c else 3) * p * 4
        else:
            rounds[k] = 0
    return {"encode": (2 * c + 1) * p * 4, "rounds": rounds, "decode": (2 * c + N - 1) * p * 4}


def phase_flops_per_worker(N, c, p):
    L = c + N - 2
    return {"encode": 2 * c * c * p, "decode": 2 * (L + 1) * c * p}


def isfinite(x):
    return math.isfinite(x)
