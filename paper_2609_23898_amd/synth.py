"""Seeded synthetic inputs: gradients shaped like the paper's workloads, the
random base matrix of the O(eps) plan and candidate node permutations for
its perturbation.

This module is the only code that both the HIP library's callers and the
oracle's callers use.  It contains none of the method's arithmetic.  It only
makes numbers.  Every value is a pure function of (seed, stream, index):

* a counter-based splitmix64 hash (Steele, Lea & Flood, "Fast splittable
  pseudorandom number generators", OOPSLA 2014; the 64-bit finaliser constants
  as published with splitmix64) gives 64 random bits per counter;
* a gradient entry's standard normal value comes from the Box-Muller
  transform (Box & Muller, "A note on the generation of random normal
  deviates", Ann. Math. Statist. 1958), z = sqrt(-2 ln u1) cos(2 pi u2), of
  two 53-bit uniforms.  The logarithm (an atanh series after an exact
  binary split) and the cosine (an octant reduction that is exact and Taylor
  series on [0, pi/4]) are written out here in IEEE double additions,
  multiplications and divisions in a fixed order, and the square root is
  the correctly rounded one, so the library's device generator
  (cerar_synth_fill, which computes the same steps without fused
  multiply-adds) produces the same bits.  The tails reach |z| = 8.57;
* the plan-side numbers (the random base matrix, the per-tensor log-normal
  scales) use an Irwin-Hall sum of twelve 32-bit uniforms minus 6 instead,
  computed exactly in integers: approximately normal, bounded at 6;
* a gradient entry is float32(normal * scale), where the scale comes from a
  per-tensor table computed once on the host.  Every path does the same
  single float64 product and the same single rounding to float32.

The workloads mirror the paper's experiments: Pythia-1.4B shaped gradients
(24 layers, d_model 2048, vocabulary 50304, d = 1,414,647,808) and a 12-layer
GPT-2-small shape (d = 124,439,808) with log-normal per-tensor scales; i.i.d.
cases; and a heavy-tailed case with 1 % of entries scaled by 100.  They stand
in for the paper's TinyStories training gradients, which are not used here.
"""

import math
from dataclasses import dataclass, field

import numpy as np

_MASK64 = (1 << 64) - 1
_GOLDEN = 0x9E3779B97F4A7C15
_MUL1 = 0xBF58476D1CE4E5B9
_MUL2 = 0x94D049BB133111EB
_HASHES_PER_ENTRY = 8            # 6 for the normal, 1 for the outlier mask, 1 spare
_SCALE_STREAM = 0x5CA1E
_BASE_STREAM = 0xBA5E
_PERM_STREAM = 0x9E7

DDP_BUCKET_FLOATS = 25 * 1024 * 1024 // 4    # 25 MiB of fp32, DDP's default cap


def _mix64_int(z):
    """splitmix64 finaliser on a Python int (mod 2^64)."""
    z &= _MASK64
    z = ((z ^ (z >> 30)) * _MUL1) & _MASK64
    z = ((z ^ (z >> 27)) * _MUL2) & _MASK64
    return z ^ (z >> 31)


def stream_key(seed, stream):
    """64-bit key of one independent stream (e.g. one worker's gradient)."""
    return _mix64_int(_mix64_int((seed * _GOLDEN + 1) & _MASK64) ^ ((stream * _MUL2) & _MASK64))


# --- NumPy path (uint64 arithmetic wraps by definition) ---------------------

def _mix64_np(z):
    z = z ^ (z >> np.uint64(30))
    z = z * np.uint64(_MUL1)
    z = z ^ (z >> np.uint64(27))
    z = z * np.uint64(_MUL2)
    return z ^ (z >> np.uint64(31))


def _hash_np(key, idx, j):
    ctr = idx.astype(np.uint64) * np.uint64(_HASHES_PER_ENTRY) + np.uint64(j + 1)
    with np.errstate(over="ignore"):
        return _mix64_np(np.uint64(key) + ctr * np.uint64(_GOLDEN))


def normal_np(key, idx):
    """Irwin-Hall(12) - 6 at the given counters, float64, exact."""
    idx = np.asarray(idx, dtype=np.int64)
    total = np.zeros(idx.shape, dtype=np.int64)
    with np.errstate(over="ignore"):
        for j in range(6):
            h = _hash_np(key, idx, j)
            total += (h & np.uint64(0xFFFFFFFF)).astype(np.int64)
            total += (h >> np.uint64(32)).astype(np.int64)
    return (total + 6 - 6 * (1 << 32)).astype(np.float64) * 2.0 ** -32


# Box-Muller in IEEE double operations in a fixed order (no fused
# multiply-add, no library transcendental), mirrored step for step by the
# device generator.
_LN2 = 0.693147180559945309417
_SQRT_HALF = 0.707106781186547524401
_PI_4 = 0.785398163397448309616


def _taylor_coefficients(first, count):
    """(-1)^k / n! for n = first + 2k: n! as an exact double product
    (n <= 18, below the 2^53 limit), then one division."""
    out = []
    for k in range(count):
        n = first + 2 * k
        f = 1.0
        for i in range(2, n + 1):
            f = f * float(i)
        out.append((-1.0 if k % 2 else 1.0) / f)
    return out


_COS_C = _taylor_coefficients(0, 10)     # 1/0!, -1/2!, ..., 1/18!
_SIN_C = _taylor_coefficients(1, 9)      # 1/1!, -1/3!, ..., 1/17!
_ATANH_N = 11                        # odd terms t^(2k+1)/(2k+1), k < 11


def _ln_unit_np(u):
    """ln u for u in (0, 1]: u = m 2^e exactly with m in [sqrt(1/2), sqrt(2)),
    ln m = 2 atanh(t), t = (m - 1) / (m + 1), |t| <= 0.172."""
    m, e = np.frexp(u)
    low = m < _SQRT_HALF
    m = np.where(low, m * 2.0, m)
    e = np.where(low, e - 1, e).astype(np.float64)
    t = (m - 1.0) / (m + 1.0)
    t2 = t * t
    acc = np.full(u.shape, 1.0 / float(2 * _ATANH_N - 1))
    for k in range(_ATANH_N - 2, -1, -1):
        acc = acc * t2 + 1.0 / float(2 * k + 1)
    return e * _LN2 + 2.0 * (t * acc)


def _cos_2pi_np(w8, o):
    """cos(2 pi u) from w8 = 8u (exact) and its octant o = floor(w8): with
    f = w8 - o, phi = (f or 1 - f) pi/4 in [0, pi/4] and a sign."""
    f = w8 - o
    odd = (o % 2) == 1
    a = np.where(odd, 1.0 - f, f)
    phi = a * _PI_4
    p2 = phi * phi
    c = np.full(phi.shape, _COS_C[-1])
    for k in range(len(_COS_C) - 2, -1, -1):
        c = c * p2 + _COS_C[k]
    s = np.full(phi.shape, _SIN_C[-1])
    for k in range(len(_SIN_C) - 2, -1, -1):
        s = s * p2 + _SIN_C[k]
    s = s * phi
    use_sin = np.isin(o, (1, 2, 5, 6))
    neg = np.isin(o, (2, 3, 4, 5))
    v = np.where(use_sin, s, c)
    return np.where(neg, -v, v)


def gauss_np(key, idx):
    """Box-Muller standard normal at the given counters, float64: u1 from
    hash slot 0 in (0, 1], u2 from slot 1 in [0, 1), 53 bits each."""
    idx = np.asarray(idx, dtype=np.int64)
    with np.errstate(over="ignore"):
        h1 = _hash_np(key, idx, 0)
        h2 = _hash_np(key, idx, 1)
    u1 = ((h1 >> np.uint64(11)) + np.uint64(1)).astype(np.float64) * 2.0 ** -53
    i2 = (h2 >> np.uint64(11)).astype(np.int64)
    o = (i2 >> 50).astype(np.int64)                    # floor(8 u2)
    w8 = i2.astype(np.float64) * 2.0 ** -50            # 8 u2, exact
    r = np.sqrt(-2.0 * _ln_unit_np(u1))
    return r * _cos_2pi_np(w8, o)


def uniform32_np(key, idx, j):
    """One 32-bit uniform integer per counter from hash slot j."""
    h = _hash_np(key, np.asarray(idx, dtype=np.int64), j)
    return (h & np.uint64(0xFFFFFFFF)).astype(np.int64)


# --- workloads ---------------------------------------------------------------

def gpt2_small_tensor_sizes():
    """Parameter sizes of a 12-layer GPT-2-small (d_model 768, 50257 tokens,
    1024 positions, tied output embedding), in parameter order."""
    d, ff, vocab, ctx = 768, 3072, 50257, 1024
    sizes = [vocab * d, ctx * d]
    for _ in range(12):
        sizes += [d, d,                 # ln_1 weight, bias
                  d * 3 * d, 3 * d,     # attention c_attn weight, bias
                  d * d, d,             # attention c_proj weight, bias
                  d, d,                 # ln_2 weight, bias
                  d * ff, ff,           # mlp c_fc weight, bias
                  ff * d, d]            # mlp c_proj weight, bias
    sizes += [d, d]                     # ln_f weight, bias
    return sizes


def pythia_1_4b_tensor_sizes():
    """Parameter sizes of Pythia-1.4B (GPT-NeoX, 24 layers, d_model 2048,
    vocabulary 50304, untied output embedding), in parameter order."""
    d, ff, vocab = 2048, 8192, 50304
    sizes = [vocab * d]                 # embed_in
    for _ in range(24):
        sizes += [d, d,                 # input_layernorm weight, bias
                  d, d,                 # post_attention_layernorm weight, bias
                  3 * d * d, 3 * d,     # query_key_value weight, bias
                  d * d, d,             # attention dense weight, bias
                  ff * d, ff,           # dense_h_to_4h weight, bias
                  d * ff, d]            # dense_4h_to_h weight, bias
    sizes += [d, d, vocab * d]          # final_layer_norm weight, bias; embed_out
    return sizes


def ddp_buckets(tensor_sizes, cap=DDP_BUCKET_FLOATS):
    """Greedy DDP-style buckets over the flat gradient: tensors are visited in
    reverse parameter order; a bucket is closed when the next tensor would push
    it past ``cap`` floats, and a tensor larger than ``cap`` gets a bucket of its
    own.  Returns (offset, length) pairs in flat-index order."""
    offsets = np.concatenate([[0], np.cumsum(tensor_sizes)]).astype(np.int64)
    buckets = []
    cur_lo = cur_hi = None
    for t in reversed(range(len(tensor_sizes))):
        lo, hi = int(offsets[t]), int(offsets[t + 1])
        if cur_lo is None:
            cur_lo, cur_hi = lo, hi
        elif (cur_hi - lo) > cap:
            buckets.append((cur_lo, cur_hi - cur_lo))
            cur_lo, cur_hi = lo, hi
        else:
            cur_lo = lo
    if cur_lo is not None:
        buckets.append((cur_lo, cur_hi - cur_lo))
    return sorted(buckets)


@dataclass
class Workload:
    """One synthetic all-reduce: N workers, c chunks, length-d fp32 gradients.

    ``tensor_sizes`` (optional) splits the flat gradient into tensors, each
    with its own log-normal scale exp(z_t), z_t ~ N(0,1); otherwise every
    entry has scale ``scale``.  ``outlier_prob`` entries are multiplied by
    ``outlier_factor``.
    """
    name: str
    N: int
    c: int
    d: int
    seed: int
    scale: float = 1.0
    tensor_sizes: list = None
    outlier_prob: float = 0.0
    outlier_factor: float = 1.0
    buckets: list = None
    _offsets: np.ndarray = field(default=None, repr=False)
    _scales: np.ndarray = field(default=None, repr=False)

    def __post_init__(self):
        if self.tensor_sizes is not None:
            assert sum(self.tensor_sizes) == self.d, (sum(self.tensor_sizes), self.d)
            self._offsets = np.concatenate([[0], np.cumsum(self.tensor_sizes)]).astype(np.int64)
            key = stream_key(self.seed, _SCALE_STREAM)
            z = normal_np(key, np.arange(len(self.tensor_sizes)))
            self._scales = np.array([np.float32(math.exp(float(v))) for v in z], dtype=np.float32)
        else:
            self._offsets = np.array([0, self.d], dtype=np.int64)
            self._scales = np.array([np.float32(self.scale)], dtype=np.float32)

    @property
    def outlier_threshold(self):
        return int(math.floor(self.outlier_prob * 2.0 ** 32))

    def worker_key(self, worker):
        return stream_key(self.seed, 1000 + worker)

    def tensor_scales(self):
        return self._scales.copy()

    def values_np(self, worker, flat_idx):
        """float32 gradient entries of ``worker`` at flat indices (int array);
        indices >= d give 0 (the zero pad)."""
        flat_idx = np.asarray(flat_idx, dtype=np.int64)
        valid = flat_idx < self.d
        idx = np.where(valid, flat_idx, 0)
        key = self.worker_key(worker)
        n = gauss_np(key, idx)
        if self.outlier_prob > 0:
            hit = uniform32_np(key, idx, 6) < self.outlier_threshold
            n = np.where(hit, n * float(self.outlier_factor), n)
        t = np.searchsorted(self._offsets, idx, side="right") - 1
        s = self._scales[t].astype(np.float64)
        v = (n * s).astype(np.float32)
        return np.where(valid, v, np.float32(0.0))


def base_matrix(seed, N, c):
    """N x c base matrix B with i.i.d. approximately N(0,1) entries (the paper's
    choice of B for the O(eps) plan, appendix on the experiments), float64."""
    return normal_np(stream_key(seed, _BASE_STREAM), np.arange(N * c)).reshape(N, c)


def node_permutations(seed, count, c):
    """count x c int32 candidate permutations of the c plan nodes: row 0 is
    the identity, row t > 0 orders 0..c-1 by 64-bit hash keys of counters
    t*c .. t*c+c-1 (ties, which have probability ~c^2 2^-64, keep index order)."""
    perms = np.empty((count, c), dtype=np.int32)
    perms[0] = np.arange(c)
    key = stream_key(seed, _PERM_STREAM)
    for t in range(1, count):
        h = _hash_np(key, np.arange(t * c, (t + 1) * c, dtype=np.int64), 0)
        perms[t] = np.argsort(h, kind="stable")
    return perms


WORKLOADS = ("tiny-n4-c4", "iid-n8-c16-16m", "gpt2-small", "pythia-1.4b", "heavytail-n16-c128")
HEADLINE = "pythia-1.4b"


def workload(name):
    """The synthetic workloads, by name (WORKLOADS)."""
    if name == "tiny-n4-c4":
        return Workload("tiny N=4 c=4 d=4096 iid N(0,1)", 4, 4, 4096, seed=1)
    if name == "iid-n8-c16-16m":
        return Workload("N=8 c=16 d=2^24 iid N(0,1e-6)", 8, 16, 1 << 24, seed=2, scale=1e-3)
    if name == "gpt2-small":
        sizes = gpt2_small_tensor_sizes()
        return Workload("GPT-2-small N=8 c=32 d=124439808 lognormal tensors, 25MiB buckets",
                        8, 32, sum(sizes), seed=3, tensor_sizes=sizes,
                        buckets=ddp_buckets(sizes))
    if name == "pythia-1.4b":
        sizes = pythia_1_4b_tensor_sizes()
        return Workload("Pythia-1.4B N=8 c=64 d=1414647808 lognormal tensors",
                        8, 64, sum(sizes), seed=4, tensor_sizes=sizes)
    if name == "heavytail-n16-c128":
        return Workload("N=16 c=128 d=4e8 iid N(0,1), 1% x100 outliers", 16, 128,
                        400_000_000, seed=5, outlier_prob=0.01, outlier_factor=100.0)
    raise ValueError(f"unknown workload {name!r}; one of {WORKLOADS}")
