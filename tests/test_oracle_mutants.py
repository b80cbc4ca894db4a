"""The oracle's pins catch plausible mistakes in it.

Each case plants one mistake in a copy of oracle/ (a wrong index or sign, a
transposed operand, a dropped or shifted term, a wrong constant), then runs
the pin tests (tests/test_oracle_protocol.py, tests/test_oracle_plan.py) on
that copy: they must fail.  The unplanted copy must pass first.  Nothing here
touches the product library or a GPU."""

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

from conftest import ROOT

PINS = ["test_oracle_protocol.py", "test_oracle_plan.py"]

# (file, original text, planted text, the mistake it models)
MUTANTS = [
    ("ring.py", "C[i] = C[i] + D[i][k - 1]", "C[i] = C[i] + D[i][k % c]",
     "Algorithm 1 step 1 adds the wrong encoded chunk"),
    ("ring.py", "C[i] = C[i] - D[i][j - 1]", "C[i] = C[i] + D[i][j - 1]",
     "step 2 adds where it must subtract"),
    ("ring.py", "C[i] = sent[(i - 1) % N].copy()", "C[i] = sent[(i + 1) % N].copy()",
     "the ring runs the wrong way"),
    ("ring.py", "Delta[(i - 1 - t) % N]", "Delta[(i - t) % N]",
     "the closed-form route's worker index is off by one"),
    ("ring.py", "return np.asarray(G, dtype=np.float64) @ np.asarray(U, dtype=np.float64)",
     "return np.asarray(G, dtype=np.float64) @ np.asarray(U, dtype=np.float64).T",
     "the encoder is transposed"),
    ("ring.py", "if k <= N - 1:\n                Bstore", "if k <= N - 2:\n                Bstore",
     "one B observation too few"),
    ("ring.py", "padded[:d] = g", "padded[:d] = g; padded[d:] = 1.0",
     "the pad is not zero"),
    ("ring.py", "return np.sum(np.asarray(grads, dtype=np.float64), axis=0)",
     "return np.sum(np.asarray(grads, dtype=np.float64)[1:], axis=0)",
     "the exact sum drops a worker"),
    ("plan.py", "col0 = N - 1 - r", "col0 = r",
     "the coefficient map places blocks in the wrong columns"),
    ("plan.py", "V_k = mpc_window(B, D, N - 1 - k)", "V_k = mpc_window(B, D, k)",
     "eq. (10) inverts the wrong window"),
    ("plan.py", "R[i, ell] = mpc_row(B, D, ell - i)", "R[i, ell] = mpc_row(B, D, ell + i)",
     "eq. (11) shifts the decoder rows the wrong way"),
    ("plan.py", "m, r = divmod(idx, N)", "m, r = divmod(abs(idx), N)",
     "negative sequence indices use D instead of its inverse"),
    ("plan.py", "rhs += W.T", "rhs += W",
     "the U-step's right-hand side is transposed"),
    ("plan.py", "W = R[(k - r) % N][s:s + c, :]", "W = R[(k + r) % N][s:s + c, :]",
     "the U-step reads the wrong worker's decoder"),
    ("plan.py", "return centre / half, centre * half", "return centre / half, centre * half * 2",
     "the projection interval misses the kappa bound"),
    ("plan.py", "B = np.vstack([z ** ell for ell in range(N)])",
     "B = np.vstack([z ** (ell + 1) for ell in range(N)])",
     "the Vandermonde base starts at the wrong power"),
    ("plan.py", "D = np.diag(z ** N)", "D = np.diag(z ** (N - 1))",
     "the Vandermonde D has the wrong power"),
    ("plan.py", "U[(i + r) % N]", "U[(i - r) % N]",
     "M_i pairs encoders with the wrong workers"),
    ("plan.py", "upper = upper + lower @ Dinv", "upper = upper + lower",
     "the Prop. 1 block identity drops D^-1"),
    ("plan.py", "return N * (N - 1) / 2.0 * float(np.sum(E * E))",
     "return N * (N + 1) / 2.0 * float(np.sum(E * E))",
     "the Prop. 2 constant is wrong"),
    ("plan.py", "return np.eye(H.shape[0]) + eps * H", "return np.eye(H.shape[0]) - eps * H",
     "the O(eps) perturbation has the wrong sign"),
    ("plan.py", "return (c + (N - 1) + 1) / c", "return (c + (N - 1)) / c",
     "the storage rate misses one observation"),
    ("plan.py", "E = [(ell + t) % N for t in range(s)]", "E = [(ell + t + 1) % N for t in range(s)]",
     "K^(l) takes the wrong remainder class rows"),
    ("plan.py", "blocks.append((B @ np.linalg.matrix_power(H, beta))[E])",
     "blocks.append((B @ np.linalg.matrix_power(H, beta - 1))[E])",
     "K^(l)'s last rows use the wrong power of H"),
    ("plan.py", "return min(float(np.linalg.svd(k_matrix(B, H, ell), compute_uv=False)[-1]) for ell in range(N))",
     "return min(float(np.linalg.svd(k_matrix(B, H, ell), compute_uv=False)[0]) for ell in range(N))",
     "gamma takes the largest singular value"),
    ("plan.py", "        if g > best:\n            best, best_t = g, t",
     "        if best < 0 or g < best:\n            best, best_t = g, t",
     "the H choice takes the smallest gamma"),
]


def _copy_tree(dst):
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(dst, "oracle"),
                    ignore=shutil.ignore_patterns("__pycache__"))
    os.makedirs(os.path.join(dst, "tests"))
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(dst, "tests", "golden"))
    for f in PINS + ["conftest.py"]:
        shutil.copy(os.path.join(ROOT, "tests", f), os.path.join(dst, "tests", f))


def _run_pins(dst):
    env = dict(os.environ, OMP_NUM_THREADS="2", OPENBLAS_NUM_THREADS="2", PYTHONDONTWRITEBYTECODE="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        *[os.path.join("tests", f) for f in PINS]],
                       cwd=dst, capture_output=True, text=True, env=env, timeout=600)
    return r.returncode, (r.stdout.strip().splitlines() or [""])[-1]


def test_every_planted_mistake_fails_the_pins(tmp_path):
    base = str(tmp_path / "base")
    _copy_tree(base)
    rc, last = _run_pins(base)
    assert rc == 0, f"the unplanted oracle must pass its pins: {last}"

    def one(k):
        f, a, b, why = MUTANTS[k]
        dst = str(tmp_path / f"m{k}")
        _copy_tree(dst)
        path = os.path.join(dst, "oracle", f)
        src = open(path).read()
        if src.count(a) != 1:
            return k, None, f"text to mutate not found once in oracle/{f}: {a!r}"
        with open(path, "w") as fh:
            fh.write(src.replace(a, b, 1))
        rc, last = _run_pins(dst)
        shutil.rmtree(dst, ignore_errors=True)
        return k, rc, last

    with ThreadPoolExecutor(4) as ex:
        results = list(ex.map(one, range(len(MUTANTS))))
    missing = [(MUTANTS[k][3], msg) for k, rc, msg in results if rc is None]
    survived = [MUTANTS[k][3] for k, rc, _ in results if rc == 0]
    assert not missing, missing
    assert not survived, f"mistakes the pins did not catch: {survived}"
