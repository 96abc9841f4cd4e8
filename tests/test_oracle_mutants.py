"""The oracle's pins catch plausible mistakes.

Each case plants one plausible mistake in a copy of the oracle (a dropped
term, a wrong comparison, a transposed operand, a reversed bit order, ...)
and runs the oracle's pins (``tests/test_oracle.py``,
``tests/test_oracle_planted.py``) against the copy in a separate process: at
least one pin must fail.  A pin set that passed a planted mistake would not
pin the oracle.

One mistake of this kind is equivalent and is not listed:
``gate_truly_positive`` deciding uncertain rows by ``approx >= 0`` instead
of ``approx > 0`` gives the same results, because a row whose float64 sum is
exactly 0 is always within the rounding bound and so always settled by the
exact sum instead.
"""

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle", "sparseinfer_ref.py")

# (what the mistake is, text in the oracle, the mistaken text)
MUTANTS = [
    ("N_pos from the padded width", "return n_neg, d - n_neg",
     "return n_neg, 32 * packed_w.shape[-1] - n_neg"),
    ("ties of Eq. (2) counted as sparse", "sparse = (a * n_pos.astype(np.float64)) < n_neg.astype(np.float64)",
     "sparse = (a * n_pos.astype(np.float64)) <= n_neg.astype(np.float64)"),
    ("batch mask as intersection", "mask = active.any(axis=0).astype(np.uint8)",
     "mask = active.all(axis=0).astype(np.uint8)"),
    ("W_down not transposed", "w_up[keep])               # [n][d]\n    WdT = fp16_to_f64(w_down[:, keep]).T",
     "w_up[keep])               # [n][d]\n    WdT = fp16_to_f64(w_down.T[:, keep]).T"),
    ("no ReLU in the gated MLP", "h1_kept = np.maximum(g_kept, 0.0)          # sigma = ReLU",
     "h1_kept = g_kept          # sigma = ReLU"),
    ("bit order reversed in the packed words", "place = np.left_shift(np.uint64(1), np.arange(32, dtype=np.uint64))\n"
     "    return (bits.astype", "place = np.left_shift(np.uint64(1), np.arange(31, -1, -1, dtype=np.uint64))\n"
     "    return (bits.astype"),
    ("bit 14 taken as the sign", "return (_as_u16(a) >> np.uint16(15)).astype(np.uint32)",
     "return (_as_u16(a) >> np.uint16(14) & np.uint16(1)).astype(np.uint32)"),
    ("h1 * g instead of h1 * u", "h3_kept = h1_kept * u_kept                 # step 3",
     "h3_kept = h1_kept * g_kept                 # step 3"),
    ("W_up work counted on h1 >= 0", '"n_up": int((h1_kept > 0).any(axis=0).sum()),',
     '"n_up": int((g_kept >= 0).any(axis=0).sum()),'),
    ("alpha taken in float64, not as its float32 value", "a = float(np.float32(alpha))", "a = float(alpha)"),
    ("no ReLU in the non-gated MLP", "h_kept = np.maximum(g_kept, 0.0)           # sigma = ReLU",
     "h_kept = g_kept           # sigma = ReLU"),
    ("RMSNorm without eps", "X = H / np.sqrt(ms + float(np.float32(eps))) * Wn[None, :]",
     "X = H / np.sqrt(ms) * Wn[None, :]"),
    ("residual dropped in the decoder block",
     'out["y"] = np.atleast_2d(np.asarray(h, dtype=np.float32)).astype(np.float64) + out["mlp_y"]',
     'out["y"] = out["mlp_y"]'),
    ("INT8 scale of max/128", "scale = (amax / np.float32(127.0)).astype(np.float32)",
     "scale = (amax / np.float32(128.0)).astype(np.float32)"),
    ("INT8 sign from bit 6", "return (np.asarray(q, dtype=np.int8).view(np.uint8) >> 7).astype(np.uint32)",
     "return (np.asarray(q, dtype=np.int8).view(np.uint8) >> 6 & 1).astype(np.uint32)"),
    ("INT8 W_down scales on the wrong axis", "WdT = dequantize_int8(q_down[:, keep], s_down).T",
     "WdT = dequantize_int8(q_down[:, keep].T, np.resize(np.asarray(s_down), keep.size))"),
    ("precision and recall swapped", '"precision": both_sparse / n_pred_sparse if n_pred_sparse else 1.0,',
     '"precision": both_sparse / n_true_sparse if n_true_sparse else 1.0,'),
]

PINS = ["tests/test_oracle.py", "tests/test_oracle_planted.py"]


def _run_mutant(tmp_root, i, old, new):
    """Copy the oracle, its pins and the input generators to a directory of
    their own, plant the mistake and run the pins; returns (exit code, tail)."""
    d = os.path.join(tmp_root, f"m{i}")
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(d, "oracle"),
                    ignore=shutil.ignore_patterns("__pycache__"))
    shutil.copytree(os.path.join(ROOT, "tests"), os.path.join(d, "tests"),
                    ignore=shutil.ignore_patterns("__pycache__", "test_gpu_*", "test_oracle_mutants.py"))
    shutil.copytree(os.path.join(ROOT, "paper_2411_12692_amd"), os.path.join(d, "paper_2411_12692_amd"),
                    ignore=shutil.ignore_patterns("__pycache__", "_build", "csrc", "*.so"))
    path = os.path.join(d, "oracle", "sparseinfer_ref.py")
    src = open(path).read()
    assert src.count(old) == 1, old
    open(path, "w").write(src.replace(old, new))
    env = dict(os.environ, OMP_NUM_THREADS="1", OPENBLAS_NUM_THREADS="1", MKL_NUM_THREADS="1")
    p = subprocess.run([sys.executable, "-m", "pytest", *PINS, "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu"], cwd=d, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True, timeout=600)
    return p.returncode, p.stdout.strip().splitlines()[-1:] if p.stdout.strip() else []


def test_every_mutant_text_is_in_the_oracle():
    src = open(ORACLE).read()
    for what, old, _ in MUTANTS:
        assert src.count(old) == 1, what


def test_every_planted_mistake_fails_a_pin(tmp_path):
    workers = max(1, min(6, (os.cpu_count() or 2) - 1))
    with cf.ThreadPoolExecutor(max_workers=workers) as ex:
        futs = {ex.submit(_run_mutant, str(tmp_path), i, old, new): what
                for i, (what, old, new) in enumerate(MUTANTS)}
        results = {futs[f]: f.result() for f in cf.as_completed(futs)}
    survived = {what: tail for what, (rc, tail) in results.items() if rc == 0}
    broken = {what: tail for what, (rc, tail) in results.items() if rc not in (0, 1)}
    assert not broken, f"pins did not run on these mutants: {broken}"
    assert not survived, f"no pin fails for: {sorted(survived)}"
