"""Strength of the oracle's pins: each plausible single mistake in the oracle
(a flipped interval end, the opposite tie order, a doubled or dropped phi, a
wrong sign of the offset, the wrong RTN divisor or rounding, the count
rounding, a wrong prefix shift, no quantile interpolation, scales of the
wrong output, a transposed prefill operand, a LUT read without nesting, a
wrong calibration mean, the sign bit kept in the magnitude key, the planes,
fields or rows of the packed layout in another order) is planted
in a copy of the oracle, and the pin tests run against the copy must fail.

CPU only; the GPU library is not involved.
"""
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = ["tests/test_oracle_pins.py", "tests/test_oracle_pins_bmax.py", "tests/test_oracle_pins_lut.py"]

MUTATIONS = {
    "threshold interval ends": ("        inside = (th[k] <= ax) & (ax < th[k + 1])",
                                "        inside = (th[k] < ax) & (ax <= th[k + 1])"),
    "top-k ties to the higher index": ("        order = np.lexsort((idx, -key))",
                                       "        order = np.lexsort((-idx, -key))"),
    "phi doubled": ("    return float(2 ** (b_max - b - 1))", "    return float(2 ** (b_max - b))"),
    "phi kept at full depth": ("    if b >= b_max:\n        return 0.0", "    if b > b_max:\n        return 0.0"),
    "offset sign": ("    z = -float(2 ** (b_max - 1)) * s", "    z = float(2 ** (b_max - 1)) * s"),
    "RTN divisor": ("    s16 = (amax / np.float32(half - 1))", "    s16 = (amax / np.float32(half))"),
    "RTN truncation": ("        r = np.rint(w32 / s32[:, :, None])", "        r = np.trunc(w32 / s32[:, :, None])"),
    "count rounding": ("        C[j] = (U * K + 5000) // 10000", "        C[j] = (U * K) // 10000"),
    "prefix shift": ("    return q >> (b_max - b)\n", "    return q >> (b_max - b + 1)\n"),
    "no quantile interpolation": ("            hi_v = srt[min(lo + 1, n - 1)]", "            hi_v = srt[lo]"),
    "scales of the wrong output": (
        "    s_full = np.repeat(np.asarray(scales, dtype=np.float16).astype(np.float64).T,\n"
        "                       group, axis=1)                          # [N, K]\n    W = np.zeros",
        "    s_full = np.repeat(np.asarray(scales, dtype=np.float16).astype(np.float64).T[::-1],\n"
        "                       group, axis=1)                          # [N, K]\n    W = np.zeros"),
    "prefill tokens swapped": ("    return X @ W.T\n", "    return (X[::-1] @ W.T)\n"),
    "LUT read without nesting": ("        qb = nested_code(codes[:, cols], b, b_max)",
                                 "        qb = codes[:, cols] & ((1 << b) - 1)"),
    "calibration mean": ("    return (acc / np.float64(count)).astype(np.float32)",
                         "    return (acc / np.float64(count + 1)).astype(np.float32)"),
    "sign bit kept in the magnitude key": ("    return bits & 0x7FFF\n", "    return bits\n"),
    "planes least significant first": ("                    field = (q >> (b_max - j * u)) & mask",
                                       "                    field = (q >> ((j - 1) * u)) & mask"),
    "fields in reversed output order": ("                    bit = o * u\n",
                                        "                    bit = (tile_n - 1 - o) * u\n"),
    "rows channel-major across tiles": ("            row = (t * K + k) * R\n",
                                        "            row = (k * (N // tile_n) + t) * R\n"),
}


def _run_pins(mutation=None):
    """Copy the oracle, tests and inputs to a fresh directory, plant the
    mutation (if any) and run the pin tests there; returns the run."""
    with tempfile.TemporaryDirectory() as tmp:
        for d in ("oracle", "tests", "synth"):
            shutil.copytree(os.path.join(ROOT, d), os.path.join(tmp, d),
                            ignore=shutil.ignore_patterns("__pycache__", "*.so", "test_oracle_mutations.py"))
        if mutation is not None:
            old, new = mutation
            path = os.path.join(tmp, "oracle", "grinqh_oracle.py")
            with open(path) as f:
                src = f.read()
            assert src.count(old) == 1, "mutation site not found exactly once"
            with open(path, "w") as f:
                f.write(src.replace(old, new))
        return subprocess.run([sys.executable, "-m", "pytest", *PINS, "-q", "-x", "-m", "not gpu",
                               "-p", "no:cacheprovider"], cwd=tmp, capture_output=True, text=True,
                              timeout=600)


_RESULTS = {}


def _results():
    # every run at once, a few in parallel (each is an independent process)
    if not _RESULTS:
        names = [None] + sorted(MUTATIONS)
        with ThreadPoolExecutor(max_workers=min(5, os.cpu_count() or 1)) as ex:
            runs = list(ex.map(lambda n: _run_pins(MUTATIONS.get(n)), names))
        _RESULTS.update(zip(names, runs))
    return _RESULTS


def test_unmutated_copy_passes():
    # the control: the copied tree runs the pins cleanly, so a failure below
    # comes from the planted mistake and not from the copy
    r = _results()[None]
    assert r.returncode == 0, r.stdout[-800:]


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name):
    r = _results()[name]
    assert r.returncode == 1, f"no pin failed for: {name}\n{r.stdout[-400:]}"   # 1: tests failed
    assert " failed" in r.stdout, r.stdout[-400:]
