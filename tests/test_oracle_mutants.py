"""The oracle's pins catch plausible mistakes: each case plants one mistake in a copy of
oracle/ (an exact source substitution that must apply) and runs the pin tests
(tests/test_oracle_attention.py, tests/test_oracle_plan.py) on that copy in a fresh
process; the run must fail. An unmodified copy must pass, so a failure is the planted
mistake's."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = ["tests/test_oracle_attention.py", "tests/test_oracle_plan.py"]

# (file, original text, planted mistake, what the mistake is)
MUTANTS = [
    ("oracle/attention.py", "            g = h // G\n            s = sm_scale",
     "            g = h % hkv\n            s = sm_scale", "interleaved instead of contiguous GQA grouping"),
    ("oracle/attention.py", "w = np.exp(s - s.max())", "w = np.exp(s)", "softmax without the max subtraction"),
    ("oracle/attention.py", "s = sm_scale * (K[:, g, :]", "s = (K[:, g, :]", "softmax scale dropped"),
    ("oracle/attention.py", "out[i, h] = (w @ V[:, g, :]) / w.sum()", "out[i, h] = (w @ K[:, g, :]) / w.sum()",
     "K read in place of V"),
    ("oracle/attention.py", "rows = cache[pages].reshape(npages * page_size, hkv, d)[:n]",
     "rows = cache[pages].transpose(0, 2, 1, 3).reshape(npages * page_size, hkv, d)[:n]",
     "pages read as [page, head, slot, d]"),
    ("oracle/attention.py", "c = np.exp(ms_ - m)", "c = np.exp(m - ms_)", "merge weight with the exponent reversed"),
    ("oracle/attention.py", "a = a + c * as_", "a = a + as_", "merge without the rescale of the accumulators"),
    ("oracle/attention.py", "return -np.inf, 0.0, np.zeros(d, dtype=np.float64)",
     "return 0.0, 0.0, np.zeros(d, dtype=np.float64)", "empty split not the neutral state"),
    ("oracle/attention.py", "    m = x.max()\n", "    m = x.min()\n", "split state maximum taken as the minimum"),
    ("oracle/plan.py", "b1 = ((s + 1) * tiles) // k", "b1 = ((s + 1) * tiles + k - 1) // k",
     "split end rounded up (off by one)"),
    ("oracle/plan.py", "active = sum(1 for n in seq_lens if int(n) > 0)", "active = len(seq_lens)",
     "empty rows counted as active"),
    ("oracle/plan.py", "min(b1 * tile_tokens, int(n))", "b1 * tile_tokens", "last split not clamped to the length"),
    ("oracle/plan.py", "if p.num_kv_heads * count <= p.target_tasks:", "if count <= p.target_tasks:",
     "quota search ignores the KV heads"),
    ("oracle/plan.py", "return [min(S, t) for t in tiles], S", "return [min(S - 1, t) for t in tiles], S",
     "one split fewer than the split count S"),
    ("oracle/plan.py", "offsets.append(offsets[-1] + len(bounds))", "offsets.append(offsets[-1] + nsplit[i] + 1)",
     "split_offsets off by one per row"),
]


def _copy(dst):
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(dst, "oracle"),
                    ignore=shutil.ignore_patterns("__pycache__"))
    os.makedirs(os.path.join(dst, "tests"))
    for f in PINS + ["tests/conftest.py"]:
        shutil.copy(os.path.join(ROOT, f), os.path.join(dst, f))
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(dst, "tests", "golden"))
    shutil.copy(os.path.join(ROOT, "pytest.ini"), os.path.join(dst, "pytest.ini"))


def _run_pins(dst):
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *PINS],
                          cwd=dst, capture_output=True, text=True, timeout=600)


def test_unmodified_copy_passes(tmp_path):
    _copy(str(tmp_path))
    res = _run_pins(str(tmp_path))
    assert res.returncode == 0, res.stdout[-2000:]


@pytest.mark.parametrize("path,orig,mutant,what", MUTANTS, ids=[m[3] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, path, orig, mutant, what):
    _copy(str(tmp_path))
    f = os.path.join(str(tmp_path), path)
    src = open(f).read()
    assert src.count(orig) == 1, f"the substitution for '{what}' no longer applies"
    open(f, "w").write(src.replace(orig, mutant))
    res = _run_pins(str(tmp_path))
    assert res.returncode != 0, f"the pins did not catch: {what}"
