"""Plant plausible mistakes in COPIES of the Python oracles (batch formation,
oracle/sched.py; storage tier, oracle/disk.py) and check that their pin tests
catch every one.  Each mutant runs the pin file in a subprocess against a
temporary copy of the oracle package; the committed oracle is never
modified."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (module, name, original text, replacement)
MUTANTS = [
    ("sched", "bundle_hits_never_join",
     "if state[pos] == _WAITING and c is not None and c in contexts_in_batch:", "if False:"),
    ("sched", "loading_bound_flipped",
     "return Fraction(load) > Fraction(ratio) * compute", "return Fraction(load) < Fraction(ratio) * compute"),
    ("sched", "loading_bound_rounded_to_double",
     "return Fraction(load) > Fraction(ratio) * compute", "return float(load) > ratio * float(compute)"),
    ("sched", "bundle_hit_load_counted",
     'return totals["load"] + (0 if shared else r.load_tokens)', 'return totals["load"] + r.load_tokens'),
    ("sched", "deprioritized_never_fill",
     "    for pos in range(n):             # set-aside", "    for pos in range(0):             # set-aside"),
    ("sched", "full_only_past_budget",
     'return totals["compute"] < max_tokens and', 'return totals["compute"] <= max_tokens and'),
    ("sched", "deferral_at_threshold",
     "deferred = [r.rid for r in queue if r.transient_matches > delay_hit_threshold]\n"
     "    eligible = [r for r in queue if r.transient_matches <= delay_hit_threshold]",
     "deferred = [r.rid for r in queue if r.transient_matches >= delay_hit_threshold]\n"
     "    eligible = [r for r in queue if r.transient_matches < delay_hit_threshold]"),
    ("sched", "deferred_go_last",
     "return batch, deferred + rest", "return batch, rest + deferred"),
    ("sched", "head_checked_like_the_rest",
     "    enter(0)                         # the head of the queue always starts the batch\n"
     "    enter_bundle_hits()\n    for pos in range(1, n):",
     "    for pos in range(0, n):"),
    ("sched", "rest_reversed",
     "rest = [queue[p].rid for p in range(n) if state[p] != _IN_BATCH]",
     "rest = [queue[p].rid for p in reversed(range(n)) if state[p] != _IN_BATCH]"),
    ("disk", "page_first_layer_page_swapped",
     "return (((page * num_layers + layer) * 2 + kv) * page_size + in_page) * row_bytes",
     "return (((layer * num_layers + page) * 2 + kv) * page_size + in_page) * row_bytes"),
    ("disk", "layer_first_stride_num_layers",
     "return (((layer * 2 + kv) * num_disk_pages + page) * page_size + in_page) * row_bytes",
     "return (((layer * 2 + kv) * num_layers + page) * page_size + in_page) * row_bytes"),
    ("disk", "in_page_dropped",
     "return (((page * num_layers + layer) * 2 + kv) * page_size + in_page) * row_bytes",
     "return (((page * num_layers + layer) * 2 + kv) * page_size) * row_bytes"),
    ("disk", "k_v_swapped_layer_first",
     "return (((layer * 2 + kv) * num_disk_pages + page) * page_size + in_page) * row_bytes",
     "return (((layer * 2 + (1 - kv)) * num_disk_pages + page) * page_size + in_page) * row_bytes"),
    ("disk", "host_token_not_scaled_by_page",
     "h = _host_off(host_layout, layer, kv, j * page_size + o, num_layers, page_size,\n"
     "                                      host_tokens, row_bytes)\n"
     "                        chunk[h:h + row_bytes]",
     "h = _host_off(host_layout, layer, kv, j + o, num_layers, page_size,\n"
     "                                      host_tokens, row_bytes)\n"
     "                        chunk[h:h + row_bytes]"),
]

PINS = {"sched": "test_oracle_sched.py", "disk": "test_oracle_disk.py"}

CONFTEST = """import os, sys
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
"""


@pytest.mark.parametrize("module,name,old,new", MUTANTS, ids=[f"{m[0]}-{m[1]}" for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, module, name, old, new):
    pkg = tmp_path / "oracle"
    shutil.copytree(os.path.join(ROOT, "oracle"), pkg, ignore=shutil.ignore_patterns("__pycache__"))
    src = (pkg / f"{module}.py").read_text()
    assert src.count(old) >= 1, f"mutant {name}: anchor text not found"
    (pkg / f"{module}.py").write_text(src.replace(old, new))
    tests = tmp_path / "tests"
    tests.mkdir()
    (tests / "conftest.py").write_text(CONFTEST)
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), tests / "golden")
    shutil.copy(os.path.join(ROOT, "tests", PINS[module]), tests / PINS[module])
    env = dict(os.environ)
    env.pop("PYTHONPATH", None)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        str(tests / PINS[module])], cwd=str(tmp_path), env=env,
                       capture_output=True, text=True, timeout=300)
    assert "passed" in r.stdout or "failed" in r.stdout, r.stdout[-2000:] + r.stderr[-2000:]
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"


def test_unmutated_copy_passes(tmp_path):
    """The harness itself: the same copy without a mutation passes both pin files."""
    shutil.copytree(os.path.join(ROOT, "oracle"), tmp_path / "oracle", ignore=shutil.ignore_patterns("__pycache__"))
    tests = tmp_path / "tests"
    tests.mkdir()
    (tests / "conftest.py").write_text(CONFTEST)
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), tests / "golden")
    for f in PINS.values():
        shutil.copy(os.path.join(ROOT, "tests", f), tests / f)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", str(tests)],
                       cwd=str(tmp_path), capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
