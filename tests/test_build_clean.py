"""__graft_entry__.build() on a copy of the tree that holds no built library:
the package refuses to import until libkvio.so exists, so build() must not
import it before compiling (hipcc cross-compiles for gfx950 without a GPU)."""
import os
import shutil
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SKIP = {".git", "_work", "gpurun_out", "__pycache__", ".pytest_cache"}


def _ignore(_dir, names):
    return [n for n in names if n in SKIP or n.endswith(".so")]


def test_build_from_a_clean_tree(tmp_path):
    tree = tmp_path / "tree"
    shutil.copytree(ROOT, tree, ignore=_ignore)
    assert not (tree / "paper_2508_18572_amd" / "libkvio.so").exists()
    r = subprocess.run([sys.executable, "-c", "import __graft_entry__ as g; g.build()"], cwd=tree,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    assert (tree / "paper_2508_18572_amd" / "libkvio.so").exists()
    assert (tree / "oracle" / "liboracle.so").exists()
