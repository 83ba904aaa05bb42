"""__graft_entry__.build() on a copy of the tree that holds no built library:
the package refuses to import until libkvio.so exists, so build() must not
import it before compiling (hipcc cross-compiles for gfx950 without a GPU)."""
import os
import shutil
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# what build() compiles and imports: the package, the oracle, the C ABI header
SOURCES = ("paper_2508_18572_amd", "oracle", "include")


def _ignore(_dir, names):
    return [n for n in names if n == "__pycache__" or n.endswith(".so")]


def test_build_from_a_clean_tree(tmp_path):
    tree = tmp_path / "tree"
    tree.mkdir()
    for d in SOURCES:
        shutil.copytree(os.path.join(ROOT, d), tree / d, ignore=_ignore)
    shutil.copy(os.path.join(ROOT, "__graft_entry__.py"), tree / "__graft_entry__.py")
    assert not (tree / "paper_2508_18572_amd" / "libkvio.so").exists()
    r = subprocess.run([sys.executable, "-c", "import __graft_entry__ as g; g.build()"], cwd=tree,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    assert (tree / "paper_2508_18572_amd" / "libkvio.so").exists()
    assert (tree / "oracle" / "liboracle.so").exists()
