"""The build entry point in a fresh checkout: the library is git-ignored, so it
does not exist before the first build, and the package refuses to import
without it.  build() must still compile it and then import the package."""
import os
import shutil
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_build_works_without_a_built_library(tmp_path):
    repo = tmp_path / "repo"
    shutil.copytree(os.path.join(ROOT, "paper_2606_17421_amd"), repo / "paper_2606_17421_amd",
                    ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    shutil.copytree(os.path.join(ROOT, "include"), repo / "include")
    shutil.copy(os.path.join(ROOT, "__graft_entry__.py"), repo)
    assert not (repo / "paper_2606_17421_amd" / "libckkslinear.so").exists()
    code = "import __graft_entry__ as g; g.build(); import paper_2606_17421_amd as ck; print(ck.LIB_PATH)"
    res = subprocess.run([sys.executable, "-c", code], cwd=repo, capture_output=True, text=True, timeout=900)
    assert res.returncode == 0, res.stderr[-3000:]
    lib = repo / "paper_2606_17421_amd" / "libckkslinear.so"
    assert lib.exists() and lib.stat().st_size > 0
    assert res.stdout.strip().endswith(str(lib))
