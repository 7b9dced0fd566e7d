"""The product path has no fallback (no GPU needed).

* Importing the package without its built HIP library raises ImportError that
  names the missing library, instead of running anything on the CPU.
* No module of the package imports, loads or runs the oracle: the oracle is
  test infrastructure only.
"""
import ast
import os
import shutil
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2608_21614_amd")


def test_import_without_the_library_raises(tmp_path):
    dst = tmp_path / "paper_2608_21614_amd"
    dst.mkdir()
    for name in os.listdir(PKG):
        if name.endswith(".py"):
            shutil.copy(os.path.join(PKG, name), dst / name)
    assert not (dst / "libsaem_moe.so").exists()
    env = dict(os.environ, PYTHONPATH=str(tmp_path))
    r = subprocess.run([sys.executable, "-c", "import paper_2608_21614_amd"], cwd=str(tmp_path), env=env,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "libsaem_moe.so is not built" in r.stderr, r.stderr[-2000:]


def test_package_never_touches_the_oracle():
    for name in sorted(os.listdir(PKG)):
        if not name.endswith(".py"):
            continue
        path = os.path.join(PKG, name)
        src = open(path).read()
        tree = ast.parse(src, filename=path)
        for node in ast.walk(tree):
            if isinstance(node, ast.Import):
                assert not any(a.name.split(".")[0] == "oracle" for a in node.names), f"{name} imports the oracle"
            elif isinstance(node, ast.ImportFrom):
                assert (node.module or "").split(".")[0] != "oracle", f"{name} imports the oracle"
        for needle in ("libmoe_oracle", "moe_oracle.c", "MOE_ORACLE_LIB", "import_module(\"oracle\")"):
            assert needle not in src, f"{name} names {needle}"
