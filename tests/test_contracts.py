"""Host-side contracts of the package (no GPU needed):

  * the product path (the package and its HIP sources) never imports, links or
    reads the oracle, and the oracle never imports the product;
  * the binding refuses to load when the HIP library has not been built, rather
    than falling back to anything else;
  * bench.py measures one GPU and refuses more, with a message.
"""
import ast
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_13804_amd")
ORACLE = os.path.join(ROOT, "oracle")


def _imported_modules(path):
    tree = ast.parse(open(path).read(), filename=path)
    names = set()
    for node in ast.walk(tree):
        if isinstance(node, ast.Import):
            names.update(a.name.split(".")[0] for a in node.names)
        elif isinstance(node, ast.ImportFrom) and node.level == 0 and node.module:
            names.add(node.module.split(".")[0])
    return names


def _py_files(top):
    for dirpath, _, files in os.walk(top):
        for f in files:
            if f.endswith(".py"):
                yield os.path.join(dirpath, f)


def test_product_never_imports_the_oracle():
    for path in _py_files(PKG):
        assert "oracle" not in _imported_modules(path), path
    for dirpath, _, files in os.walk(os.path.join(PKG, "csrc")):
        for f in files:
            text = open(os.path.join(dirpath, f)).read()
            assert "oracle" not in text.lower(), os.path.join(dirpath, f)


def test_oracle_never_imports_the_product():
    for path in _py_files(ORACLE):
        mods = _imported_modules(path)
        assert "paper_2609_13804_amd" not in mods, path
        assert "torch" not in mods, path


def test_binding_refuses_to_load_without_the_library(tmp_path):
    pkg = tmp_path / "paper_2609_13804_amd"
    pkg.mkdir()
    for f in ("__init__.py", "binding.py"):
        shutil.copy(os.path.join(PKG, f), pkg / f)
    r = subprocess.run([sys.executable, "-c", "import paper_2609_13804_amd.binding"],
                       cwd=tmp_path, capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "libstepprune.so is missing" in r.stderr


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}),
                                      ([], {"WORLD_SIZE": "2"})])
def test_bench_refuses_more_than_one_gpu(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + argv,
                       cwd=ROOT, capture_output=True, text=True, timeout=120,
                       env={**os.environ, **env})
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
