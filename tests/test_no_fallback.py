"""The product path has no CPU fallback: without libaspis.so every entry of
the binding raises, and the package never reaches the oracle."""
import ast
import os

import pytest

from paper_2108_02416_amd import aspis

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2108_02416_amd")


@pytest.fixture
def no_library(monkeypatch, tmp_path):
    monkeypatch.setattr(aspis, "LIB_PATH", str(tmp_path / "libaspis.so"))
    monkeypatch.setattr(aspis, "_lib", None)


@pytest.mark.parametrize("call", [
    lambda: aspis.lib(),
    lambda: aspis.num_files(15, 3),
    lambda: aspis.assign(15, 3),
    lambda: aspis.worker_rows(15, 3),
    lambda: aspis.simulate(15, 3, 4),
])
def test_missing_library_raises(no_library, call):
    with pytest.raises(ImportError, match="libaspis.so is missing"):
        call()


def test_missing_library_raises_before_any_device_work(no_library):
    import numpy as np
    rows = np.zeros((7, 1), dtype=np.uint64)
    with pytest.raises(ImportError):
        aspis.clique(rows, 7, 2)


def _imports(path):
    tree = ast.parse(open(path).read(), path)
    for node in ast.walk(tree):
        if isinstance(node, ast.Import):
            yield from (a.name for a in node.names)
        elif isinstance(node, ast.ImportFrom) and node.module:
            yield node.module


def test_package_never_imports_the_oracle():
    for name in os.listdir(PKG):
        if name.endswith(".py"):
            mods = list(_imports(os.path.join(PKG, name)))
            assert not any(m == "oracle" or m.startswith("oracle.") for m in mods), name
    # nor does the native library name any oracle source
    for name in os.listdir(os.path.join(PKG, "csrc")):
        text = open(os.path.join(PKG, "csrc", name)).read()
        assert '#include "oracle' not in text and "oracle.h" not in text, name
