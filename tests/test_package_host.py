"""Host-side guarantees of the product path (no GPU needed): the binding
refuses to run without the HIP library, and no module of the package imports
the oracle (the oracle is test infrastructure; the package has no CPU
fallback)."""
import ast
import glob
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2010_13359_amd")


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    from paper_2010_13359_amd import dqgan
    monkeypatch.setattr(dqgan, "LIB_PATH", str(tmp_path / "libdqgan.so"))
    monkeypatch.setattr(dqgan, "_lib", None)
    with pytest.raises(ImportError, match="not built"):
        dqgan.load()


def _imported_modules(path):
    with open(path, encoding="utf-8") as f:
        tree = ast.parse(f.read(), path)
    for node in ast.walk(tree):
        if isinstance(node, ast.Import):
            for a in node.names:
                yield a.name
        elif isinstance(node, ast.ImportFrom):
            yield node.module or ""
            for a in node.names:
                yield a.name


def test_package_never_imports_the_oracle():
    sources = glob.glob(os.path.join(PKG, "**", "*.py"), recursive=True)
    assert sources
    for path in sources:
        for mod in _imported_modules(path):
            assert "oracle" not in mod.split("."), "%s imports %s" % (os.path.relpath(path, ROOT), mod)


def test_library_sources_never_name_the_oracle_library():
    for path in glob.glob(os.path.join(PKG, "csrc", "*")):
        with open(path, encoding="utf-8") as f:
            text = f.read()
        assert "dqgan_oracle" not in text and "oracle/" not in text, os.path.relpath(path, ROOT)
