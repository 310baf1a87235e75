"""The oracle is test infrastructure: the library and its binding never use
it, and outside the tests only the CPU-baseline leg of bench.py and the
build/smoke entry points load it. Checked statically on the sources and on
the built library's dynamic dependencies."""
import ast
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_1909_10616_amd")


def _oracle_imports(path):
    """(enclosing top-level function or None, line) of every import of the
    oracle package in a Python source."""
    found = []

    def walk(node, fn):
        for ch in ast.iter_child_nodes(node):
            name = fn
            if isinstance(ch, (ast.FunctionDef, ast.AsyncFunctionDef)) and fn is None:
                name = ch.name
            if isinstance(ch, ast.Import) and any(a.name.split(".")[0] == "oracle" for a in ch.names):
                found.append((name, ch.lineno))
            if isinstance(ch, ast.ImportFrom) and (ch.module or "").split(".")[0] == "oracle":
                found.append((name, ch.lineno))
            walk(ch, name)

    with open(path) as f:
        walk(ast.parse(f.read()), None)
    return found


def test_package_never_imports_the_oracle():
    for path in glob.glob(os.path.join(PKG, "**", "*.py"), recursive=True):
        assert _oracle_imports(path) == [], path


@pytest.mark.parametrize("path,allowed", [
    ("bench.py", {"cpu_baseline", "componentwise_error", "single_core_oracle", "oracle_side"}),
    ("__graft_entry__.py", {"build", "smoke"}),
])
def test_entry_points_load_the_oracle_only_where_allowed(path, allowed):
    found = _oracle_imports(os.path.join(ROOT, path))
    assert found and all(fn in allowed for fn, _ in found), found


def test_native_sources_share_nothing_with_the_oracle():
    for path in glob.glob(os.path.join(PKG, "csrc", "*")) + glob.glob(os.path.join(ROOT, "include", "*")):
        with open(path, errors="replace") as f:
            text = f.read()
        assert "oracle.h" not in text and "liboracle" not in text, path
    with open(os.path.join(ROOT, "oracle", "oracle.c")) as f:
        text = f.read()
    assert "gemmtune.h" not in text and "csrc/" not in text


def test_library_does_not_link_the_oracle():
    from paper_1909_10616_amd import gemmtune
    if not os.path.exists(gemmtune.LIB_PATH):
        pytest.skip("library not built")
    out = subprocess.run(["readelf", "-d", gemmtune.LIB_PATH], capture_output=True, text=True).stdout
    needed = [line for line in out.splitlines() if "(NEEDED)" in line]
    assert needed and not any("oracle" in line for line in needed), needed


def test_product_path_fails_loudly_without_the_library():
    """With the built library absent the binding raises; there is no CPU
    fallback to fall into."""
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_1909_10616_amd import gemmtune as gt\n"
            "gt.LIB_PATH = '/nonexistent/libgemmtune.so'\n"
            "try:\n"
            "    gt.Space(64, 64, 64, (2, 2, 2), 'f32', False).size()\n"
            "except gt.GemmTuneError as e:\n"
            "    print('raised', e)\n") % ROOT
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0 and out.stdout.startswith("raised") and "missing" in out.stdout, \
        out.stdout + out.stderr[-1000:]
