"""The product path has no fallback and never touches the oracle (CPU only).

* Nothing under the package imports ``oracle``; outside ``tests/`` only the benchmark's
  ``cpu_baseline`` leg and the smoke entry point do, inside those functions.
* A missing library raises instead of running anything else, both when loaded directly and
  when a sampler is created.
"""
import ast
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_36522_amd")


def _oracle_imports(path):
    """(function name or None, line) of every import of the oracle package in a Python file."""
    tree = ast.parse(open(path).read())
    found = []

    def visit(node, func):
        for child in ast.iter_child_nodes(node):
            f = child.name if isinstance(child, (ast.FunctionDef, ast.AsyncFunctionDef)) else func
            if isinstance(child, ast.Import) and any(a.name.split(".")[0] == "oracle" for a in child.names):
                found.append((func, child.lineno))
            if isinstance(child, ast.ImportFrom) and (child.module or "").split(".")[0] == "oracle":
                found.append((func, child.lineno))
            visit(child, f)

    visit(tree, None)
    return found


def test_package_never_imports_the_oracle():
    for dirpath, _, files in os.walk(PKG):
        for f in files:
            p = os.path.join(dirpath, f)
            if f.endswith(".py"):
                assert not _oracle_imports(p), p
            if f.endswith((".hip", ".cpp", ".h")):
                assert "oracle" not in open(p).read().lower(), p


def test_oracle_only_in_the_cpu_baseline_and_the_smoke_check():
    assert {fn for fn, _ in _oracle_imports(os.path.join(ROOT, "bench.py"))} == {"cpu_baseline"}
    assert {fn for fn, _ in _oracle_imports(os.path.join(ROOT, "__graft_entry__.py"))} == {"smoke"}


def test_missing_library_raises():
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "from paper_2609_36522_amd import binding as B\n"
        "try:\n"
        "    B.load_library('/nonexistent/libparaanya.so')\n"
        "except RuntimeError as e:\n"
        "    assert 'missing' in str(e)\n"
        "else:\n"
        "    raise SystemExit('loaded a missing library')\n"
        "B.load_library.__defaults__ = ('/nonexistent/libparaanya.so',)\n"
        "try:\n"
        "    B.Sampler((1, 4, 8, 8), 10, 4, 0.05, 1e-3, 'linear', c=[1.0] * 10)\n"
        "except RuntimeError as e:\n"
        "    assert 'missing' in str(e)\n"
        "else:\n"
        "    raise SystemExit('created a sampler without the library')\n"
        "print('ok')\n" % ROOT)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
