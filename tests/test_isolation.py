"""The oracle and the HIP path share no code: the package and its kernels never
reference the oracle, the oracle never references the package, and bench.py
reaches the oracle only from inside functions (its CPU-baseline leg), never at
import time."""
import ast
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _files(folder, exts):
    for dirpath, _, names in os.walk(os.path.join(ROOT, folder)):
        if "__pycache__" in dirpath:
            continue
        for n in names:
            if n.endswith(exts):
                yield os.path.join(dirpath, n)


def test_package_does_not_reference_the_oracle():
    for f in _files("paper_2601_20332_amd", (".py", ".hip", ".h", ".cpp")):
        text = open(f, encoding="utf-8").read()
        assert not re.search(r"\boracle\b", text), f


def test_oracle_does_not_reference_the_package():
    for f in _files("oracle", (".py", ".c", ".h")):
        text = open(f, encoding="utf-8").read()
        assert "paper_2601_20332_amd" not in text and "csrc" not in text, f
        assert "libwd" not in text, f


def test_bench_imports_the_oracle_only_inside_functions():
    tree = ast.parse(open(os.path.join(ROOT, "bench.py"), encoding="utf-8").read())
    for node in tree.body:  # module level only
        if isinstance(node, ast.Import):
            assert not any(a.name.split(".")[0] == "oracle" for a in node.names)
        if isinstance(node, ast.ImportFrom):
            assert (node.module or "").split(".")[0] != "oracle"
    inside = [n for n in ast.walk(tree) if isinstance(n, ast.ImportFrom)
              and (n.module or "").startswith("oracle")]
    assert inside, "the CPU-baseline leg is expected to import the oracle"
