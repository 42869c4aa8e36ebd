"""The oracle and the product share no code: neither imports the other, and neither imports
anything from the scratch area. Only the seeded input generator (``synth``) is shared, and it
holds none of the method's arithmetic."""

import ast
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _imports(path):
    tree = ast.parse(open(path).read(), path)
    names = set()
    for node in ast.walk(tree):
        if isinstance(node, ast.Import):
            names.update(a.name.split(".")[0] for a in node.names)
        elif isinstance(node, ast.ImportFrom):
            if node.level == 0 and node.module:
                names.add(node.module.split(".")[0])
    return names


def _py_files(sub):
    base = os.path.join(ROOT, sub)
    for dirpath, _, files in os.walk(base):
        for f in files:
            if f.endswith(".py"):
                yield os.path.join(dirpath, f)


def test_product_does_not_import_the_oracle():
    for path in _py_files("paper_2609_32415_amd"):
        bad = _imports(path) & {"oracle", "_work", "tests"}
        assert not bad, f"{path} imports {bad}"


def test_oracle_does_not_import_the_product():
    for path in _py_files("oracle"):
        bad = _imports(path) & {"paper_2609_32415_amd", "_work", "tests", "torch"}
        assert not bad, f"{path} imports {bad}"


def test_bench_uses_the_oracle_only_for_the_cpu_baseline():
    tree = ast.parse(open(os.path.join(ROOT, "bench.py")).read())
    users = set()
    for fn in (n for n in ast.walk(tree) if isinstance(n, ast.FunctionDef)):
        for node in ast.walk(fn):
            if isinstance(node, ast.ImportFrom) and node.module and node.module.split(".")[0] == "oracle":
                users.add(fn.name)
    assert users == {"cpu_baseline"}
