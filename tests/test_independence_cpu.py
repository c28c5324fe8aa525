"""The oracle and the HIP path share no code: the package never imports the
oracle, the oracle never imports the package, the HIP sources include
nothing from oracle/, and the only entry points that reach the oracle are
bench.py's CPU baseline and __graft_entry__.smoke().  The tests hand both
sides the same seeded inputs from paper_2102_13272_amd/workloads.py, which
holds none of the method's arithmetic."""
import ast
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2102_13272_amd")
ORACLE = os.path.join(ROOT, "oracle")


def _py_files(d):
    for base, _, files in os.walk(d):
        for f in files:
            if f.endswith(".py"):
                yield os.path.join(base, f)


def _imports(tree):
    """(top-level module name, enclosing function name or None) per import"""
    out = []

    def visit(node, fn):
        for child in ast.iter_child_nodes(node):
            f = child.name if isinstance(child, (ast.FunctionDef, ast.AsyncFunctionDef)) else fn
            if isinstance(child, ast.Import):
                out.extend((a.name.split(".")[0], fn) for a in child.names)
            elif isinstance(child, ast.ImportFrom) and child.module and child.level == 0:
                out.append((child.module.split(".")[0], fn))
            visit(child, f)

    visit(tree, None)
    return out


def _parse(path):
    with open(path) as fh:
        return ast.parse(fh.read(), filename=path)


@pytest.mark.parametrize("path", sorted(_py_files(PKG)), ids=lambda p: os.path.relpath(p, ROOT))
def test_package_never_imports_the_oracle(path):
    assert "oracle" not in [m for m, _ in _imports(_parse(path))]


@pytest.mark.parametrize("path", sorted(_py_files(ORACLE)), ids=lambda p: os.path.relpath(p, ROOT))
def test_oracle_never_imports_the_package(path):
    assert "paper_2102_13272_amd" not in [m for m, _ in _imports(_parse(path))]


def test_hip_sources_include_nothing_from_the_oracle():
    csrc = os.path.join(PKG, "csrc")
    for f in os.listdir(csrc):
        with open(os.path.join(csrc, f)) as fh:
            for inc in re.findall(r'#include\s+[<"]([^>"]+)[>"]', fh.read()):
                assert "oracle" not in inc, (f, inc)


@pytest.mark.parametrize("entry,allowed", [("bench.py", {"cpu_baseline"}),
                                           ("__graft_entry__.py", {"smoke"})])
def test_entry_points_reach_the_oracle_only_from_their_cpu_checks(entry, allowed):
    uses = [fn for m, fn in _imports(_parse(os.path.join(ROOT, entry))) if m == "oracle"]
    assert uses and set(uses) <= allowed, uses
