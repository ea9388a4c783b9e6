"""The oracle and the HIP path share no code, and the product path never
reaches the oracle (CPU only, static checks of the sources).

- Nothing in the package (Python binding, build script, seeded inputs, C++
  and HIP sources, the C header) imports, loads or names the oracle module.
- The oracle imports nothing of the package: it takes plain arrays.
- In ``bench.py`` the oracle is imported only inside ``cpu_baseline``, the
  leg that times it beside the GPU; the timed decision steps cannot reach it.
- ``__graft_entry__.smoke`` reaches the oracle only through the test harness
  that checks the GPU against it.
- The binding refuses to run without the built library (no fallback).
"""
import ast
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_27193_amd")
ORACLE = os.path.join(ROOT, "oracle")


def _sources(top, exts):
    for d, _, files in os.walk(top):
        if "__pycache__" in d:
            continue
        for f in files:
            if f.endswith(exts):
                yield os.path.join(d, f)


def _imports(tree):
    """(module name, enclosing function names) of every import statement."""
    out = []

    def visit(node, funcs):
        for child in ast.iter_child_nodes(node):
            if isinstance(child, (ast.FunctionDef, ast.AsyncFunctionDef)):
                visit(child, funcs + [child.name])
            elif isinstance(child, ast.Import):
                out.extend((a.name, tuple(funcs)) for a in child.names)
                visit(child, funcs)
            elif isinstance(child, ast.ImportFrom):
                out.append((child.module or "", tuple(funcs)))
                visit(child, funcs)
            else:
                visit(child, funcs)

    visit(tree, [])
    return out


def test_package_never_names_the_oracle():
    # "oracle" may appear in prose (a docstring saying what may use the
    # inputs); what must not appear is an import, a load or a path into it.
    pat = re.compile(r"(^|[^A-Za-z_])(import\s+oracle|from\s+oracle|oracle[./\\]|layercheck_oracle)")
    bad = []
    for p in _sources(PKG, (".py", ".cpp", ".hip", ".h")):
        text = open(p, encoding="utf-8").read()
        if pat.search(text):
            bad.append(os.path.relpath(p, ROOT))
    for p in _sources(os.path.join(ROOT, "include"), (".h",)):
        if "oracle" in open(p, encoding="utf-8").read():
            bad.append(os.path.relpath(p, ROOT))
    assert not bad, bad


def test_package_python_imports_no_oracle_or_tests():
    for p in _sources(PKG, (".py",)):
        for mod, _ in _imports(ast.parse(open(p, encoding="utf-8").read())):
            assert not mod.startswith(("oracle", "tests")), (p, mod)


def test_oracle_imports_nothing_of_the_package():
    for p in _sources(ORACLE, (".py",)):
        for mod, _ in _imports(ast.parse(open(p, encoding="utf-8").read())):
            assert not mod.startswith(("paper_2609_27193_amd", "tests", "bench")), (p, mod)
    # the oracle's C part, if any, includes no header of the library
    for p in _sources(ORACLE, (".c", ".h", ".cpp")):
        text = open(p, encoding="utf-8").read()
        assert "layercheck.h" not in text and "lc_" not in text, p


def test_bench_imports_the_oracle_only_in_its_cpu_leg():
    tree = ast.parse(open(os.path.join(ROOT, "bench.py"), encoding="utf-8").read())
    sites = [(m, f) for m, f in _imports(tree) if m.startswith("oracle") or m.startswith("tests")]
    assert sites, "the CPU baseline leg times the oracle"
    for mod, funcs in sites:
        assert mod.startswith("oracle") and funcs == ("cpu_baseline",), (mod, funcs)


def test_smoke_reaches_the_oracle_only_through_the_test_harness():
    tree = ast.parse(open(os.path.join(ROOT, "__graft_entry__.py"), encoding="utf-8").read())
    for mod, funcs in _imports(tree):
        if mod.startswith(("oracle", "tests")):
            assert funcs == ("smoke",) and mod == "tests.gpu_harness", (mod, funcs)
    for mod, funcs in _imports(tree):
        if funcs == ("build",):
            assert not mod.startswith(("oracle", "tests")), mod


def test_binding_refuses_a_missing_library(tmp_path):
    from paper_2609_27193_amd import layercheck as LC

    saved = LC._LIB
    try:
        LC._LIB = None
        with pytest.raises(RuntimeError, match="not built"):
            LC.load_library(str(tmp_path / "no_such_liblayercheck.so"))
    finally:
        LC._LIB = saved
