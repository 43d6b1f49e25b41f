"""The product and the oracle stay apart (no GPU): read from the sources, the library and its
binding never import, include or load anything under ``oracle/``; the oracle takes nothing from
the package but the seeded input generators; ``bench.py`` and ``__graft_entry__`` reach the oracle
only inside the CPU-baseline leg and ``smoke()``; and the binding raises when the library is
missing instead of falling back."""

import ast
import glob
import os
import re

import pytest

from paper_2010_14109_amd import ooc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2010_14109_amd")


def imported_modules(tree):
    """(module name, enclosing top-level function or None) for every import in ``tree``."""
    out = []

    def visit(node, fn):
        for child in ast.iter_child_nodes(node):
            f = fn
            if fn is None and isinstance(child, (ast.FunctionDef, ast.AsyncFunctionDef)):
                f = child.name
            if isinstance(child, ast.Import):
                out.extend((a.name, f) for a in child.names)
            elif isinstance(child, ast.ImportFrom):
                base = "." * child.level + (child.module or "")
                out.append((base, f))
                out.extend((base + a.name if base.endswith(".") else f"{base}.{a.name}", f)
                           for a in child.names)
            visit(child, f)

    visit(tree, None)
    return out


def parse(path):
    return ast.parse(open(path).read(), path)


def is_oracle(mod):
    mod = mod.lstrip(".")           # a relative import names the same top-level package
    return mod == "oracle" or mod.startswith("oracle.")


def test_package_never_imports_the_oracle():
    files = glob.glob(os.path.join(PKG, "**", "*.py"), recursive=True)
    assert len(files) >= 5
    for f in files:
        for mod, _ in imported_modules(parse(f)):
            assert not is_oracle(mod), (f, mod)


def test_native_sources_never_reach_the_oracle():
    srcs = [f for ext in ("cpp", "hip", "h") for f in
            glob.glob(os.path.join(PKG, "csrc", f"*.{ext}")) + glob.glob(os.path.join(ROOT, "include", f"*.{ext}"))]
    assert any(f.endswith("gemm.hip") for f in srcs) and any(f.endswith("ooc.h") for f in srcs)
    for f in srcs:
        text = open(f).read()
        for inc in re.findall(r'#\s*include\s*[<"]([^>"]+)[>"]', text):
            assert "oracle" not in inc, (f, inc)
        assert "oracle/" not in text and "oracle." not in text, f


def test_build_compiles_no_oracle_source_into_the_library():
    text = open(os.path.join(PKG, "build.py")).read()
    assert "oracle" not in text


def test_oracle_takes_only_the_seeded_generators_from_the_package():
    for f in glob.glob(os.path.join(ROOT, "oracle", "*.py")):
        for mod, _ in imported_modules(parse(f)):
            if mod.startswith("paper_2010_14109_amd"):
                assert mod in ("paper_2010_14109_amd", "paper_2010_14109_amd.synth"), (f, mod)


def test_synth_holds_no_method_arithmetic():
    """The one module both sides use draws inputs: it imports NumPy and a thread pool, nothing of
    either side's compute."""
    for mod, _ in imported_modules(parse(os.path.join(PKG, "synth.py"))):
        assert mod.split(".")[0] in ("numpy", "math", "__future__", "concurrent"), mod


@pytest.mark.parametrize("path,allowed", [
    ("bench.py", {"oracle_schedule_ms", "cpu_baseline"}),
    ("__graft_entry__.py", {"smoke"}),
])
def test_entry_points_reach_the_oracle_only_in_their_baseline_legs(path, allowed):
    uses = [(mod, fn) for mod, fn in imported_modules(parse(os.path.join(ROOT, path))) if is_oracle(mod)]
    assert uses, path
    for mod, fn in uses:
        assert fn in allowed, (path, mod, fn)


def test_bench_calls_the_oracle_only_with_the_cpu_baseline_on():
    """The schedule timing and the oracle step run only under ``if not args.no_cpu_baseline``."""
    tree = parse(os.path.join(ROOT, "bench.py"))
    guarded = set()
    for node in ast.walk(tree):
        if isinstance(node, ast.If) and "no_cpu_baseline" in ast.unparse(node.test):
            for sub in ast.walk(node):
                if isinstance(sub, ast.Call) and isinstance(sub.func, ast.Name):
                    guarded.add(id(sub))
    calls = [n for n in ast.walk(tree) if isinstance(n, ast.Call) and isinstance(n.func, ast.Name)
             and n.func.id in ("oracle_schedule_ms", "cpu_baseline")]
    assert calls
    for c in calls:
        assert id(c) in guarded, ast.unparse(c)


def test_binding_raises_without_the_library(tmp_path, monkeypatch):
    monkeypatch.setattr(ooc, "_lib", None)         # as in a process that has not loaded it yet
    with pytest.raises(RuntimeError, match="no fallback"):
        ooc.load(str(tmp_path / "libooc.so"))
