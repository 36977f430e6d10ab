"""The CPU oracle and the GPU path stay independent: checked from the source.

- The package (Python binding and native sources) never imports, loads or names the
  oracle; the oracle never imports the package or loads the library.
- bench.py touches the oracle only inside its CPU-baseline functions.
- The module both sides share, workloads.py, imports neither side and holds no
  attention arithmetic (no exponentials, no matrix products, no reductions).
"""
import ast
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2502_06155_amd")
ORACLE = os.path.join(ROOT, "oracle")


def _py_files(d):
    return sorted(os.path.join(d, f) for f in os.listdir(d) if f.endswith(".py"))


def _imported_modules(tree):
    """(top-level module name, enclosing function name or None) for every import."""
    out = []

    def visit(node, func):
        for child in ast.iter_child_nodes(node):
            f = child.name if isinstance(child, (ast.FunctionDef, ast.AsyncFunctionDef)) else func
            if isinstance(child, ast.Import):
                out.extend((a.name.split(".")[0], f) for a in child.names)
            elif isinstance(child, ast.ImportFrom) and child.module and child.level == 0:
                out.append((child.module.split(".")[0], f))
            elif isinstance(child, ast.ImportFrom) and child.level > 0:
                out.append(("<relative>", f))
            visit(child, f)

    visit(tree, None)
    return out


def _parse(path):
    with open(path) as fh:
        return ast.parse(fh.read(), path)


def test_package_never_imports_the_oracle():
    for path in _py_files(PKG):
        mods = {m for m, _ in _imported_modules(_parse(path))}
        assert "oracle" not in mods, path
    for sub in ("csrc",):
        for f in os.listdir(os.path.join(PKG, sub)):
            with open(os.path.join(PKG, sub, f)) as fh:
                assert "oracle" not in fh.read().lower(), f
    for f in os.listdir(os.path.join(ROOT, "include")):
        with open(os.path.join(ROOT, "include", f)) as fh:
            assert "oracle" not in fh.read().lower(), f


def test_oracle_never_imports_the_package_or_loads_native_code():
    for path in _py_files(ORACLE):
        tree = _parse(path)
        mods = {m for m, _ in _imported_modules(tree)}
        assert "paper_2502_06155_amd" not in mods, path
        assert "ctypes" not in mods and "torch" not in mods, path
        with open(path) as fh:
            src = fh.read()
        assert "libtileattn" not in src and "csrc" not in src, path


def test_bench_uses_the_oracle_only_for_its_cpu_baseline():
    uses = [(m, f) for m, f in _imported_modules(_parse(os.path.join(ROOT, "bench.py"))) if m == "oracle"]
    assert uses, "bench.py times the oracle for its cpu_baseline"
    assert all(f is not None and f.startswith("cpu_baseline") for _, f in uses), uses


def test_shared_input_module_holds_no_attention_arithmetic():
    path = os.path.join(ROOT, "workloads.py")
    tree = _parse(path)
    mods = {m for m, _ in _imported_modules(tree)}
    assert mods <= {"__future__", "dataclasses", "numpy"}, mods
    banned = {"exp", "exp2", "log", "logsumexp", "softmax", "matmul", "dot", "einsum", "tensordot",
              "sum", "max", "amax", "cumsum"}
    for node in ast.walk(tree):
        if isinstance(node, ast.Attribute):
            assert node.attr not in banned, f"workloads.py uses {node.attr}"
        if isinstance(node, ast.BinOp):
            assert not isinstance(node.op, ast.MatMult), "workloads.py multiplies matrices"
