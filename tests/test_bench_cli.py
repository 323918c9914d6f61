"""bench.py's command-line modes: every mode function main() dispatches to exists (host only)."""
import ast
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_every_dispatched_mode_is_defined():
    tree = ast.parse(open(os.path.join(ROOT, "bench.py")).read())
    defined = {n.name for n in tree.body if isinstance(n, ast.FunctionDef)}
    main = next(n for n in tree.body if isinstance(n, ast.FunctionDef) and n.name == "main")
    called = {c.func.id for c in ast.walk(main) if isinstance(c, ast.Call) and isinstance(c.func, ast.Name)}
    modes = {name for name in called if name.endswith("_main")}
    assert modes, "main() dispatches to no mode function"
    assert modes <= defined, f"main() calls undefined mode functions: {sorted(modes - defined)}"
