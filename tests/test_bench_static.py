"""bench.py on the CPU: it parses, and every name a function reads is defined
(an argument, a local, a module-level name or a builtin).  bench.py only runs
where there is a GPU, so this catches a missing import on the CPU first."""
import ast
import builtins
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _names(tree):
    top = set()
    for b in tree.body:
        if isinstance(b, (ast.Import, ast.ImportFrom)):
            top |= {(a.asname or a.name).split(".")[0] for a in b.names}
        elif isinstance(b, (ast.FunctionDef, ast.ClassDef)):
            top.add(b.name)
        elif isinstance(b, (ast.Assign, ast.AnnAssign)):
            targets = b.targets if isinstance(b, ast.Assign) else [b.target]
            top |= {x.id for t in targets for x in ast.walk(t) if isinstance(x, ast.Name)}
    return top


def test_bench_functions_read_only_defined_names():
    tree = ast.parse(open(os.path.join(ROOT, "bench.py")).read())
    top = _names(tree) | set(dir(builtins))
    for fn in (n for n in tree.body if isinstance(n, ast.FunctionDef)):
        local = set()
        for n in ast.walk(fn):
            if isinstance(n, (ast.Import, ast.ImportFrom)):
                local |= {(a.asname or a.name).split(".")[0] for a in n.names}
            elif isinstance(n, ast.Name) and isinstance(n.ctx, ast.Store):
                local.add(n.id)
            elif isinstance(n, ast.arg):
                local.add(n.arg)
            elif isinstance(n, (ast.FunctionDef, ast.ClassDef)):
                local.add(n.name)
        used = {n.id for n in ast.walk(fn) if isinstance(n, ast.Name) and isinstance(n.ctx, ast.Load)}
        assert not (used - local - top), (fn.name, sorted(used - local - top))
