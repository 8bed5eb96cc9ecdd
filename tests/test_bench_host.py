"""Host checks of bench.py (no GPU): every module-level name its functions
call is defined, the multi-GPU request exits with a message before touching
the device."""
import ast
import builtins
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def test_every_called_module_name_is_defined():
    tree = ast.parse(open(BENCH).read())
    defined = set(dir(builtins))
    for node in tree.body:
        if isinstance(node, (ast.FunctionDef, ast.ClassDef)):
            defined.add(node.name)
        elif isinstance(node, (ast.Import, ast.ImportFrom)):
            defined.update((a.asname or a.name).split(".")[0] for a in node.names)
        elif isinstance(node, ast.Assign):
            defined.update(t.id for t in node.targets if isinstance(t, ast.Name))
    missing = set()
    # each top-level function with everything nested in it is one scope
    for fn in [n for n in tree.body if isinstance(n, ast.FunctionDef)]:
        local = set()
        for n in ast.walk(fn):
            if isinstance(n, ast.Name) and isinstance(n.ctx, ast.Store):
                local.add(n.id)
            elif isinstance(n, (ast.FunctionDef, ast.Lambda)):
                a = n.args
                local.update(x.arg for x in a.args + a.kwonlyargs)
                if isinstance(n, ast.FunctionDef):
                    local.add(n.name)
            elif isinstance(n, (ast.Import, ast.ImportFrom)):
                local.update((x.asname or x.name).split(".")[0] for x in n.names)
        for n in ast.walk(fn):
            if isinstance(n, ast.Call) and isinstance(n.func, ast.Name):
                if n.func.id not in local and n.func.id not in defined:
                    missing.add(n.func.id)
    assert not missing, sorted(missing)


def test_multi_gpu_request_exits_with_a_message():
    r = subprocess.run([sys.executable, BENCH, "--gpus", "2"], capture_output=True, text=True,
                       cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]
