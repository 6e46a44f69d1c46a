"""The oracle and the product path share no code: the package (binding,
generators, build script) never imports the oracle, the oracle never imports
the package or its HIP sources, and only the allowed places (tests, smoke(),
the bench's CPU-baseline functions) reach the oracle."""
import ast
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _imports(path):
    tree = ast.parse(open(path).read(), path)
    out = []
    for node in ast.walk(tree):
        if isinstance(node, ast.Import):
            out += [(a.name, node) for a in node.names]
        elif isinstance(node, ast.ImportFrom) and node.module:
            out.append((node.module, node))
    return out


def _py(dirname):
    d = os.path.join(ROOT, dirname)
    return [os.path.join(d, f) for f in sorted(os.listdir(d)) if f.endswith(".py")]


def test_package_never_imports_the_oracle():
    for path in _py("paper_2509_17863_amd"):
        for mod, _ in _imports(path):
            assert not mod.split(".")[0] == "oracle", (path, mod)


def test_oracle_never_imports_the_package():
    for path in _py("oracle"):
        for mod, _ in _imports(path):
            assert not mod.startswith("paper_2509_17863_amd"), (path, mod)
        text = open(path).read()
        assert "csrc" not in text and "libeaas" not in text, path


def test_oracle_reached_only_from_allowed_places():
    allowed = {("bench.py", "cpu_baseline"), ("bench.py", "cpu_baseline_w8a8"),
               ("__graft_entry__.py", "smoke")}
    for name in ("bench.py", "__graft_entry__.py"):
        path = os.path.join(ROOT, name)
        tree = ast.parse(open(path).read(), path)
        for fn in [n for n in ast.walk(tree) if isinstance(n, ast.FunctionDef)]:
            for node in ast.walk(fn):
                mod = node.module if isinstance(node, ast.ImportFrom) else None
                if isinstance(node, ast.Import):
                    mod = node.names[0].name
                if mod and mod.split(".")[0] == "oracle":
                    assert (name, fn.name) in allowed, (name, fn.name)
        # and nothing at module level
        for node in tree.body:
            if isinstance(node, (ast.Import, ast.ImportFrom)):
                mod = node.module if isinstance(node, ast.ImportFrom) else node.names[0].name
                assert not (mod or "").startswith("oracle"), (name, mod)
