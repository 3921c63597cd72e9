"""The oracle and the library share no code, and only the test side calls the oracle.

- nothing in the package (Python, C++, HIP) imports, includes or names the oracle;
- the oracle includes no library header and imports nothing of the package;
- the seeded input generator, which both sides use, imports neither;
- outside tests/, the oracle is imported only by bench.py's cpu_baseline and by
  __graft_entry__'s build (which compiles it) and smoke (which checks against it).
"""
import ast
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_14779_amd")


def _files(top, exts):
    for d, _, names in os.walk(top):
        if "__pycache__" in d or "_build" in d:
            continue
        for n in names:
            if n.endswith(exts):
                yield os.path.join(d, n)


def _imports(path):
    """(module, enclosing function or None) for every import in a Python file."""
    tree = ast.parse(open(path).read(), path)
    out = []

    def walk(node, fn):
        for child in ast.iter_child_nodes(node):
            f = child.name if isinstance(child, (ast.FunctionDef, ast.AsyncFunctionDef)) else fn
            if isinstance(child, ast.Import):
                out.extend((a.name.split(".")[0], fn) for a in child.names)
            elif isinstance(child, ast.ImportFrom) and child.module:
                out.append((child.module.split(".")[0], fn))
            walk(child, f)
    walk(tree, None)
    return out


def test_package_never_touches_the_oracle():
    for path in _files(PKG, (".py",)):
        assert "oracle" not in {m for m, _ in _imports(path)}, path
    for path in _files(os.path.join(PKG, "csrc"), (".cpp", ".hpp", ".hip", ".h")):
        src = open(path).read()
        assert not re.search(r"#\s*include\s*[<\"][^>\"]*oracle", src), path
        assert "liboracle" not in src and "oracle_" not in src, path


def test_oracle_never_touches_the_package():
    src = open(os.path.join(ROOT, "oracle", "oracle.c")).read()
    includes = re.findall(r"#\s*include\s*[<\"]([^>\"]+)[>\"]", src)
    assert not [h for h in includes if "kvpool" in h or "internal" in h or "hip" in h], includes
    mods = {m for m, _ in _imports(os.path.join(ROOT, "oracle", "__init__.py"))}
    assert "paper_2606_14779_amd" not in mods and "kvgen" not in mods, mods


def test_input_generator_imports_neither_side():
    for path in _files(os.path.join(ROOT, "kvgen"), (".py",)):
        mods = {m for m, _ in _imports(path)}
        assert "oracle" not in mods and "paper_2606_14779_amd" not in mods, (path, mods)
    src = open(os.path.join(ROOT, "kvgen", "kvgen.c")).read()
    assert not re.search(r"#\s*include[^\n]*(kvpool|oracle|internal)", src)
    assert "oracle_" not in src and "kv_pool_" not in src


def test_oracle_callers_outside_tests():
    allowed = {"bench.py": {"cpu_baseline"}, "__graft_entry__.py": {"build", "smoke"}}
    for name in os.listdir(ROOT):
        if not name.endswith(".py"):
            continue
        for mod, fn in _imports(os.path.join(ROOT, name)):
            if mod == "oracle":
                assert fn in allowed.get(name, set()), "%s imports the oracle in %s" % (name, fn)
