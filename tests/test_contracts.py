"""Host-side contracts: the product fails loudly without its HIP library, the
bench measures one GPU only, and the product never reaches the oracle."""
import ast
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2512_22147_amd")


def test_binding_raises_without_library(tmp_path):
    """With libmep.so absent the binding raises; there is no fallback path."""
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "from paper_2512_22147_amd import mep\n"
        "mep.LIB_PATH = %r\n"
        "mep._lib = None\n"
        "try:\n"
        "    mep.mep_version()\n"
        "except RuntimeError as e:\n"
        "    print('raised:', e)\n"
        "    sys.exit(0)\n"
        "sys.exit(3)\n" % (ROOT, str(tmp_path / "absent" / "libmep.so")))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "no fallback" in r.stdout


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def _imports(path):
    tree = ast.parse(open(path).read(), filename=path)
    names = set()
    for node in ast.walk(tree):
        if isinstance(node, ast.Import):
            names.update(a.name.split(".")[0] for a in node.names)
        elif isinstance(node, ast.ImportFrom) and node.module:
            names.add(node.module.split(".")[0])
    return names


def test_product_does_not_import_the_oracle():
    """Nothing under the package imports or loads anything under oracle/."""
    for dirpath, _, files in os.walk(PKG):
        for f in files:
            path = os.path.join(dirpath, f)
            if f.endswith(".py"):
                assert "oracle" not in _imports(path), path
            if f.endswith((".py", ".hip", ".hpp", ".inc", ".c", ".h")):
                text = open(path, errors="replace").read()
                assert "liboracle" not in text and "oracle.c" not in text, path
