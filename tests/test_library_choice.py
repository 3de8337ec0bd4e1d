"""Which library a test session loads (host logic; runs without a GPU).

Importing every test module and tool module must leave the binding on the
product library: a module that switched the binding to the timing-trace
build at import time would make the GPU suite check that build instead.
"""
import glob
import importlib
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_importing_every_module_keeps_the_product_library():
    mods = sorted(os.path.splitext(os.path.basename(p))[0] for p in glob.glob(os.path.join(ROOT, "tests", "test_*.py")))
    code = "\n".join([
        "import os, sys, importlib",
        f"sys.path.insert(0, {ROOT!r}); sys.path.insert(0, {os.path.join(ROOT, 'tests')!r})",
        "from paper_2607_07862_amd import binding, tracesum, profsum  # tools as well",
        *[f"importlib.import_module({m!r})" for m in mods],
        "assert os.environ.get('MLP2_TRACE') is None, 'a module set MLP2_TRACE'",
        "assert binding.loaded_path() is None, binding.loaded_path()",
        "lib_default = binding.LIB_PATH",
        "print('OK', lib_default)",
    ])
    env = {k: v for k, v in os.environ.items() if k != "MLP2_TRACE"}
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().endswith("libmlp2.so")


def test_load_defaults_to_the_product_library_and_refuses_a_second_one():
    code = "\n".join([
        "import os, sys",
        f"sys.path.insert(0, {ROOT!r})",
        "from paper_2607_07862_amd import binding as B",
        "lib = B.load()",
        "assert os.path.abspath(B.loaded_path()) == os.path.abspath(B.LIB_PATH), B.loaded_path()",
        "assert B.load() is lib",
        "try:\n    B.load(B.TRACE_LIB_PATH)\nexcept RuntimeError:\n    print('refused')\nelse:\n    raise SystemExit('second library accepted')",
    ])
    if not os.path.exists(os.path.join(ROOT, "paper_2607_07862_amd", "libmlp2.so")):
        import pytest

        pytest.skip("library not built")
    env = {k: v for k, v in os.environ.items() if k != "MLP2_TRACE"}
    env["MLP2_TRACE"] = "1"  # ignored: the binding no longer reads it
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "refused" in r.stdout
