"""Host-side checks of the C ABI (no GPU needed).

The library must load and export every function ``include/mlp2.h`` declares,
and argument errors that are detected before any device call must come back
as the documented codes with no side effects.
"""
import ctypes
import os
import re

import pytest

from paper_2607_07862_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mlp2.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2607_07862_amd import build

        build.build()
    return B.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mlp2_[a-z_]+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(B.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
    # and they are real dynamic symbols of the shared object
    out = os.popen(f"nm -D --defined-only {B.LIB_PATH}").read()
    for name in declared_functions():
        assert re.search(rf"\bT {name}$", out, re.M), name


def test_strerror_is_total(lib):
    for code in list(range(-10, 3)) + [12345, -99999]:
        s = lib.mlp2_strerror(code)
        assert s is not None and len(s) > 0
    assert lib.mlp2_strerror(B.ERR_TIMEOUT) == b"device flag wait timed out"


@pytest.mark.parametrize(
    "args,code",
    [
        ((0, 512, 2048, 0, 0), B.ERR_INVALID_ARG),
        ((64, 0, 2048, 0, 0), B.ERR_INVALID_ARG),
        ((64, 512, -1, 0, 0), B.ERR_INVALID_ARG),
        ((64, 512, 2048, 3, 0), B.ERR_INVALID_ARG),
        ((64, 512, 2048, -1, 0), B.ERR_INVALID_ARG),
        ((64, 512, 2048, 0, 1), B.ERR_INVALID_ARG),
        ((64, 500, 2048, 0, 0), B.ERR_UNSUPPORTED),
        ((64, 512, 2000, 1, 0), B.ERR_UNSUPPORTED),
        ((1 << 21, 512, 2048, 0, 0), B.ERR_UNSUPPORTED),
    ],
)
def test_plan_rejects_bad_arguments_before_touching_a_device(lib, args, code):
    assert not lib.mlp2_plan(*args)
    assert lib.mlp2_last_error() == code


def test_plan_ex_rejects_bad_tuning(lib):
    t = B.Tuning()
    t.order = 9
    assert not lib.mlp2_plan_ex(64, 512, 2048, 0, 0, ctypes.byref(t))
    assert lib.mlp2_last_error() == B.ERR_UNSUPPORTED
    t = B.Tuning()
    t.bm = -32
    assert not lib.mlp2_plan_ex(64, 512, 2048, 0, 0, ctypes.byref(t))
    assert lib.mlp2_last_error() == B.ERR_UNSUPPORTED


def test_null_plan_calls_fail_cleanly(lib):
    assert lib.mlp2_run(None, 16, 16, 16, 16, None, 0) == B.ERR_INVALID_ARG
    assert lib.mlp2_check(None) == B.ERR_INVALID_ARG
    assert lib.mlp2_plan_info(None, None) == B.ERR_INVALID_ARG
    assert lib.mlp2_set_option(None, B.OPT_GRID, 4) == B.ERR_INVALID_ARG
    assert not lib.mlp2_intermediate(None)
    lib.mlp2_destroy(None)  # NULL-safe
    assert lib.mlp2_last_error() == B.ERR_INVALID_ARG


def test_last_error_is_per_thread(lib):
    import threading

    lib.mlp2_plan(0, 1, 1, 0, 0)
    seen = []

    def other():
        seen.append(lib.mlp2_last_error())

    th = threading.Thread(target=other)
    th.start()
    th.join()
    assert seen == [B.OK]
    assert lib.mlp2_last_error() == B.ERR_INVALID_ARG


def test_binding_constants_match_the_header():
    """Every enum constant the header defines has the same value in the binding
    (MLP2_MODE_WORKQUEUE -> binding.MODE_WORKQUEUE, MLP2_OK -> binding.OK, ...)."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    consts = {}
    for body in re.findall(r"enum\s+\w+\s*\{(.*?)\}", text, flags=re.S):
        for name, value in re.findall(r"\b(MLP2_[A-Z0-9_]+)\s*=\s*(-?\d+)", body):
            consts[name] = int(value)
    assert "MLP2_MODE_WORKQUEUE" in consts and len(consts) >= 20
    for name, value in consts.items():
        attr = name[len("MLP2_"):]
        assert getattr(B, attr) == value, name
