"""The C ABI without a GPU: libgp.so loads and exports every entry point that
include/gp.h declares, the Python binding's constants match the header, and
argument checks that need no device reject bad calls.  (No kernel runs.)"""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gp.h")


def header_text():
    with open(HEADER) as f:
        return f.read()


def declared_functions():
    return set(re.findall(r"^(?:gp_status|const char\s*\*)\s*(gp_\w+)\s*\(", header_text(), re.M))


def enum_names(prefix, terminator):
    h = header_text()
    blk = h[h.index(prefix):h.index(terminator)]
    return re.findall(r"\b(" + prefix.split("_")[0] + r"_[A-Z0-9_]+)\b", blk)


@pytest.fixture(scope="module")
def lib():
    from paper_1811_06965_amd import build, gp
    if not os.path.exists(gp.LIB_PATH):
        build.build()
    return gp.load()


def test_header_declares_the_binding_exports():
    from paper_1811_06965_amd import gp
    assert declared_functions() == set(gp.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    from paper_1811_06965_amd import gp
    out = subprocess.run(["nm", "-D", "--defined-only", gp.LIB_PATH], capture_output=True, text=True, check=True)
    exported = set(re.findall(r"\bT (gp_\w+)$", out.stdout, re.M))
    missing = declared_functions() - exported
    assert not missing, missing
    for name in declared_functions():
        assert hasattr(lib, name)


def test_library_has_no_unresolved_internal_symbols(lib):
    from paper_1811_06965_amd import gp
    out = subprocess.run(["nm", "-DC", "--undefined-only", gp.LIB_PATH], capture_output=True, text=True, check=True)
    assert "gp::" not in out.stdout


def test_status_and_enum_values_match_header():
    from paper_1811_06965_amd import gp
    h = header_text()
    for name, val in [("GP_OK", gp.GP_OK), ("GP_ERR_INVALID_ARG", gp.GP_ERR_INVALID_ARG),
                      ("GP_ERR_STATE", gp.GP_ERR_STATE), ("GP_ERR_OOM", gp.GP_ERR_OOM), ("GP_ERR_HIP", gp.GP_ERR_HIP),
                      ("GP_ERR_NONFINITE", gp.GP_ERR_NONFINITE), ("GP_ERR_UNSUPPORTED", gp.GP_ERR_UNSUPPORTED),
                      ("GP_F32", gp.GP_F32), ("GP_BF16", gp.GP_BF16)]:
        m = re.search(name + r"\s*=\s*(\d+)", h)
        assert m and int(m.group(1)) == val, name
    # parameter ids: header order is the binding's order
    blk = h[h.index("GP_P_LN1_G = 0"):h.index("GP_P_COUNT")]
    ids = re.findall(r"GP_P_(\w+)", blk)
    assert [x.lower() for x in ids] == gp.PARAM_IDS
    # kernel roles
    blk = h[h.index("GP_K_NONE = 0"):h.index("} gp_kernel_role")]
    roles = re.findall(r"GP_K_(\w+)", blk)
    assert roles[-1] == "COUNT" and len(roles) - 1 == len(gp.KERNEL_ROLES)
    assert [r.lower().replace("_fwd", ".fwd").replace("_dx", ".dx").replace("_dw", ".dw").replace("_bwd", ".bwd")
            for r in roles[:-1]] == gp.KERNEL_ROLES


def test_config_struct_matches_header():
    from paper_1811_06965_amd import gp
    h = header_text()
    blk = h[h.index("typedef struct {", h.index("gp_loss")):h.index("} gp_config;")]
    fields = re.findall(r"^\s*(?:int|float)\s+(\w+);", blk, re.M)
    assert fields == [f for f, _ in gp.gp_config._fields_]


def test_create_rejects_bad_dimensions_without_a_device(lib):
    h = ctypes.c_void_p()
    assert lib.gp_partition_create(0, 1024, 8192, 16, ctypes.byref(h)) == 1
    assert b"positive" in lib.gp_last_error()
    assert lib.gp_partition_create(2, 1000, 8192, 16, ctypes.byref(h)) == 1
    assert lib.gp_partition_create(2, 64, 128, 1, None) == 1


def test_calls_on_a_null_partition_are_rejected(lib):
    assert lib.gp_forward_microbatch(None, 0, None, None, None, None) == 1
    assert lib.gp_backward_microbatch_remat(None, 0, None, None, None, None) == 1
    assert lib.gp_accumulate_and_step(None, ctypes.c_float(0.1), None, None) == 1
    assert lib.gp_timer_select(None, 0) == 1
    assert lib.gp_timer_sample(None, 1) == 1
    assert lib.gp_partition_destroy(None) == 0
    assert lib.gp_stream_create(None) == 1
    assert lib.gp_stream_destroy(None) == 1


def test_host_logic_program():
    """Validation, parameter plan and state machine of sched.hpp, compiled for
    the host with g++ (address and undefined-behaviour sanitizers on)."""
    import shutil
    import tempfile
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "sched_test")
        src = os.path.join(ROOT, "tests", "host", "sched_test.cpp")
        subprocess.run([gxx, "-std=c++17", "-O1", "-Wall", "-Werror", "-fsanitize=address,undefined",
                        "-I" + os.path.join(ROOT, "include"), src, "-o", exe], check=True)
        r = subprocess.run([exe], capture_output=True, text=True)
        assert r.returncode == 0, r.stdout
        assert "0 failures" in r.stdout
