"""The host C++ of the library (the planners and the semantic map) built with
AddressSanitizer and UndefinedBehaviorSanitizer (host code only, g++),
running their test files in a child process: the C ABI tests (bit-exact
against the oracle planner on the figures, the workloads and random forests;
argument validation), the decoded device tables and the semantic map.  Any
out-of-bounds access, use after free, signed overflow or other undefined
behaviour aborts the child.

The sanitized library links the host sources, compiled here, with the HIP
objects the regular build left in _build (their device code is not
instrumented and never runs here).
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2608_28158_amd")


def _runtime(name):
    out = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True)
    path = out.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


HOST_SOURCES = ("plan.cpp", "semantic.cpp", "mbplan.cpp", "kda_plan.cpp")
HIP_OBJECTS = ("la.hip.o", "logp.hip.o", "conv.hip.o", "attn.hip.o", "kda.hip.o")


def test_planner_under_asan_and_ubsan(tmp_path):
    hip_objs = [os.path.join(PKG, "_build", o) for o in HIP_OBJECTS]
    if shutil.which("g++") is None or not all(os.path.exists(o) for o in hip_objs):
        pytest.skip("needs g++ and the regular build's HIP objects")
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("sanitizer runtimes not found")
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    objs = []
    for src in HOST_SOURCES:
        obj = str(tmp_path / (src + ".o"))
        subprocess.run(["g++", "-O1", "-g", "-fno-omit-frame-pointer", "-std=c++17", "-fPIC"] +
                       san + ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc"),
                              "-c", os.path.join(PKG, "csrc", src), "-o", obj], check=True)
        objs.append(obj)
    lib = str(tmp_path / "libharts_san.so")
    subprocess.run(["g++", "-shared"] + san + objs + hip_objs +
                   ["-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", lib],
                   check=True)
    env = dict(os.environ, HARTS_LIB=lib, LD_PRELOAD=f"{asan}:{ubsan}",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    code = ("import sys, pytest\n"
            "from paper_2608_28158_amd import _lib\n"
            f"assert _lib.LIB_PATH == {lib!r}\n"
            "sys.exit(pytest.main(['-q', '-x', '-p', 'no:cacheprovider', "
            "'tests/test_abi_plan.py', 'tests/test_plan_tables.py', "
            "'tests/test_semantic_map.py', 'tests/test_abi_mbplan.py']))\n")
    res = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True,
                         text=True, timeout=600)
    out = res.stdout + res.stderr
    print(out[-3000:])
    assert res.returncode == 0, out[-3000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out
    assert " passed" in out
