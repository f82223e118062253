"""The C ABI from C: moe_offload.h compiles as strict C99 and a C program
linked against the library gets the documented results from the calls that
need no GPU."""
import os
import subprocess

import pytest

from paper_2511_05814_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_c99_client_links_and_runs(tmp_path):
    lib = build.OUT
    if not os.path.exists(lib):
        pytest.fail(f"library not built: {lib}")
    exe = tmp_path / "abi_host_calls"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c", "abi_host_calls.c"),
           "-o", str(exe), lib, "-Wl,-rpath," + os.path.dirname(lib)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.strip().endswith("ok")


def test_header_is_valid_cxx():
    subprocess.run(["g++", "-std=c++17", "-Wall", "-Wextra", "-Werror", "-fsyntax-only", "-x", "c++",
                    "-I", os.path.join(ROOT, "include"), "-"],
                   input='#include "moe_offload.h"\nint main() { return MOE_OK; }\n',
                   check=True, capture_output=True, text=True)
