"""The CPU oracle and the library's host code under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only, no GPU call).

- oracle: tests/sanitize/oracle_drive.c calls every exported routine of
  oracle/huge_oracle.c on small inputs and on argument errors; built with gcc.
- host code: tests/sanitize/host_drive.cpp calls the entry points that run on
  the host alone (workspace planning, the alias-table builder, status
  strings, argument checks) with api.hip's host side and alias.cpp
  instrumented -- the GPU code of api.hip is compiled without a sanitizer --
  and linked with the library's kernel objects.
A sanitizer finding aborts the driver (no recovery), so each test checks the
exit status, the driver's own expectations and the absence of a report.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2307_14490_amd", "csrc")
INC = os.path.join(ROOT, "include")
ROCM_BIN = "/opt/rocm/bin"
CLANGXX = "/opt/rocm/lib/llvm/bin/clang++"

ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


def _check_clean(r, banner):
    assert r.returncode == 0, f"exit {r.returncode}\n{r.stdout}\n{r.stderr}"
    assert banner in r.stdout
    for marker in ("ERROR: AddressSanitizer", "runtime error:", "ERROR: LeakSanitizer"):
        assert marker not in r.stderr, r.stderr


def test_oracle_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_drive")
    _run(["gcc", "-std=gnu99", "-g", "-O1", "-fno-omit-frame-pointer", "-ffp-contract=off",
          "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          os.path.join(HERE, "sanitize", "oracle_drive.c"),
          os.path.join(ROOT, "oracle", "huge_oracle.c"), "-lm", "-o", exe])
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=120)
    _check_clean(r, "oracle sanitizer drive: ok")


def _kernel_objects():
    """The library's kernel objects, rebuilt when a source is newer."""
    from paper_2307_14490_amd import build as b
    objs = [os.path.join(b.BUILD, s + ".o") for s in b.SOURCES
            if s.endswith(".hip") and s != "api.hip"]
    srcs = [os.path.join(CSRC, f) for f in os.listdir(CSRC)]
    newest = max(os.path.getmtime(p) for p in srcs)
    if not all(os.path.exists(o) and os.path.getmtime(o) >= newest for o in objs):
        b.build()
    return objs


def test_host_code_under_asan_and_ubsan(tmp_path):
    hipcc = os.path.join(ROCM_BIN, "hipcc")
    assert os.path.exists(hipcc) and os.path.exists(CLANGXX), "the ROCm toolchain is missing"
    objs = _kernel_objects()
    api = str(tmp_path / "api.o")
    # host side instrumented; the device side of api.hip is built as usual
    _run([hipcc, "-c", "-g", "-O1", "-std=c++17", "--offload-arch=gfx950",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
          "-Xarch_host", "-fno-sanitize-recover=all", "-I", INC,
          "-x", "hip", os.path.join(CSRC, "api.hip"), "-o", api])
    alias = str(tmp_path / "alias.o")
    drive = str(tmp_path / "drive.o")
    for src, obj in ((os.path.join(CSRC, "alias.cpp"), alias),
                     (os.path.join(HERE, "sanitize", "host_drive.cpp"), drive)):
        _run([CLANGXX, "-c", "-g", "-O1", "-std=c++17", "-fsanitize=address,undefined",
              "-fno-sanitize-recover=all", "-I", INC, src, "-o", obj])
    exe = str(tmp_path / "host_drive")
    _run([hipcc, "-fsanitize=address", "-fsanitize=undefined", "-fno-gpu-sanitize",
          drive, api, alias, *objs, "-o", exe])
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=120)
    _check_clean(r, "host sanitizer drive: ok")
