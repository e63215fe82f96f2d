"""The oracle's C loops and the library's C-ABI layer built with the address
and undefined-behaviour sanitizers on the host, and run on the CPU.

* oracle: tests/sanitize/oracle_sanitize.c drives oracle/lora_loops.c on
  exact-size arrays (gcc, -fsanitize=address,undefined);
* C ABI: tests/sanitize/abi_sanitize.cpp calls every entry point with invalid
  arguments (each must be rejected, with its status, before any HIP call),
  sweeps the host-only launch plans and workspace sizes, and calls
  lora_status_string from C with codes past the enumerators.  lora_abi.cpp is
  compiled with host-only sanitizers (-fno-gpu-sanitize) and linked with the
  library's device objects from build().

No GPU is used: every call either fails validation or is host-only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
PKG = os.path.join(ROOT, "paper_2403_11366_amd")
HOST_SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=300, **kw)
    assert res.returncode == 0, f"{' '.join(cmd)}\n{res.stdout}\n{res.stderr}"
    return res


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_oracle_loops_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    _run(["gcc"] + HOST_SAN + ["-fopenmp", os.path.join(SAN, "oracle_sanitize.c"),
                               os.path.join(ROOT, "oracle", "lora_loops.c"), "-lm", "-o", exe])
    res = _run([exe], env=dict(os.environ, UBSAN_OPTIONS="print_stacktrace=1"))
    assert "oracle sanitizer driver: ok" in res.stdout


def test_abi_layer_under_sanitizers(tmp_path):
    from paper_2403_11366_amd import build
    objs = [os.path.join(build.BUILD, s + ".o") for s in build.SOURCES if s.endswith(".hip")]
    if not all(os.path.exists(o) for o in objs):
        build.build()
    hipcc = build.hipcc()
    host = HOST_SAN + ["-fno-gpu-sanitize"]   # instrument the host code only
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc")]
    abi_o, drv_o, st_o = (str(tmp_path / x) for x in ("abi.o", "drv.o", "status.o"))
    _run([hipcc] + host + ["-std=c++17"] + inc + ["-c", os.path.join(PKG, "csrc", "lora_abi.cpp"), "-o", abi_o])
    _run([hipcc] + host + ["-std=c++17"] + inc + ["-c", os.path.join(SAN, "abi_sanitize.cpp"), "-o", drv_o])
    _run(["gcc"] + HOST_SAN + inc + ["-c", os.path.join(SAN, "status_codes.c"), "-o", st_o])
    exe = str(tmp_path / "abi_san")
    _run([hipcc, "-fsanitize=address,undefined", "-fno-gpu-sanitize", drv_o, st_o, abi_o] + objs + ["-o", exe])
    # the HIP runtime's own allocations outlive main: leak checking off
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1")
    res = _run([exe], env=env)
    assert "abi sanitizer driver: ok" in res.stdout
    assert int(res.stdout.split("plans checked:")[1].split()[0]) > 10000
