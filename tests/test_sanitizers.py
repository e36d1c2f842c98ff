"""Address and undefined-behaviour sanitizer builds of the host code, run on the CPU.

* oracle/eqref.c with tests/sanitize/oracle_driver.c (gcc): every oracle entry
  point on exactly-sized heap buffers across group orders and edge shapes;
* libeqlinear's host side (csrc/eql_api.cpp, eql_dispatch.cpp; hipcc with the
  sanitizers on the host pass only) with tests/sanitize/abi_driver.cpp:
  status strings, size queries, the weight-gradient planning over many shapes
  and argument errors, all of which return before any kernel launch.  It links
  the kernel objects of the regular build (paper_2607_21271_amd/_build).

Any sanitizer report aborts the driver (no recovery), which fails the test.
"""
import glob
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2607_21271_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, (" ".join(cmd), r.stdout[-4000:], r.stderr[-4000:])
    return r


def test_oracle_under_asan_ubsan():
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    d = tempfile.mkdtemp()
    exe = os.path.join(d, "oracle_driver")
    _run(["gcc", "-O1", "-g", "-std=gnu11", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          "-fno-fast-math", "-ffp-contract=off", os.path.join(ROOT, "oracle", "eqref.c"),
          os.path.join(HERE, "oracle_driver.c"), "-lm", "-o", exe])
    r = _run([exe])
    assert "oracle driver: ok" in r.stdout


def _no_gpu_visible():
    try:
        import torch
        return torch.cuda.device_count() == 0
    except Exception:
        return True


def test_library_host_code_under_asan_ubsan():
    objs = sorted(glob.glob(os.path.join(ROOT, "paper_2607_21271_amd", "_build", "inst_*", "inst_*.o")))
    if len(objs) != 32 or not os.path.exists(HIPCC):
        pytest.skip("needs the regular build's kernel objects (run __graft_entry__.build()) and hipcc")
    d = tempfile.mkdtemp()
    common = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
              "-O1", "-g", "-std=c++20", "-I" + os.path.join(ROOT, "include")]
    host_objs = []
    for src in ("eql_api.cpp", "eql_dispatch.cpp"):
        o = os.path.join(d, src + ".o")
        _run([HIPCC, *common, *SAN, "-Xarch_host", "-fno-sanitize-recover=all", "-fPIC", "-x", "hip", "-c",
              os.path.join(CSRC, src), "-o", o])
        host_objs.append(o)
    drv = os.path.join(d, "abi_driver.o")
    _run([HIPCC, "-O1", "-g", "-std=c++20", "-I" + os.path.join(ROOT, "include"), *SAN,
          "-Xarch_host", "-fno-sanitize-recover=all", "-x", "c++", "-c",
          os.path.join(HERE, "abi_driver.cpp"), "-o", drv])
    exe = os.path.join(d, "abi_driver")
    _run([HIPCC, "--offload-arch=gfx950", *SAN, *host_objs, drv, *objs, "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    r = _run([exe] + (["nodev"] if _no_gpu_visible() else []), env=env)
    assert "abi driver: ok" in r.stdout
