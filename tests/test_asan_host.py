"""Host code of libsmoes under AddressSanitizer (CPU only, no GPU).

Every HIP source is compiled for gfx950 as in the product build, with only
the host side instrumented (each -fsanitize flag behind -Xarch_host), into a
separate library under paper_2604_23996_amd/_build_asan/; tests/asan/
host_checks.cpp, built with the sanitizer, then drives the host-only paths
of the C ABI: descriptor validation, workspace sizes and the carving of the
layer workspace (each buffer written in full on a host allocation of exactly
the reported size), and the argument and shape errors that return before any
device call. The build is reused while its sources are unchanged."""
from __future__ import annotations

import concurrent.futures as cf
import glob
import hashlib
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2604_23996_amd")
OUT = os.path.join(PKG, "_build_asan")
DRIVER = os.path.join(ROOT, "tests", "asan", "host_checks.cpp")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang++"
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]
FLAGS = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         f"-I{os.path.join(ROOT, 'include')}"] + HOST_SAN


def _sources():
    return sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip")))


def _digest() -> str:
    h = hashlib.sha256(" ".join(FLAGS).encode())
    for p in _sources() + sorted(glob.glob(os.path.join(PKG, "csrc", "*.h"))) + \
            [os.path.join(ROOT, "include", "smoes.h"), DRIVER]:
        with open(p, "rb") as f:
            h.update(p.encode() + f.read())
    return h.hexdigest()


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l)
        raise RuntimeError(f"{' '.join(cmd[:3])} ... failed:\n{msgs}")


def _build() -> str:
    exe = os.path.join(OUT, "host_checks")
    stamp = os.path.join(OUT, "stamp")
    dig = _digest()
    if os.path.exists(exe) and os.path.exists(stamp) and open(stamp).read() == dig:
        return exe
    os.makedirs(OUT, exist_ok=True)
    objs = [os.path.join(OUT, os.path.basename(s) + ".o") for s in _sources()]
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        list(ex.map(lambda so: _run([HIPCC, *FLAGS, "-c", so[0], "-o", so[1]]), zip(_sources(), objs)))
    lib = os.path.join(OUT, "libsmoes_asan.so")
    # host links with the sanitizer runtime (clang, not hipcc: no device code is built here)
    _run([CLANG, "-shared", "-fPIC", "-fsanitize=address", *objs, "-L/opt/rocm/lib", "-lamdhip64",
          "-Wl,-rpath,/opt/rocm/lib", "-o", lib])
    _run([CLANG, "-O1", "-g", "-std=c++17", "-fsanitize=address", "-fno-omit-frame-pointer",
          f"-I{os.path.join(ROOT, 'include')}", DRIVER, f"-L{OUT}", "-lsmoes_asan", f"-Wl,-rpath,{OUT}",
          "-o", exe])
    with open(stamp, "w") as f:
        f.write(dig)
    return exe


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm compilers not found")
def test_host_paths_under_address_sanitizer():
    exe = _build()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:exitcode=23")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert "host checks passed" in r.stdout
