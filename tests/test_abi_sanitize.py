"""CPU-only: the library's host code built with AddressSanitizer and UndefinedBehaviorSanitizer
(host side only; device code is unchanged), driven through every entry point's validation and
no-device error paths by tests/abi_sanitize.cpp.  Any out-of-bounds access, use of freed
memory or undefined behaviour in the host-side argument checks, workspace carving or status
handling aborts the driver."""

import concurrent.futures
import hashlib
import os
import shutil
import subprocess

import pytest

from paper_2505_04846_amd import build as B

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(B.PKG_DIR, "_build", "asan")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]


def _digest():
    h = hashlib.sha256()
    for name in sorted(os.listdir(B.CSRC)) + [os.path.join(HERE, "abi_sanitize.cpp"),
                                              os.path.join(B.INCLUDE, "hiperrag.h")]:
        path = name if os.path.isabs(name) else os.path.join(B.CSRC, name)
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _build():
    exe = os.path.join(OUT, "abi_sanitize_" + _digest())
    if os.path.exists(exe):
        return exe
    shutil.rmtree(OUT, ignore_errors=True)
    os.makedirs(OUT)
    hipcc = B._hipcc()

    def comp(src):
        obj = os.path.join(OUT, os.path.splitext(os.path.basename(src))[0] + ".o")
        cmd = [hipcc, *B.COMMON_FLAGS, *B.FILE_FLAGS.get(os.path.basename(src), []), *SAN,
               "-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr[-3000:]}")
        return obj

    srcs = [os.path.join(B.CSRC, s) for s in B.SOURCES] + [os.path.join(HERE, "abi_sanitize.cpp")]
    with concurrent.futures.ThreadPoolExecutor(8) as ex:
        objs = list(ex.map(comp, srcs))
    # link on the host with the C++ driver (no device file on this line)
    rocm = os.path.dirname(os.path.dirname(hipcc))
    cmd = ["g++", *objs, "-fsanitize=address,undefined", "-o", exe, f"-L{rocm}/lib",
           f"-Wl,-rpath,{rocm}/lib", "-lamdhip64"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode:
        raise RuntimeError(f"link failed:\n{r.stderr[-3000:]}")
    return exe


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++ for the host link")
@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="for machines without a GPU: the driver "
                    "calls entry points with fake device pointers")
def test_host_code_under_asan_and_ubsan():
    exe = _build()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, f"{r.stdout}\n{r.stderr[-4000:]}"
    assert "ok: 0 failures" in r.stdout
