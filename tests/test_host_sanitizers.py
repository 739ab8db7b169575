"""The library's host code (argument checks, dispatch, the plan generator,
the plan search's workspace carving) built with AddressSanitizer and
UndefinedBehaviorSanitizer, running the ABI tests on the CPU.

The host sources are compiled by g++ with the sanitizers; the HIP sources are
compiled as usual (no sanitizer reaches device code) and linked in, so the
library is complete.  The ABI tests run in a child process that preloads the
ASan runtime and loads the sanitized library through DFA_LIBRARY; any sanitizer report
makes the child fail (halt on the first error, no recovery)."""
import hashlib
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2406_08552_amd")
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build", "hostsan")
HOST_SOURCES = ["dfa_api.cpp", "dfa_search.cpp"]


def _run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, **kw)
    noise = "is not a recognized feature for this target"
    out = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
    assert res.returncode == 0, f"{' '.join(cmd[:3])} ... failed:\n{out[-4000:]}"
    return out


def _device_objects():
    """The HIP sources compiled as the library compiles them (cached by content)."""
    sys.path.insert(0, ROOT)
    from paper_2406_08552_amd import build
    objs = []
    flags = [f for f in build.HIPCC_FLAGS if f != "-shared"]
    for src in build.SOURCES:
        if not src.endswith(".hip"):
            continue
        path = os.path.join(CSRC, src)
        key = hashlib.sha256(open(path, "rb").read() + open(os.path.join(CSRC, "dfa_internal.h"), "rb").read()
                             + " ".join(flags).encode()).hexdigest()[:16]
        obj = os.path.join(BUILD, f"{src}.{key}.o")
        if not os.path.exists(obj):
            _run([build.hipcc(), *flags, "-c", f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}", path, "-o", obj])
        objs.append(obj)
    return objs


def test_abi_tests_under_host_sanitizers():
    gxx = shutil.which("g++")
    if gxx is None or not os.path.exists("/opt/rocm/lib/libamdhip64.so"):
        pytest.skip("g++ or the HIP runtime library is missing")
    libasan = subprocess.run([gxx, "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(libasan) or not os.path.exists(libasan):
        pytest.skip("the ASan runtime of g++ is missing")
    os.makedirs(BUILD, exist_ok=True)
    objs = _device_objects()
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    host_objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".san.o")
        _run([gxx, "-std=c++17", "-O1", "-g", "-fPIC", *san, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
              f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}", "-c", os.path.join(CSRC, src), "-o", obj])
        host_objs.append(obj)
    lib = os.path.join(BUILD, "libdfa_hostsan.so")
    _run([gxx, "-shared", *san, *host_objs, *objs, "-L/opt/rocm/lib", "-Wl,-rpath,/opt/rocm/lib", "-lamdhip64",
          "-o", lib])
    env = dict(os.environ)
    env.update({"LD_PRELOAD": libasan, "DFA_LIBRARY": lib,
                "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0",
                "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
                "HIP_VISIBLE_DEVICES": "", "CUDA_VISIBLE_DEVICES": ""})
    probe = subprocess.run([sys.executable, "-c", "from paper_2406_08552_amd import dfa; print(dfa.lib()._name)"],
                           capture_output=True, text=True, env=env, cwd=ROOT, timeout=300)
    assert probe.returncode == 0 and probe.stdout.strip().endswith("libdfa_hostsan.so"), probe.stdout + probe.stderr
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                          os.path.join(ROOT, "tests", "test_abi.py")], capture_output=True, text=True, env=env,
                         cwd=ROOT, timeout=600)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-6000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert " passed" in out, out[-2000:]
