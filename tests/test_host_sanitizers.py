"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU, no GPU needed): tests/native/host_sanitize.cpp drives workspace planning,
adpsgd_init's validation and plan (released again when the runtime has no
device), the host controller and learning rates over every mode, and the
refusals of calls that must not reach a device.  Every source is built with
the sanitizers on the host side only (each -fsanitize after -Xarch_host): the
device code of the HIP sources is compiled as usual and never launched here.
About a minute, most of it compiling kernels.hip."""
import os
import shutil
import subprocess
import tempfile

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "paper_2007_06134_amd", "csrc")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all"]


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    pytest.skip("hipcc not found")


@pytest.mark.slow
def test_library_host_code_is_clean_under_sanitizers():
    cc = _hipcc()
    base = [cc, "-O1", "-g", "-std=c++17", "-fno-omit-frame-pointer", *SAN, "-I", os.path.join(ROOT, "include"),
            "-I", SRC, "-ffp-contract=off"]
    with tempfile.TemporaryDirectory(prefix="host_san_") as tmp:
        objs = []
        jobs = [([*base, "-D__HIP_PLATFORM_AMD__", "-c", os.path.join(SRC, f)], f) for f in ("runtime.cpp", "controller.cpp")]
        jobs += [([*base, "-x", "hip", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
                   "-packed-fp32-ops", "-c", os.path.join(SRC, f)], f)
                 for f in ("kernels.hip", "noalloc.hip")]
        jobs.append(([*base, "-c", os.path.join(HERE, "native", "host_sanitize.cpp")], "host_sanitize.cpp"))
        procs = []
        for cmd, name in jobs:
            obj = os.path.join(tmp, name + ".o")
            procs.append((subprocess.Popen([*cmd, "-o", obj], stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                                           text=True), name))
            objs.append(obj)
        for p, name in procs:
            out, err = p.communicate(timeout=600)
            assert p.returncode == 0, f"{name}: {err[-3000:]}"
        exe = os.path.join(tmp, "host_sanitize")
        r = subprocess.run([cc, *SAN, *objs, "-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-lamdhip64",
                            "-Wl,-rpath,/opt/rocm/lib", "-o", exe], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1",
                   HIP_VISIBLE_DEVICES="")
        r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
        assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-4000:]
        assert r.stdout.strip().endswith("all ok"), r.stdout[-2000:]
        # the same build with a planted heap overflow in the driver is caught
        drv = objs[-1]
        subprocess.run([*base, "-DHOST_SANITIZE_PLANT", "-c", os.path.join(HERE, "native", "host_sanitize.cpp"),
                        "-o", drv], check=True, capture_output=True)
        subprocess.run([cc, *SAN, *objs, "-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-lamdhip64",
                        "-Wl,-rpath,/opt/rocm/lib", "-o", exe], check=True, capture_output=True)
        r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr, r.stderr[-2000:]
