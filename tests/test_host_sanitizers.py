"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

Every library source is compiled with the sanitizers on its host pass only
(device code as in the product build), linked with host_checks.cpp and
host_checks_c.c into one executable, and run: size queries over shapes up to
and past the largest layers, the schedule helper, status strings (as a C
caller passes them) and each entry point's argument validation.  All of
these return before anything is enqueued, so no GPU is needed."""
import concurrent.futures as cf
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_38978_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SOURCES = ["k_metric.hip", "k_sort.hip", "k_kmeans.hip", "k_pama.hip", "k_attn.hip",
           "k_kfilter.hip", "k_probe.hip", "park_api.hip"]
# sanitizer options for the host pass only, each behind its own -Xarch_host
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
DEVICE = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-w", "-Xclang",
          "-target-feature", "-Xclang", "-packed-fp32-ops", "-mllvm", "-amdgpu-mfma-vgpr-form"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_host_code_clean_under_asan_ubsan(tmp_path):
    objs = [str(tmp_path / (os.path.splitext(s)[0] + ".o")) for s in SOURCES]
    cmds = [[HIPCC, *DEVICE, *HOST_SAN, "-c", os.path.join(CSRC, s), "-o", o]
            for s, o in zip(SOURCES, objs)]
    inc = ["-I", os.path.join(ROOT, "include")]
    drv = [str(tmp_path / "host_checks.o"), str(tmp_path / "host_checks_c.o")]
    cmds.append([HIPCC, "-O1", "-std=c++17", *HOST_SAN, *inc, "-c",
                 os.path.join(ROOT, "tests", "host_checks.cpp"), "-o", drv[0]])
    cc = shutil.which("gcc") or "cc"
    cmds.append([cc, "-O1", "-std=c11", "-Wall", "-Werror", *inc, "-c",
                 os.path.join(ROOT, "tests", "host_checks_c.c"), "-o", drv[1]])
    with cf.ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
        list(ex.map(_run, cmds))
    # the library's host code carries the instrumentation
    syms = subprocess.run(["nm", objs[-1]], capture_output=True, text=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms
    exe = str(tmp_path / "host_checks")
    _run([HIPCC, "--offload-arch=gfx950", *HOST_SAN, "-o", exe, *drv, *objs])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "host checks passed" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr
