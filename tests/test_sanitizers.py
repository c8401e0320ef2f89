"""AddressSanitizer / UndefinedBehaviorSanitizer runs of the host code (CPU).

* the float64 oracle, built with gcc and both sanitizers, runs its pins;
* libags's host code (argument validation, workspace layout, state and
  planner), built by hipcc with the sanitizers on the host pass only and
  without the step, finalize, correction and update kernels (launcher
  stubs stand in for them; the two table kernels of the no-alloc entry
  point, which live beside the host code, are compiled for the GPU without
  sanitizers), runs the C-ABI and planner tests.

Each run is a subprocess with the matching sanitizer runtime preloaded; a
report makes it fail.  GPU code is never built with a sanitizer here.
"""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2603_18112_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _gcc_runtime(name):
    try:
        p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                           check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return p if os.path.isabs(p) and os.path.exists(p) else None


def _run(code, env_extra, logdir, timeout=600):
    """Run code in a subprocess; sanitizer reports go to files in logdir
    (pytest's capture of the child's stderr would hide them)."""
    logdir = os.path.join(str(logdir), "sanitizer_logs")
    os.makedirs(logdir, exist_ok=True)
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = f"detect_leaks=0:log_path={logdir}/asan"
    env["UBSAN_OPTIONS"] = f"print_stacktrace=1:log_path={logdir}/ubsan"
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=timeout)
    out = r.stdout + r.stderr
    reports = "".join(open(p, errors="replace").read() for p in sorted(glob.glob(f"{logdir}/*")))
    assert not reports, reports[:6000]
    assert r.returncode == 0, out[-4000:]
    return out


def test_oracle_under_asan_and_ubsan(tmp_path):
    asan, ubsan = _gcc_runtime("libasan.so"), _gcc_runtime("libubsan.so")
    if not (shutil.which("gcc") and asan and ubsan):
        pytest.skip("gcc sanitizer runtimes not available")
    lib = str(tmp_path / "liboracle_ags_san.so")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    "-ffp-contract=off", os.path.join(ROOT, "oracle", "ags_oracle.c"), "-o", lib,
                    "-lm"], check=True)
    code = ("import sys, pytest; sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', "
            "'tests/test_oracle_pins.py']))")
    out = _run(code, {"LD_PRELOAD": f"{asan}:{ubsan}", "AGS_ORACLE_LIB": lib}, tmp_path)
    assert " passed" in out


def test_libags_host_code_under_asan_and_ubsan(tmp_path):
    rts = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not (os.path.exists(HIPCC) and rts):
        pytest.skip("hipcc or the clang sanitizer runtime not available")
    lib = str(tmp_path / "libags_san_host.so")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-fPIC", "-shared", "-shared-libasan",
           "-Xarch_host", "-fsanitize=address",
           "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "ags_api.hip"), os.path.join(CSRC, "ags_plan.cpp"),
           os.path.join(ROOT, "tests", "sanitizer_stubs.hip"), "-o", lib]
    subprocess.run(cmd, check=True, capture_output=True)
    code = ("import sys; sys.path.insert(0, 'tests')\n"
            "from paper_2603_18112_amd import ags\n"
            f"ags.load_library({lib!r})\n"
            "import pytest\n"
            "sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', 'tests/test_abi.py', "
            "'tests/test_plan_parity.py']))")
    out = _run(code, {"LD_PRELOAD": sorted(rts)[-1]}, tmp_path)
    assert " passed" in out
