"""The C-ABI host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only).

csrc/api.cpp (argument checks, workspace sizing, kernel choice, timing hooks)
is compiled for the host alone with both sanitizers, linked with host
stand-ins for the HIP runtime and the kernel launchers
(tests/host_sanitize/runtime_stub.cpp), and driven through every status path
of every entry point (tests/host_sanitize/abi_errors.cpp). Any sanitizer
report aborts the program; the test needs exit status 0 and no report.
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "host_sanitize")
CSRC = os.path.join(ROOT, "paper_2606_06256_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
HIPCC = "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang++"

# host-only compile; the sanitizer flags apply to the host pass (the only pass)
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


@pytest.fixture(scope="module")
def sanitized_program(tmp_path_factory):
    if not (os.path.exists(HIPCC) and os.path.exists(CLANG)):
        pytest.fail("hipcc / clang++ of ROCm not found")
    out = tmp_path_factory.mktemp("host_sanitize")
    objs = []
    defs = []
    for src in (os.path.join(CSRC, "api.cpp"), os.path.join(HERE, "runtime_stub.cpp"),
                os.path.join(HERE, "abi_errors.cpp")):
        o = str(out / (os.path.splitext(os.path.basename(src))[0] + ".o"))
        _run([HIPCC, "-xhip", "--offload-arch=gfx950", "--cuda-host-only", "-O1", "-g",
              "-std=c++17", *SAN, *defs, "-I", INCLUDE, "-I", CSRC, "-I", HERE, "-c", src, "-o", o])
        objs.append(o)
        if not defs:
            # api.cpp holds a device variable: its host code refers to the code-object
            # bundle by a name derived from the compilation unit; the stand-ins define it
            nm = _run(["/opt/rocm/llvm/bin/llvm-readelf", "-s", o]).stdout
            names = [m for m in re.findall(r"UND (__hip_fatbin_\w+)", nm)]
            assert len(set(names)) == 1, nm
            defs = [f"-DSEGPA_FATBIN_SYMBOL={names[0]}"]
    exe = str(out / "abi_errors")
    # linked without the HIP runtime: every HIP call the host code makes is a stand-in
    _run([CLANG, "-fsanitize=address,undefined", "-o", exe, *objs])
    return exe


def test_every_status_path_is_clean_under_asan_and_ubsan(sanitized_program):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=86",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1:exitcode=87")
    r = subprocess.run([sanitized_program], capture_output=True, text=True, env=env, timeout=120)
    report = r.stdout + r.stderr
    assert "runtime error" not in report, report
    assert "AddressSanitizer" not in report and "LeakSanitizer" not in report, report
    assert r.returncode == 0, report
    assert " 0 failed" in r.stdout, report
