"""Host sanitizer builds (CPU only): the oracle and the input generator, and
the C ABI's argument validation (api.cpp with host-only launcher stubs),
compiled with gcc/g++ -fsanitize=address,undefined and run; any sanitizer
finding aborts the driver, any failed check makes it exit non-zero."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer"]
HIP_INC = "/opt/rocm/include"
HIP_LIB = "/opt/rocm/lib"


def _run(cmd, cwd):
    r = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


def _env():
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1"
    return env


def test_oracle_and_generator_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "osd")
    _run(["gcc", "-std=c11"] + SAN + ["-fopenmp",
          os.path.join(ROOT, "tests", "sanitize", "oracle_synth_driver.c"),
          os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(ROOT, "synth", "gen.c"),
          "-lm", "-pthread", "-o", exe], str(tmp_path))
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=_env())
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout


@pytest.mark.skipif(not os.path.isdir(HIP_INC) or shutil.which("g++") is None,
                    reason="needs the HIP headers and g++")
def test_abi_validation_under_asan_ubsan(tmp_path):
    inc = ["-D__HIP_PLATFORM_AMD__", "-I" + HIP_INC, "-I" + os.path.join(ROOT, "include")]
    objs = []
    for src, lang in [(os.path.join(ROOT, "paper_2607_22578_amd", "csrc", "api.cpp"), "g++"),
                      (os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp"), "g++"),
                      (os.path.join(ROOT, "tests", "sanitize", "abi_driver.c"), "gcc")]:
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        std = ["-std=c++17"] if lang == "g++" else ["-std=c11"]
        _run([lang] + std + SAN + inc + ["-c", src, "-o", obj], str(tmp_path))
        objs.append(obj)
    exe = str(tmp_path / "abi")
    _run(["g++", "-fsanitize=address,undefined"] + objs +
         ["-L" + HIP_LIB, "-lamdhip64", "-Wl,-rpath," + HIP_LIB, "-o", exe], str(tmp_path))
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=_env())
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
