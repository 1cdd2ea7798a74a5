"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The planner, the C ABI's host paths and the evictor (``plan.cpp``,
``api.cpp``, ``evictor.cpp``) and the oracle (``oracle/*.c``) are compiled
with g++/gcc ``-fsanitize=address,undefined`` into a scratch directory; the
kernel launchers and the no-allocation entry point, which need device code,
are replaced by stubs that host-only plans never reach
(``tests/sanitize/host_stubs.cpp``).  The plan-structure tests, the CPU
interpreter of plans, the block-table validator tests, the oracle pins and
the evictor tests then run in a child process that loads those builds
(``MSA_LIBRARY`` / ``MSA_ORACLE_LIBRARY``) with the ASan runtime preloaded.
Any sanitizer report fails the run.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_02964_amd", "csrc")
ROCM = "/opt/rocm"

# tests that compile or start programs of their own (plain C consumer, HIP
# runtime identity, ISA) or plant mutants stay out of the instrumented run
SUITE = ["tests/test_abi_host.py", "tests/test_oracle_pins.py", "tests/test_oracle_append.py",
         "tests/test_oracle_evictor.py", "tests/test_evictor.py"]
DESELECT = "not plain_c_consumer and not one_hip_runtime"

SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
       "-g", "-O1", "-fPIC", "-shared"]


def _runtime(name):
    out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.fixture(scope="module")
def sanitized_builds(tmp_path_factory):
    asan = _runtime("libasan.so")
    if not (shutil.which("g++") and shutil.which("gcc") and asan
            and os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime_api.h"))):
        pytest.skip("g++/gcc with ASan or the HIP headers not available")
    out = tmp_path_factory.mktemp("sanitized")
    lib = str(out / "libmsa.so")
    cmd = ["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"),
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           *(os.path.join(CSRC, f) for f in ("plan.cpp", "api.cpp", "evictor.cpp")),
           os.path.join(ROOT, "tests", "sanitize", "host_stubs.cpp"),
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-o", lib]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-3000:]
    olib = str(out / "libmsa_oracle.so")
    cmd = ["gcc", "-std=c11", *SAN, "-ffp-contract=off", "-fno-fast-math", "-pthread",
           os.path.join(ROOT, "oracle", "msa_oracle.c"), os.path.join(ROOT, "oracle", "evictor_oracle.c"),
           "-o", olib, "-lm"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-3000:]
    return lib, olib, asan


def test_host_code_is_clean_under_asan_and_ubsan(sanitized_builds):
    lib, olib, asan = sanitized_builds
    env = dict(os.environ)
    env.update({
        "MSA_LIBRARY": lib,
        "MSA_ORACLE_LIBRARY": olib,
        "LD_PRELOAD": asan,
        # Python and torch keep memory until exit: leaks are not checked
        "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "PYTHONDONTWRITEBYTECODE": "1",
    })
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-n", "4", "-p", "no:cacheprovider", "-m", "not gpu",
           "-k", DESELECT, *SUITE]
    res = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=1500)
    text = res.stdout + res.stderr
    assert "AddressSanitizer" not in text and "runtime error:" not in text, text[-6000:]
    assert res.returncode == 0, text[-6000:]
    assert " passed" in res.stdout


def test_the_instrumented_run_reports_a_planted_overflow(sanitized_builds, tmp_path):
    """The harness itself: a copy of the oracle whose score buffer is one
    element short must make the same child-process setup report a heap
    overflow (the mistake is planted in the copy, on the CPU)."""
    _, _, asan = sanitized_builds
    src = open(os.path.join(ROOT, "oracle", "msa_oracle.c")).read()
    good = "malloc(sizeof(double) * ((size_t)J->max_pos + 1))"
    assert src.count(good) == 1
    bad_src = tmp_path / "msa_oracle_short.c"
    bad_src.write_text(src.replace(good, "malloc(sizeof(double) * ((size_t)J->max_pos))"))
    olib = str(tmp_path / "libmsa_oracle_short.so")
    res = subprocess.run(["gcc", "-std=c11", *SAN, "-pthread", str(bad_src), "-o", olib, "-lm"],
                         capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-3000:]
    env = dict(os.environ, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               PYTHONDONTWRITEBYTECODE="1")
    code = ("import oracle, workloads\n"
            f"lib = oracle.load_library({olib!r})\n"
            "oracle.forward(workloads.make_config(1), lib=lib, num_threads=1)\n")
    res = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                         timeout=300)
    assert res.returncode != 0
    assert "AddressSanitizer: heap-buffer-overflow" in res.stderr, res.stderr[-3000:]
