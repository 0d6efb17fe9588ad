"""Sanitizer runs of the host code (CPU only, no GPU code is built):

* AddressSanitizer + UndefinedBehaviorSanitizer: the C oracle and the
  library's host sources (planner, step plan, gate, storage-tier I/O engine,
  preloader, ring, validation; the entry points that live in HIP translation
  units are stubs, tests/sanitize/device_stubs.cpp) are built with g++ / gcc,
  and the CPU tests of the oracle, ABI, planners, gate, storage tier and
  preloader run against those builds in a child process.
* ThreadSanitizer: tests/sanitize/preload_stress.cpp hammers the preloader
  from eight threads (fetches, restore-side holds, a lookahead of hints) and
  checks every image; built with ROCm's clang (GCC 11's libtsan reports
  libstdc++ condition-variable waits as double locks).

Each test first checks that its sanitizer is active (a planted heap overflow /
data race in a one-line program is reported)."""
import os
import shutil
import subprocess
import sys

import pytest

pytestmark = pytest.mark.slow

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_11744_amd", "csrc")
HOST_SOURCES = ["kvx_api.cpp", "kvx_gate.cpp", "kvx_io.cpp", "kvx_plan.cpp", "kvx_preload.cpp",
                "kvx_ring.cpp", "kvx_walk.cpp"]
INC = ["-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"),
       "-I" + CSRC]
ASAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
        "-fno-sanitize-recover=undefined"]
CLANG = "/opt/rocm/llvm/bin/clang++"


def _need(*tools):
    for t in tools:
        if not (os.path.exists(t) or shutil.which(t)):
            pytest.skip(f"{t} not available")
    if not os.path.exists("/opt/rocm/lib/libamdhip64.so"):
        pytest.skip("ROCm runtime library not available")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)} failed:\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    return r


def _compile_all(jobs):
    procs = [(cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                                    text=True)) for cmd in jobs]
    for cmd, p in procs:
        out, err = p.communicate()
        assert p.returncode == 0, f"{' '.join(cmd)} failed:\n{err[-3000:]}"


def _asan_env():
    libs = [subprocess.run(["gcc", f"-print-file-name={n}"], capture_output=True,
                           text=True).stdout.strip() for n in ("libasan.so", "libubsan.so")]
    env = dict(os.environ, LD_PRELOAD=" ".join(libs),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", KVX_NO_AUTOBUILD="1")
    return env


def test_asan_ubsan_host_builds(tmp_path):
    _need("g++", "gcc")
    # the sanitizer is active: a planted heap overflow is reported
    bad = tmp_path / "overflow.c"
    bad.write_text("#include <stdlib.h>\nint main(int c,char**v){volatile char*p=malloc(8);"
                   "p[7+c]=1;free((void*)p);return 0;}\n")
    # (ASan alone: UBSan's own checks would report this store first)
    _run(["gcc", "-O1", "-g", "-fsanitize=address", "-o", str(tmp_path / "overflow"), str(bad)])
    r = subprocess.run([str(tmp_path / "overflow")], capture_output=True, text=True)
    assert r.returncode != 0 and "AddressSanitizer" in r.stderr
    objs, jobs = [], []
    for f in HOST_SOURCES + ["../../tests/sanitize/device_stubs.cpp"]:
        src = os.path.normpath(os.path.join(CSRC, f))
        o = str(tmp_path / (os.path.basename(f) + ".o"))
        objs.append(o)
        jobs.append(["g++", *ASAN, "-std=c++17", "-fPIC", *INC, "-c", src, "-o", o])
    _compile_all(jobs)
    lib = str(tmp_path / "libkvx_asan.so")
    _run(["g++", "-shared", "-fsanitize=address,undefined", "-o", lib, *objs,
          "-L/opt/rocm/lib", "-lamdhip64", "-lhsa-runtime64", "-lpthread"])
    olib = str(tmp_path / "liboracle_asan.so")
    _run(["gcc", *ASAN, "-fPIC", "-shared", "-o", olib, os.path.join(ROOT, "oracle", "kvx_oracle.c")])
    env = _asan_env()
    env.update(KVX_TEST_LIB=lib, KVX_ORACLE_LIB=olib)
    tests = ["tests/test_oracle_pins.py", "tests/test_abi.py", "tests/test_step_plan.py",
             "tests/test_breakeven.py", "tests/test_storage_tier.py", "tests/test_preload.py",
             "tests/test_kvtest_util.py"]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu",
                        "-p", "no:cacheprovider", *tests,
                        # kvx_probe_stream is a stub in the host-only library
                        "--deselect", "tests/test_abi.py::test_probe_rejects_bad_arguments_on_the_host"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, f"tests under ASan/UBSan failed:\n{r.stdout[-4000:]}\n{r.stderr[-4000:]}"
    assert "passed" in r.stdout and "AddressSanitizer" not in r.stderr + r.stdout


def test_tsan_preloader_stress(tmp_path):
    _need(CLANG)
    tsan = ["-O1", "-g", "-fsanitize=thread", "-std=c++17"]
    race = tmp_path / "race.cpp"
    race.write_text("#include <thread>\nint x;\nint main(){std::thread t([]{x++;});x++;t.join();"
                    "return 0;}\n")
    _run([CLANG, *tsan, "-o", str(tmp_path / "race"), str(race)])
    r = subprocess.run([str(tmp_path / "race")], capture_output=True, text=True)
    assert "WARNING: ThreadSanitizer: data race" in r.stderr
    objs, jobs = [], []
    for f in ("kvx_io.cpp", "kvx_preload.cpp"):
        o = str(tmp_path / (f + ".o"))
        objs.append(o)
        jobs.append([CLANG, *tsan, "-fPIC", *INC, "-c", os.path.join(CSRC, f), "-o", o])
    _compile_all(jobs)
    exe = str(tmp_path / "preload_stress")
    _run([CLANG, *tsan, *INC, os.path.join(ROOT, "tests", "sanitize", "preload_stress.cpp"), *objs,
          "-o", exe, "-L/opt/rocm/lib", "-lamdhip64", "-lpthread", "-Wl,-rpath,/opt/rocm/lib"])
    files = tmp_path / "files"
    files.mkdir()
    # (slots, reserve, largest file KiB, slot KiB): roomy, tight, one slot short of the files
    for cfg in (("10", "2", "1536", "2048"), ("4", "0", "3072", "4096"), ("3", "0", "6144", "8192")):
        r = subprocess.run([exe, str(files), *cfg], capture_output=True, text=True, timeout=600,
                           env=dict(os.environ, TSAN_OPTIONS="halt_on_error=0"))
        assert r.returncode == 0, f"stress {cfg} failed:\n{r.stdout[-2000:]}\n{r.stderr[-4000:]}"
        assert "WARNING: ThreadSanitizer" not in r.stderr, r.stderr[-6000:]
        assert r.stdout.startswith("bad 0 "), r.stdout
