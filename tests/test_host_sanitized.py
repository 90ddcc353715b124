"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer.

1. The oracle (oracle/dm_oracle.c) built by gcc with address and undefined
   behaviour checks, no recovery, runs the whole pin suite in a child process
   with gcc's sanitizer runtime preloaded.
2. The engine's host code (argument and configuration checks, scratch
   planning, the entry points' error paths) built by hipcc with the same
   checks on the host side only -- device code is built as usual -- runs the
   host-only library tests in a child process with clang's runtime preloaded.

A read or write out of bounds, a use after free, a signed overflow, a bad
shift or a misaligned access on any path these suites reach fails the test.
Nothing here touches a GPU."""
import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2602_06502_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _gcc_runtime(name):
    p = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


def _clang_runtime():
    hits = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    return hits[0] if hits else None


def _env(preload, **extra):
    env = dict(os.environ)
    env["LD_PRELOAD"] = preload + ((" " + env["LD_PRELOAD"]) if env.get("LD_PRELOAD") else "")
    # the interpreter's own allocations are not ours: no leak report
    env["ASAN_OPTIONS"] = "detect_leaks=0:exitcode=86"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env.update(extra)
    return env


def _check(r):
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in r.stdout, out[-2000:]


@pytest.mark.timeout(600)
def test_oracle_pin_suite_sanitized(tmp_path):
    asan = _gcc_runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc has no AddressSanitizer runtime here")
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
                           *SAN, "-o", lib, os.path.join(ROOT, "oracle", "dm_oracle.c")])
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-s", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=_env(asan, DM_ORACLE_LIB=lib), capture_output=True, text=True,
                       timeout=580)
    _check(r)


def _host_sanitized_engine(objdir, lib):
    flags = ["-O1", "-g", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC]
    for f in SAN:
        flags += ["-Xarch_host", f]

    def one(src):
        obj = os.path.join(objdir, os.path.basename(src)[:-4] + ".o")
        r = subprocess.run([HIPCC, *flags, "-c", src, "-o", obj], capture_output=True, text=True)
        assert r.returncode == 0, r.stdout + r.stderr
        return obj

    with cf.ThreadPoolExecutor(max_workers=8) as ex:
        objs = list(ex.map(one, sorted(glob.glob(os.path.join(CSRC, "*.hip")))))
    link = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libsan"]
    for f in SAN[:1]:
        link += ["-Xarch_host", f]
    r = subprocess.run([*link, "-o", lib, *objs], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr


@pytest.mark.timeout(600)
def test_engine_host_checks_sanitized(tmp_path):
    asan = _clang_runtime()
    if asan is None:
        pytest.skip("no clang AddressSanitizer runtime under /opt/rocm/llvm")
    lib = str(tmp_path / "libdualmap_san.so")
    _host_sanitized_engine(str(tmp_path), lib)
    child = ("import sys; sys.path.insert(0, %r)\n"
             "import paper_2602_06502_amd as pk\n"
             "pk.load_library(%r)\n"
             "import pytest\n"
             "sys.exit(pytest.main(['-q', '-s', '-x', '-p', 'no:cacheprovider', %r]))\n"
             % (ROOT, lib, os.path.join(ROOT, "tests", "test_lib_cpu.py")))
    r = subprocess.run([sys.executable, "-c", child], cwd=ROOT, env=_env(asan), capture_output=True,
                       text=True, timeout=580)
    _check(r)
