"""AddressSanitizer + UndefinedBehaviorSanitizer runs of the host code (CPU):

* the C oracle (oracle/mc_oracle.c, serial: the OpenMP pragmas are left out)
  driven by tests/native/sanitize_driver.c over every orc_* function, with
  leak detection;
* the C-ABI library's host code (api.hip compiled with host-only sanitizers,
  linked with the library's other objects) driven over the size queries,
  every validation path that returns before a launch, the pruning
  threshold, the PMQ significance and the Eq. 4 allocation -- no GPU needed.

A memory or undefined-behaviour error aborts the run with the sanitizer's
report; an unmet expectation exits non-zero."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OUT = os.path.join(ROOT, "_build", "san")
CLANG = "/opt/rocm/llvm/bin/clang"
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
ORACLE = os.path.join(ROOT, "oracle", "mc_oracle.c")
DRIVER = os.path.join(ROOT, "tests", "native", "sanitize_driver.c")
API = os.path.join(ROOT, "paper_2410_06270_amd", "csrc", "api.hip")


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, "%s\n%s" % (" ".join(cmd), r.stdout[-4000:])
    return r.stdout


def _env(leaks):
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=%d:abort_on_error=1" % int(leaks)
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    return env


@pytest.fixture(scope="module")
def outdir():
    if not os.path.exists(CLANG):
        pytest.skip("ROCm clang not found")
    os.makedirs(OUT, exist_ok=True)
    return OUT


def test_oracle_asan_ubsan(outdir):
    o = os.path.join(outdir, "oracle.o")
    _run([CLANG, "-O1", "-g", "-std=c99", "-ffp-contract=off", "-Wno-unknown-pragmas", *SAN, "-c", ORACLE, "-o", o])
    d = os.path.join(outdir, "driver.o")
    _run([CLANG, "-O1", "-g", "-std=c99", *SAN, "-c", DRIVER, "-o", d])
    exe = os.path.join(outdir, "oracle_san")
    _run([CLANG, *SAN, d, o, "-lm", "-o", exe])
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, env=_env(True))
    assert r.returncode == 0 and "sanitized run ok" in r.stdout, r.stdout[-4000:]


def test_api_host_asan_ubsan(outdir):
    from paper_2410_06270_amd import build
    objdir = build.OBJ
    if not all(os.path.exists(os.path.join(objdir, os.path.basename(s)[:-4] + ".o")) for s in build.sources()):
        build.build()
    o = os.path.join(outdir, "oracle.o")
    _run([CLANG, "-O1", "-g", "-std=c99", "-ffp-contract=off", "-Wno-unknown-pragmas", *SAN, "-c", ORACLE, "-o", o])
    d = os.path.join(outdir, "driver_api.o")
    _run([CLANG, "-O1", "-g", "-std=c99", *SAN, "-DWITH_API", "-c", DRIVER, "-o", d])
    a = os.path.join(outdir, "api.o")
    host_san = []
    for f in SAN:                      # host code only: never the GPU code
        host_san += ["-Xarch_host", f]
    _run(["hipcc", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-ffp-contract=off",
          *host_san, "-c", API, "-o", a])
    others = [os.path.join(objdir, os.path.basename(s)[:-4] + ".o") for s in build.sources()
              if os.path.basename(s) != "api.hip"]
    exe = os.path.join(outdir, "api_san")
    _run([CLANG + "++", *SAN, d, o, a, *others, "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib",
          "-o", exe])
    # the HIP runtime's own allocations are not instrumented: no leak check here
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, env=_env(False))
    assert r.returncode == 0 and "sanitized run ok" in r.stdout, r.stdout[-4000:]
