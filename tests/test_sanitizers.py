"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The oracle (oracle/oracle.cpp) is built with -fsanitize=address,undefined
  (undefined behaviour aborts: -fno-sanitize-recover) and its pins run in a
  child process that preloads the sanitizer runtimes: the golden example,
  the brute-force list models, the chain list model, the error rules, the
  special cases, the RL sampler, the dual update, the blackbox proxy and the
  executor.
* The C-ABI library is built with the sanitizers on its host code only (the
  GPU code is compiled as usual) and the CPU tests of the boundary run
  against it: loading, exports, and the argument checks of every entry point
  (NULL pools, rejected descriptions), which run before any device work.
A report from either sanitizer fails the child process and so the test."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _gcc_runtime(name):
    r = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True)
    p = os.path.realpath(r.stdout.strip())
    if not os.path.exists(p):
        pytest.skip(f"{name} not available")
    return p


def _run_child(args, env_extra):
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, *args], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    return out


def test_oracle_pins_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.check_call(["g++", "-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-pthread",
                           "-ffp-contract=off", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
                           "-o", lib, os.path.join(ROOT, "oracle", "oracle.cpp")])
    pre = ":".join([_gcc_runtime("libasan.so"), _gcc_runtime("libubsan.so")])
    files = ["tests/test_oracle_golden.py", "tests/test_oracle_bruteforce.py",
             "tests/test_oracle_chains.py", "tests/test_oracle_errors.py",
             "tests/test_oracle_special.py", "tests/test_oracle_rl.py", "tests/test_oracle_dual.py",
             "tests/test_oracle_rpm.py", "tests/test_oracle_executor.py"]
    out = _run_child(["-m", "pytest", *files, "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu"],
                     {"LD_PRELOAD": pre, "IM_ORACLE_LIB": lib})
    assert " passed" in out


def test_boundary_checks_under_asan_ubsan(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    clang_rt = None
    for root, _, names in os.walk("/opt/rocm/llvm/lib/clang"):
        if "libclang_rt.asan-x86_64.so" in names:
            clang_rt = os.path.join(root, "libclang_rt.asan-x86_64.so")
    if clang_rt is None:
        pytest.skip("clang AddressSanitizer runtime not available")
    csrc = os.path.join(ROOT, "paper_2606_11440_amd", "csrc")
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-omit-frame-pointer",
             "-I", os.path.join(ROOT, "include"), "-I", csrc]
    procs, objs = [], []
    for src in ("route.hip", "schedule.hip", "rows.hip", "pool.hip"):
        obj = str(tmp_path / (src + ".o"))
        objs.append(obj)
        procs.append(subprocess.Popen([HIPCC, *flags, "-c", os.path.join(csrc, src), "-o", obj],
                                      stdout=subprocess.DEVNULL, stderr=subprocess.PIPE))
    for p in procs:
        _, err = p.communicate(timeout=900)
        assert p.returncode == 0, err.decode()[-2000:]
    lib = str(tmp_path / "libinframind_san.so")
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC",
                           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                           "-o", lib, *objs])
    code = ("import sys; sys.path.insert(0, %r); import paper_2606_11440_amd._lib as L; "
            "L.LIB_PATH = %r; import pytest; "
            "sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', 'tests/test_abi.py']))" % (ROOT, lib))
    out = _run_child(["-c", code], {"LD_PRELOAD": clang_rt})
    assert " passed" in out
