"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

The library is rebuilt with both sanitizers on its host pass only (argument
validation, split and workspace planning, layouts; device code as shipped)
and tests/test_abi.py -- every validation path, the struct layouts and the
planners, none of which launches a kernel -- runs against that build in a
child process, with the clang ASan runtime loaded first.  Any invalid memory
access or undefined operation aborts the child, failing this test.  CPU only.
"""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_checks_pass_under_host_asan_and_ubsan():
    sys.path.insert(0, ROOT)
    from paper_2604_07725_amd import build
    lib = build.build_sevo(8, sanitize=True)
    syms = subprocess.check_output(["nm", "-D", lib], text=True)
    assert "__asan_report" in syms and "__ubsan_handle" in syms, "build is not instrumented"
    env = dict(os.environ)
    # the ASan runtime must come first; anything already preloaded stays
    env["LD_PRELOAD"] = ":".join(p for p in (build.asan_runtime(), env.get("LD_PRELOAD")) if p)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["SEVO_LIBRARY"] = lib
    code = ("import sys, pytest; from paper_2604_07725_amd import sevo; "
            "assert sevo.LIB_PATH == sys.argv[1]; "
            "sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', '-m', 'not gpu', "
            "'tests/test_abi.py']))")
    r = subprocess.run([sys.executable, "-c", code, lib], cwd=ROOT, env=env,
                       stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-4000:]
    assert " passed" in r.stdout and "failed" not in r.stdout, r.stdout[-2000:]
