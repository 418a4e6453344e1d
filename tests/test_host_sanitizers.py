"""The host code of the library (descriptor and pointer validation,
workspace layout, the no-allocation entry point's size check, the offload
residency plan caee_lru_step) built with AddressSanitizer and
UndefinedBehaviorSanitizer, and exercised by the CPU tests of the C ABI and
of the residency plan.  Device code is built as usual.  No GPU."""
import importlib.util
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _build_module():
    spec = importlib.util.spec_from_file_location("caee_build", os.path.join(ROOT, "paper_2606_29982_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_host_code_under_asan_and_ubsan(tmp_path):
    b = _build_module()
    lib = b.build(out=str(tmp_path / "libcaee_host_sanitized.so"), sanitize_host=True)
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
    assert "__asan_report_load" in syms and "__ubsan_handle" in syms   # instrumented host code
    env = dict(os.environ, CAEE_LIBRARY=lib, LD_PRELOAD=b.asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(ROOT, "tests", "test_abi.py"), os.path.join(ROOT, "tests", "test_lru_host.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    print(r.stdout[-3000:], r.stderr[-3000:])
    assert r.returncode == 0
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr
    # the sanitized build was the one loaded
    assert "passed" in r.stdout
