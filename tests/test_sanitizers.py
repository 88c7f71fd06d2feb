"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU
only; GPU sanitizers are not used):

- the oracle built with both sanitizers (MTDAO_ORACLE_SANITIZE=1), its
  pins, planted mutants and hypothesis properties run in a child process
  with gcc's ASan runtime preloaded;
- the C ABI's host code built with both sanitizers, driven through every
  host path by a plain-C program (tests/sanitize)."""

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _gcc_runtime(name: str) -> str:
    return subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                          check=True).stdout.strip()


def test_oracle_pins_mutants_properties_under_sanitizers():
    env = dict(os.environ, MTDAO_ORACLE_SANITIZE="1", LD_PRELOAD=_gcc_runtime("libasan.so"),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    probe = subprocess.run([sys.executable, "-c", "import oracle; oracle.build(); oracle.lib(); "
                            "print('libasan' in open('/proc/self/maps').read())"],
                           cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert probe.returncode == 0 and probe.stdout.strip().endswith("True"), probe.stdout + probe.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-n", "4",
                        "tests/test_oracle_pins.py", "tests/test_oracle_mutants.py", "tests/test_oracle_properties.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=1200)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-4000:]


def test_host_abi_paths_under_sanitizers():
    import importlib.util

    spec = importlib.util.spec_from_file_location("sanitize_build", os.path.join(ROOT, "tests", "sanitize", "build.py"))
    san_build = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(san_build)
    binary = san_build.build()
    r = subprocess.run([binary], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1"))
    assert r.returncode == 0, r.stdout + r.stderr
    assert "clean under the sanitizers" in r.stdout
    assert "runtime error" not in r.stderr
