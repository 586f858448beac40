"""The oracle's pins (tests/test_oracle.py) against an AddressSanitizer +
UndefinedBehaviorSanitizer build of oracle.c, in a subprocess with the
sanitizer runtimes preloaded: an out-of-bounds access, a use after free or
undefined arithmetic anywhere the pins reach aborts the run.  CPU only."""
import os
import subprocess
import sys
import tempfile

from oracle import build as OB

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_pins_pass_under_address_and_ub_sanitizers():
    with tempfile.TemporaryDirectory() as d:
        lib = OB.build(sanitize=True, out=os.path.join(d, "liboracle_asan.so"))
        syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
        assert "__asan_report" in syms and "__ubsan_handle" in syms  # really instrumented
        pre = OB.sanitizer_preload()
        if os.environ.get("LD_PRELOAD"):
            pre += ":" + os.environ["LD_PRELOAD"]
        env = dict(os.environ, ORACLE_LIB_OVERRIDE=lib, PYTHONDONTWRITEBYTECODE="1",
                   LD_PRELOAD=pre,
                   ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0:abort_on_error=1",
                   UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                            os.path.join(ROOT, "tests", "test_oracle.py")],
                           cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
        out = r.stdout + r.stderr
        assert r.returncode == 0, out[-3000:]
        assert "AddressSanitizer" not in out and "runtime error" not in out, out[-3000:]
        assert " passed" in out
