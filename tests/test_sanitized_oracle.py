"""The oracle and the workload generator built with AddressSanitizer and UndefinedBehavior
Sanitizer (host code only, gcc), with the CPU pins run against that build: an out-of-bounds
access, a use after free or undefined arithmetic anywhere on the paths the pins reach fails the
run instead of passing silently."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g"]
# the CPU pins of the oracle (resolve and attention), the comparison policies and the generator
PINS = ["tests/test_oracle_resolve.py", "tests/test_oracle_attention.py",
        "tests/test_policy_study.py", "tests/test_workload.py"]


def _runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                       check=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


def test_pins_pass_under_address_and_undefined_sanitizers(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc has no AddressSanitizer runtime here")
    sys.path.insert(0, ROOT)
    import oracle
    import workload
    olib = oracle.build(force=True, path=str(tmp_path / "libhisparse_oracle.so"),
                        extra_flags=SAN)
    wlib = workload.build(force=True, path=str(tmp_path / "libhs_workload.so"), extra_flags=SAN)
    env = dict(os.environ)
    # the sanitizer runtime must come first among preloaded libraries (Python is not built
    # with it); anything already preloaded stays after it
    env["LD_PRELOAD"] = ":".join(x for x in (asan, env.get("LD_PRELOAD", "")) if x)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["HISPARSE_ORACLE_LIB"] = olib
    env["HS_WORKLOAD_LIB"] = wlib
    # --capture=sys: a sanitizer report (written to file descriptor 2) reaches this process
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "--capture=sys",
                        "-m", "not gpu", *PINS], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error:" not in tail, tail
