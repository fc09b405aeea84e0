"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU
only, no GPU code is built here):

- the library's argument validation and planning (csrc/plan.cpp, which makes
  no HIP call) linked into tests/sanitize/plan_driver.cpp with a stub
  compute-unit count: malformed and extreme arguments, a sweep of valid
  shapes through every planner, and the plans' invariants;
- the fp64 oracle (oracle/oracle.c) built with the sanitizers and driven by
  every oracle pin, in a child process that preloads the sanitizer runtime.

Any out-of-bounds access, use after free, signed overflow or other undefined
behaviour aborts the run with a report."""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True,
                          text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


pytestmark = pytest.mark.skipif(_runtime("libasan.so") is None,
                                reason="gcc's AddressSanitizer runtime is not installed")


def test_plan_code_under_sanitizers(tmp_path):
    exe = tmp_path / "plan_driver"
    subprocess.run(["g++", "-std=c++17", "-O1", *SAN,
                    "-I", os.path.join(ROOT, "include"),
                    "-I", os.path.join(ROOT, "paper_2408_11049_amd", "csrc"),
                    os.path.join(ROOT, "paper_2408_11049_amd", "csrc", "plan.cpp"),
                    os.path.join(ROOT, "tests", "sanitize", "plan_driver.cpp"),
                    "-o", str(exe)], check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300,
                       env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1:abort_on_error=0"})
    assert r.returncode == 0, r.stdout + r.stderr
    assert "plan driver: ok" in r.stdout
    # Every pass of the sweep reached balanced-verify plans (the driver
    # checks the counts; the line shows them).
    assert "balanced plans per pass:" in r.stdout


def test_oracle_pins_under_sanitizers(tmp_path):
    from oracle import build as obuild
    lib = obuild.build(out=str(tmp_path / "liboracle_san.so"), extra_flags=SAN)
    script = textwrap.dedent(f"""
        import sys
        sys.path[:0] = [{os.path.join(ROOT, 'tests')!r}, {ROOT!r}]
        import oracle
        from oracle_pins import ALL_PINS
        lib = oracle.open_library({lib!r})
        for pin in ALL_PINS:
            pin(lib=lib)
            print("pin ok:", pin.__name__, flush=True)
        print("all pins ok")
    """)
    env = {**os.environ, "LD_PRELOAD": _runtime("libasan.so"),
           "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}
    r = subprocess.run([sys.executable, "-c", script], capture_output=True, text=True,
                       timeout=900, env=env)
    assert r.returncode == 0 and "all pins ok" in r.stdout, (r.stdout[-3000:] + r.stderr[-3000:])
