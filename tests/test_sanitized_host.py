"""The library's host code under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only): the layer allocator against the
oracle on random instances and every invalid-argument path, the dry-run
memory model against its closed form, and the stage calls that must reject
their arguments before touching a device.  The sanitized library is built by
paper_2202_11836_amd.build.build_sanitized (host code instrumented, device
code as usual) and exercised in a child process that preloads the sanitizer
runtime and does not import torch (tests/_sanitized_driver.py).  Any
sanitizer report ends the child with a non-zero status."""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.timeout(900)
def test_host_paths_under_address_and_undefined_behaviour_sanitizers():
    from paper_2202_11836_amd import build as B
    try:
        lib = B.build_sanitized()
        rt = B.sanitizer_runtime()
    except (RuntimeError, OSError) as e:  # no hipcc / sanitizer runtime here
        pytest.skip(str(e))
    env = dict(os.environ)
    env["LD_PRELOAD"] = rt
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([sys.executable, os.path.join(HERE, "_sanitized_driver.py"), lib], env=env,
                       capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "sanitized host paths: ok" in r.stdout
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
