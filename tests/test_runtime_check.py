"""The C ABI driven by `cas_runtime_check` (csrc/runtime_check.c), an
executable whose runtime host code is built under AddressSanitizer and
UndefinedBehaviorSanitizer: any invalid host memory access or undefined
operation in the runtime aborts it with a non-zero status.

- CPU: tree metadata, configuration checks and the argument checks of the
  kernel-level entry points (no device is opened).
- GPU: the same, then small fp32 and bf16 GQA decoders through 90 rounds of
  drafts, verify, top-K, acceptance and compaction over more tree shapes than
  the graph cache keeps, profiling, direct launches, KV load and read, and the
  error paths.
"""
import os
import subprocess

import pytest

from paper_2510_26843_amd import build

# the harness may preload a library of its own: the statically linked
# sanitizer runtime does not need to come first; leaks of the HIP runtime at
# exit are not the runtime's
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1:verify_asan_link_order=0",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _exe():
    if not os.path.exists(build.RUNTIME_CHECK):
        try:
            build.build_runtime_check()
        except RuntimeError as e:
            pytest.skip(str(e))
    return build.RUNTIME_CHECK


def _run(args, timeout):
    r = subprocess.run([_exe(), *args], capture_output=True, text=True, timeout=timeout, env=ENV)
    print(r.stdout[-2000:], r.stderr[-4000:])
    return r


def test_runtime_check_host_paths():
    r = _run(["--host-only"], 120)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "all checks passed (host only)" in r.stdout


@pytest.mark.gpu
@pytest.mark.timeout(300)
def test_runtime_check_on_device():
    r = _run([], 240)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "all checks passed (host and device)" in r.stdout
