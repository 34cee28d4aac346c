"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
while it decodes on the GPU (device code as usual): the driver built by
tests/sanitize/build.py (__graft_entry__.build builds it) runs a tiny fp32
model through prefill, forced / Q-network / sampled / exit-policy steps,
injected failures with rollback, two steps in flight, truncation and resume,
and a four-page KV pool running out.  Leak detection on (the ROCm runtime's
own allocations kept at exit are suppressed)."""
import os
import subprocess

import pytest

from tests.parity import say
from tests.sanitize import build as sb

pytestmark = pytest.mark.gpu


@pytest.mark.skipif(not os.path.exists(sb.RUNTIME_CHECK), reason="sanitizer driver not built (tests/sanitize/build.py)")
def test_runtime_host_clean_under_asan_ubsan_while_decoding():
    say("running %s" % sb.RUNTIME_CHECK)
    p = subprocess.run([sb.RUNTIME_CHECK], capture_output=True, text=True, timeout=600, env=sb.env())
    out = p.stdout + p.stderr
    say(out[-3000:])
    assert p.returncode == 0 and "runtime sanitizer run: clean" in out and "decoded on the GPU" in out, out[-6000:]
