"""Host logic of libaugtree without a GPU, under AddressSanitizer and
UndefinedBehaviorSanitizer: the host library source (augtree.cpp) is compiled
with g++ together with CPU stand-ins for the HIP runtime and the kernel
launchers (tests/host/fake_hip.cpp) and a test program
(tests/host/host_abi_test.cpp) that runs every entry point on ragged batches,
checks every launch's tile schedule (bounds, causal geometry, each output row
written once, visible pairs equal to the method's counts), the validation
errors, and the HIP-error path (each launch or the schedule copy failing in
turn returns AUGTREE_ERR_HIP with a message, no crash)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_33133_amd", "csrc")
HOST = os.path.join(ROOT, "tests", "host")


@pytest.mark.timeout(600)
def test_host_logic_under_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not found")
    exe = str(tmp_path / "host_abi_test")
    # host-only build (no HIP source on this line): the sanitizers apply to host code
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
           os.path.join(CSRC, "augtree.cpp"), os.path.join(HOST, "fake_hip.cpp"), os.path.join(HOST, "host_abi_test.cpp"),
           "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=500)
    assert r.returncode == 0 and r.stdout.startswith("ok"), (r.stdout[-4000:] + r.stderr[-4000:])
    chunked = int(r.stdout.split(",")[1].split()[0])
    assert chunked >= 40, r.stdout   # the chunked tree backward was exercised
