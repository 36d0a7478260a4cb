"""The host driver's stream-capture sequences against a model of HIP's
documented capture rules (tests/hipsim): the library's lstmss_api.cpp is
built for the CPU against a stand-in runtime that tracks which capture every
stream and event belongs to, with the layer-stack capture path compiled in,
and driven through the call sequences of the GPU tests (stack calls recorded,
replayed and re-recorded, single-layer captures in between, direct calls,
side streams, bidirectional calls).  No sequence may break a rule; the model
itself must flag every forbidden sequence planted in its self-test.  Built
with AddressSanitizer on the host code."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CXX = "/opt/rocm/llvm/bin/clang++"


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    if not os.path.exists(CXX) or shutil.which("ld") is None:
        pytest.skip("no host clang++")
    out = tmp_path_factory.mktemp("hipsim")
    flags = ["-std=c++17", "-O1", "-g", "-fsanitize=address", "-fno-omit-frame-pointer",
             "-I" + os.path.join(ROOT, "tests", "hipsim"), "-DLSTMSS_STACK_GRAPHS=1"]
    srcs = [os.path.join(ROOT, "paper_1806_00512_amd", "csrc", "lstmss_api.cpp"),
            os.path.join(ROOT, "tests", "hipsim", "hipsim_runtime.cpp"),
            os.path.join(ROOT, "tests", "hipsim", "hipsim_stubs.cpp"),
            os.path.join(ROOT, "tests", "hipsim", "hipsim_driver.cpp")]
    objs = []
    for i, src in enumerate(srcs):
        obj = str(out / ("o%d.o" % i))
        subprocess.run([CXX] + flags + ["-c", src, "-o", obj], check=True)
        objs.append(obj)
    exe = str(out / "driver")
    subprocess.run([CXX, "-fsanitize=address", "-o", exe] + objs + ["-lpthread"], check=True)
    return exe


def run(exe, *args):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0")
    return subprocess.run([exe] + list(args), capture_output=True, text=True, env=env,
                          timeout=120)


def test_model_flags_forbidden_sequences(driver):
    r = run(driver, "--selftest")
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.count(": flagged") == 7 and "NOT FLAGGED" not in r.stdout


def test_capture_sequences_follow_the_rules(driver):
    r = run(driver)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "violations 0" in r.stdout and "streams left capturing 0" in r.stdout
    assert "call failed" not in r.stdout
