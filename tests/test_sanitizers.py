"""AddressSanitizer / UndefinedBehaviorSanitizer runs of the host code (CPU only, gcc/g++; no GPU code is
built with a sanitizer): the C ABI layer of libmurmur with a stub of its kernel launchers, driven through
every host-only entry point on random inputs and every argument check of the device calls; and the fp64
oracle on random layouts, policies and caches.  The two are built and run as separate programs."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="needs gcc")


def build_and_run(tmp_path, name, cmd):
    exe = str(tmp_path / name)
    subprocess.run(cmd + ["-o", exe], check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "ERROR" not in res.stderr and "runtime error" not in res.stderr, res.stderr
    return res.stdout


def test_abi_layer_under_sanitizers(tmp_path):
    csrc = os.path.join(ROOT, "paper_2606_01483_amd", "csrc")
    out = build_and_run(tmp_path, "host_driver", [
        "g++", "-std=c++17", *SAN, f"-I{ROOT}/include", f"-I{csrc}", os.path.join(csrc, "api.cpp"),
        os.path.join(HERE, "launch_stub.cpp"), os.path.join(HERE, "host_driver.cpp")])
    assert "host driver: ok" in out


def test_oracle_under_sanitizers(tmp_path):
    out = build_and_run(tmp_path, "oracle_driver", [
        "gcc", "-std=c11", *SAN, "-pthread", os.path.join(ROOT, "oracle", "murmur_oracle.c"),
        os.path.join(HERE, "oracle_driver.c"), "-lm"])
    assert "oracle driver: ok" in out
