"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer: oracle.c
and the brute-force checker are rebuilt with both sanitizers (any report
aborts), then the pin harness and the oracle's own test files run against
that build in a child process, over the worked examples, the invariants on
all five workloads (the prefill layer's count, plan, dispatch, pack and
relay trees included), the fuzz corpus, the relay and the combine and
reduction pins.  CPU only."""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "oracle", "oracle.c")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer", "-g", "-O1"]
ORACLE_TESTS = ["test_oracle_pins.py", "test_oracle_invariants.py",
                "test_oracle_relay.py", "test_oracle_combine_reduce.py"]


def _asan_runtime():
    path = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True, check=True).stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip("gcc has no AddressSanitizer runtime here")
    return path


@pytest.fixture(scope="module")
def san_build(tmp_path_factory):
    d = tmp_path_factory.mktemp("san")
    lib = str(d / "liboracle_san.so")
    bf = str(d / "bruteforce_san")
    subprocess.run(["gcc", "-std=c11", "-ffp-contract=off", *SAN, "-fPIC", "-shared",
                    "-o", lib, SRC], check=True)
    subprocess.run(["gcc", *SAN, "-o", bf, os.path.join(HERE, "native", "bruteforce.c")],
                   check=True)
    env = dict(os.environ)
    # the sanitizer runtime must come first; whatever the environment
    # already preloads stays after it
    pre = env.get("LD_PRELOAD")
    env["LD_PRELOAD"] = _asan_runtime() + (":" + pre if pre else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["ULTRAEP_ORACLE_LIB"] = lib
    return lib, bf, env


def _no_report(r):
    text = r.stdout + r.stderr
    assert "AddressSanitizer" not in text and "runtime error" not in text, text[-4000:]
    assert r.returncode == 0, text[-4000:]


def test_pin_harness_under_sanitizers(san_build):
    lib, bf, env = san_build
    r = subprocess.run([sys.executable, os.path.join(HERE, "mutation_runner.py"), lib, bf],
                       capture_output=True, text=True, env=env, timeout=600)
    _no_report(r)


def test_oracle_tests_under_sanitizers(san_build):
    lib, _, env = san_build
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "-m", "not gpu", *[os.path.join(HERE, t) for t in ORACLE_TESTS]],
                       capture_output=True, text=True, env=env, timeout=900, cwd=ROOT)
    _no_report(r)
    assert " passed" in r.stdout


def test_child_loads_the_sanitized_build(san_build):
    lib, _, env = san_build
    code = ("import sys; sys.path.insert(0, %r); import oracle; oracle.lib(); "
            "maps = open('/proc/self/maps').read(); "
            "print(oracle._LIB, 'liboracle_san' in maps, 'libasan' in maps)" % ROOT)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env)
    _no_report(r)
    assert r.stdout.split() == [lib, "True", "True"]
