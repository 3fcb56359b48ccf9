"""The CPU checkers under AddressSanitizer and UndefinedBehaviorSanitizer.

The oracle and the condition-sequential Alg. 3 reference are rebuilt with
-fsanitize=address,undefined (PCCL_ORACLE_SANITIZE=1 makes oracle/ load those
copies) and a subset of their pins runs in a child process that preloads
libasan, so that an out-of-bounds access, a use after free, a leak-free
double free or undefined integer behaviour in the C code fails this test.
The whole CPU suite runs the same way with

    PCCL_ORACLE_SANITIZE=1 LD_PRELOAD=$(gcc -print-file-name=libasan.so) \
        ASAN_OPTIONS=detect_leaks=0 python -m pytest tests -m "not gpu"
"""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SUBSET = [
    "tests/test_oracle_pins.py::test_config1_exact",
    "tests/test_oracle_pins.py::test_parent_tie_smallest_device_id",
    "tests/test_oracle_pins.py::test_rail_cluster_routes_uplink_first_small",
    "tests/test_oracle_pins.py::test_invariants_fuzz",
    "tests/test_oracle_pins.py::test_errors",
    "tests/test_oracle_pins.py::test_empty_and_trivial_collectives",
    "tests/test_oracle_pins.py::test_allreduce_is_reversed_then_forward",
    "tests/test_oracle_pins.py::test_plain_and_idle_skip_modes_agree",
    "tests/test_switch_model.py",
    "tests/test_alg3_reference.py",
]


def _libasan():
    try:
        p = subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return p if os.path.isabs(p) and os.path.exists(p) else None


def test_oracle_pins_clean_under_asan_and_ubsan():
    asan = _libasan()
    if asan is None:
        pytest.skip("gcc has no libasan")
    env = dict(os.environ)
    env.update({
        "PCCL_ORACLE_SANITIZE": "1",
        "LD_PRELOAD": asan,
        # Python itself is not instrumented: its allocations are not leaks of the oracle
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
    })
    # build the sanitized copies first, in this process's view of the tree
    build = ("import os, sys; sys.path.insert(0, os.getcwd()); "
             "from oracle import oracle, alg3; oracle.build(force=True); alg3.build(force=True)")
    subprocess.run([sys.executable, "-c", build], cwd=ROOT, env=env, check=True, timeout=300)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider"] + SUBSET,
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    for marker in ("ERROR: AddressSanitizer", "runtime error:", "ERROR: LeakSanitizer"):
        assert marker not in out, out[-4000:]
