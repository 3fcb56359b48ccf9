"""Host-side checks of the C ABI that need no GPU: the library loads and
exports every function include/pccl.h declares, and the Python binding
names them one for one."""

import ctypes
import os
import re
import subprocess

import pytest

from paper_2606_07019_amd import build as B
from paper_2606_07019_amd import pccl as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared():
    text = open(os.path.join(ROOT, "include", "pccl.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pccl_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB):
        B.build()
    return P.load_library()


def test_header_declares_the_documented_calls():
    names = declared()
    for n in ["pccl_create", "pccl_destroy", "pccl_load_topology", "pccl_set_collective",
              "pccl_set_switch_model",
              "pccl_workspace_bytes", "pccl_set_workspace", "pccl_synthesize",
              "pccl_get_schedule", "pccl_get_stats", "pccl_get_setup", "pccl_get_profile",
              "pccl_last_error"]:
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.check_output(["nm", "-D", "--defined-only", B.LIB], text=True)
    exported = set(line.split()[-1] for line in out.splitlines() if " T " in line)
    for n in declared():
        assert n in exported, n
        assert hasattr(lib, n)


def test_binding_has_the_same_names(lib):
    for n in declared():
        assert callable(getattr(P, n)), n


def test_pccl_send_layout():
    assert ctypes.sizeof(P.pccl_send) == 16


def test_null_arguments_are_rejected(lib):
    assert lib.pccl_create(None, 0, 0) == 1            # PCCL_EINVAL
    assert lib.pccl_synthesize(None, None, None) == 1
    assert lib.pccl_last_error(None) == b"null context"
