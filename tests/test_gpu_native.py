"""The C ABI from a native program: tests/native/abi_roundtrip.cpp encodes
four 1,000,003-value shards, decodes them from one buffer and checks the
values and both sides' caches on its own, with no Python or torch in the
process. Built by __graft_entry__.build()."""
import os
import subprocess

import pytest

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native",
                   "abi_roundtrip")


def test_native_binary_links():
    """Built, and every shared library it needs resolves (no GPU needed)."""
    assert os.path.exists(EXE), "run __graft_entry__.build() first"
    out = subprocess.run(["ldd", EXE], capture_output=True, text=True,
                         check=True).stdout
    assert "libciera.so" in out and "not found" not in out, out


@pytest.mark.gpu
def test_native_roundtrip():
    assert os.path.exists(EXE), "run __graft_entry__.build() first"
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "round trip exact" in r.stdout, r.stdout
