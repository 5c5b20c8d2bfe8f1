"""The C ABI from C++ alone (tests/c_abi/abi_check.cpp): plain device pointers
from hipMalloc and a HIP stream, no Python binding and no torch in the process.
The program samples, packs and assembles one group and checks, on the host,
what the header's contract fixes for any input: the frontier rule hop by hop,
each edge against the CSR graph, the fan-out counts and draw order, P_b, every
packed and assembled row, the address tables, U, the sizes, the membership
words left clear, and a null argument rejected; and the two calls the one call
stands for (dg_sample_group, then dg_pack_group) give the same outputs.  It is built by
__graft_entry__.build() (python tests/c_abi/build.py builds it alone)."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "abi_check")


def test_c_abi_program():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(EXE):
        pytest.skip("tests/c_abi/abi_check is not built (run __graft_entry__.build())")
    print("[c abi] running tests/c_abi/abi_check", flush=True)
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "C ABI check ok" in r.stdout
