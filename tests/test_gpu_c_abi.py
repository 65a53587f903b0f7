"""The C ABI from a C++ program with no Python or torch (tests/c_abi/
kq_abi_client.cpp): HIP runtime buffers, kq_pack_factors, kq_quantize_packed,
kq_quantize and kq_quantize_exact on one stream, checked in the program against
the C oracle (scales identical, codes within tie flips, y within 1e-5; the
fixed-order path bit for bit) and a refused bad size."""
import os
import subprocess

import pytest

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "kq_abi_client")


@pytest.mark.gpu
def test_c_abi_client_matches_oracle():
    assert os.path.exists(BIN), "tests/c_abi/kq_abi_client is not built: run __graft_entry__.build()"
    res = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    print(res.stdout, res.stderr)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.startswith("c_abi ok:"), res.stdout
