"""The C ABI from a native program: paper_2609_36864_amd/abi_check (built by
the package's build step from csrc/tools/abi_check.cpp) allocates plain HIP
buffers, runs the re-scoring path through include/hdl.h alone and checks the
properties its results must have (log p <= 0 on scored rows and 0 on masked
ones; identical contexts give a zero divergence bit for bit and the first k
eligible positions; every root's branch points ordered by score then
position with score = |delta|; argument errors reported synchronously)."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2609_36864_amd",
                   "abi_check")


def test_native_abi_consumer():
    if not os.path.exists(EXE):
        pytest.fail(f"{EXE} is not built (python -m paper_2609_36864_amd.build)")
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi_check: ok" in r.stdout
