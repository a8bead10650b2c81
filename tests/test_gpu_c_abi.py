"""The library driven from plain C: tests/native/abi_c_step.c (built by
__graft_entry__.build() into paper_2609_39859_amd/_build/abi_c_step) runs
one step through fork_step with device buffers from the HIP runtime's C API
and checks the statistics and the fallback decision against closed forms."""
import os
import subprocess

import pytest

from paper_2609_39859_amd import build

pytestmark = pytest.mark.gpu


def test_one_step_from_plain_c():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    exe = build.C_EXAMPLE
    if not os.path.exists(exe):
        build.build_c_example()
    print("c abi: running %s" % exe, flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert "c step ok" in r.stdout
