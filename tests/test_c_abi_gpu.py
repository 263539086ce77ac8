"""The C consumer of the ABI on the GPU (tests/c_abi/kashin_abi_check.c): plain device pointers
from the HIP runtime, no Python binding.  Decomposes a few rows and checks w = u + P vhat + r
through kashin_apply_p (fp32 rounding), then quantises and reconstructs them."""
import subprocess
import sys

import pytest

from test_abi_host import _abi_check_binary


@pytest.mark.gpu
def test_c_program_uses_the_abi_on_the_gpu():
    print("C ABI check, gpu mode", flush=True)
    sys.stdout.flush()
    res = subprocess.run([_abi_check_binary(), "gpu"], capture_output=True, text=True, timeout=120)
    print(res.stdout, flush=True)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.strip().endswith("ok")
