"""Fuzz parity: about 200 seeded random call shapes spread over every kernel
of the library (the implicit-GEMM kernel at every tile width, the head, both
1x1 kernels at temporal strides 1-3, fp32, split-K with a workspace, single
temporal taps, forced and unsupported fallbacks), each compared in full with
the oracle on NaN-filled outputs inside NaN guard bands; the cache bit-exact.
The cases and the kernel each one reaches are in fuzz_cases.py (checked on
the CPU by test_fuzz_cases.py)."""
import pytest

from paper_2609_31938_amd import c3c

from fuzz_cases import cases
from test_gpu_parity import _case

pytestmark = pytest.mark.gpu

CASES = cases()


@pytest.mark.parametrize("i", range(len(CASES)))
def test_fuzz(i):
    dtype, sp, kernel, mode, ws = CASES[i]
    ctx, _, m = _case(sp, dtype, mode, seed=1000 + i, ws=ws, kernel=kernel)
    c = ctx.counters()
    assert c["calls"] == 1 and c["failed"] == c["fast_error"] == 0
    assert c["fast"] == (0 if mode & c3c.MODE_FORCE_FALLBACK or kernel == "fallback_direct" else 1)
