"""The allocation-free decode entry point (hack_attend_decode_noalloc) against
hack_attend_decode on the same inputs: the two share their kernels, so the outputs
must be identical, on two calls in a row (the second with a smaller batch and
shorter contexts, so the static scratch keeps the first call's records)."""
import numpy as np
import pytest
import torch

from oracle import hack_oracle as O

pytestmark = pytest.mark.gpu
TOL = 2e-3


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util
    return gpu_util


@pytest.mark.parametrize("bits,pi,group,first,second", [
    (2, 32, 4, [4096, 3000, 17, 2222, 4000, 1], [1000, 5, 999]),
    (4, 64, 8, [3000, 2048, 700], [300, 64]),
    (2, 128, 4, [4096, 2500, 9], [1024, 129]),
])
def test_noalloc_matches_workspace_call_twice(bits, pi, group, first, second):
    gu = _gpu()
    from paper_2502_03589_amd import hack as hk
    for i, lens in enumerate((first, second)):
        gu.announce(f"noalloc call {i}: bits={bits} pi={pi} G={group} lens={lens}")
        case = gu.Case(700 + 10 * i + bits + pi, len(lens), 2, lens, bits, pi, group=group).quantize()
        q = torch.from_numpy(case.q).to(gu.DEV)
        got = hk.hack_attend_decode_noalloc(case.layout, case.cache, q, case.lens_dev, case.max_len)
        want = hk.hack_attend_decode(case.layout, case.cache, q, case.lens_dev, case.max_len)
        torch.cuda.synchronize()
        assert torch.equal(got, want), f"call {i}"
        err = gu.rel_err(got.cpu().numpy(), O.attend_decode(case.q, case.oracle_seqs(), case.H))
        print(f"call {i}: max|d|/|O|inf vs the oracle = {err:.3e}")
        assert err <= TOL
