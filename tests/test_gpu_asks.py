"""Parity of the HIP ASKS similarity (rksc_asks_similarity) with the float64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_09937_amd as rk
import workloads
from gpu_util import SIM_ATOL, log

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("L,B,d,alpha", [
    (2, 4, 256, 0.5), (32, 16, 4096, 0.1), (48, 32, 4096, 0.1), (28, 8, 3584, 1.5), (1, 3, 7, -2.0),
    (5, 1, 64, 0.0),
])
def test_asks_matches_oracle(L, B, d, alpha):
    log(f"asks L={L} B={B} d={d} alpha={alpha}")
    h = workloads.make_hidden(L, B, d, seed=L + B, device=DEV, scale=3.0)
    if B >= 3:
        h[:, 2] = h[:, 0] * 0.25                     # same direction as branch 0
    S = rk.asks_similarity(h.contiguous(), alpha)
    torch.cuda.synchronize()
    got = S.cpu().numpy()
    ref = oracle.asks_similarity(h.cpu().numpy(), alpha)
    assert np.abs(got - ref).max() <= SIM_ATOL
    np.testing.assert_array_equal(got, got.T)
    if B >= 3:
        assert abs(got[0, 2] - 1.0) <= SIM_ATOL


def test_asks_zero_and_antipodal_rows():
    h = workloads.make_hidden(6, 4, 128, seed=1, device=DEV)
    h[:, 1] = -h[:, 0]
    h[:, 3] = 0.0
    S = rk.asks_similarity(h.contiguous(), 1.5).cpu().numpy()
    assert abs(S[0, 1] + 1.0) <= SIM_ATOL
    assert (S[3] == 0.0).all() and (S[:, 3] == 0.0).all()
    np.testing.assert_allclose(np.diag(S)[:3], 1.0, atol=SIM_ATOL)
