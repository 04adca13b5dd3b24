"""The CE / KL gradient comparison: rows below float32's range are measured
against a floor; rows within it stay norm-wise relative."""

import numpy as np
import pytest
import torch

from paper_2606_12370_amd import workloads as W
from tests.parity import KL_GRAD_FLOOR, TOL, compare_kl


def _ref(gr):
    return {"grad": gr}


def test_row_below_float32_range_compares_against_the_floor():
    gr = np.zeros((2, 1, 8))
    gr[0, 0, :3] = [1e-37, -6e-38, -4e-38]  # the draft's exponentials underflow in float32
    gr[1, 0, :2] = [0.25, -0.25]
    g = gr.copy()
    g[0, 0, :3] = 0.0
    rep = compare_kl(None, None, torch.tensor(g, dtype=torch.float32), _ref(gr), W.F32, loss_exact=False)
    assert rep["max_normwise_grad"] == pytest.approx(1e-37 / KL_GRAD_FLOOR)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_rows_within_range_stay_relative(dtype):
    gr = np.zeros((2, 1, 8))
    gr[0, 0, :2] = [3e-20, -3e-20]  # small but within float32's range: relative as before
    gr[1, 0, :2] = [0.25, -0.25]
    g = gr.copy()
    g[0, 0, 0] *= 1.0 + 2.0 * TOL[dtype]
    with pytest.raises(AssertionError):
        compare_kl(None, None, torch.tensor(g, dtype=torch.float32), _ref(gr), dtype, loss_exact=False)
    g = gr.copy()
    g[1, 0, 1] *= 1.0 + 2.0 * TOL[dtype]
    with pytest.raises(AssertionError):
        compare_kl(None, None, torch.tensor(g, dtype=torch.float32), _ref(gr), dtype, loss_exact=False)
