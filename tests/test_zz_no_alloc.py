"""spec_verify_noalloc (the library's own scratch array, no workspace)
against spec_verify on the same inputs through the C ABI: two calls in a row,
the second with a smaller input, outputs identical bit for bit; a shape
beyond the scratch array is refused."""

import numpy as np
import pytest
import torch

from paper_2606_12370_amd import binding
from paper_2606_12370_amd import workloads as W
from tests.parity import device_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    binding.load_library()
    yield
    torch.cuda.synchronize()


def _inputs(B, K, V, dtype, seed):
    d = W.verify_inputs_numpy(B, K, V, dtype, "rollout_t", seed)
    tgt, drf = device_inputs(d)
    return tgt, drf, torch.from_numpy(d["ids"]).cuda(), torch.from_numpy(d["temperature"]).cuda()


@pytest.mark.parametrize("dtype", [W.BF16, W.F32])
def test_noalloc_matches_workspace_entry_point_twice(dtype):
    for B, K, V, seed in ((48, 3, 151936, 5), (7, 2, 40000, 6)):  # the second call smaller
        tgt, drf, ids, T = _inputs(B, K, V, dtype, seed)
        ref = binding.verify(tgt, drf, ids, T, 11, 3, want_debug=True)
        got = binding.verify(tgt, drf, ids, T, 11, 3, want_debug=True, noalloc=True)
        torch.cuda.synchronize()
        assert set(got) == set(ref)
        for key in ref:
            assert torch.equal(torch.nan_to_num(got[key], nan=-7.0), torch.nan_to_num(ref[key], nan=-7.0)), (B, key)
        assert int(got["accept_len"].min()) >= 0


def test_noalloc_refuses_a_shape_beyond_its_scratch():
    lib = binding.load_library()
    cap = int(lib.spec_verify_noalloc_max_workspace())
    assert cap == 32 << 20
    B, K, V = 4096, 8, 262144
    assert int(lib.spec_verify_workspace_size(B, K, V, 1)) > cap
    tgt = torch.empty((1, 1, 16), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(binding.SpecError) as e:
        lib_ret = lib.spec_verify_noalloc(binding._ptr(tgt), 0, 0, binding._ptr(tgt), 0, 0, 1, B, K, V,
                                          binding._ptr(tgt), None, 1.0, 0, 0, binding._ptr(tgt), binding._ptr(tgt),
                                          None, None, None, None, None, None)
        if lib_ret != 0:
            raise binding.SpecError("spec_verify_noalloc", lib_ret)
    assert "SPEC_EWORKSPACE" in str(e.value)
