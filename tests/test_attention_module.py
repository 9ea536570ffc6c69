"""The PyTorch drop-in rejects bad inputs before any library call (CPU)."""
import pytest
import torch

from paper_2605_12193_amd.attention import BlockFilteredAttention, _layout


def _t(*shape, dtype=torch.bfloat16):
    return torch.zeros(*shape, dtype=dtype)


@pytest.mark.parametrize("q,k,msg", [
    (_t(2, 4, 8, 64), _t(2, 2, 8, 64), "on the GPU"),
    (_t(2, 4, 8, 64, dtype=torch.float16), _t(2, 2, 8, 64), "bfloat16"),
    (_t(4, 8, 64), _t(2, 2, 8, 64), "expected q"),
])
def test_rejects_bad_inputs(q, k, msg):
    with pytest.raises(ValueError, match=msg):
        BlockFilteredAttention()(q, k, k)


def test_shape_rules():
    # _layout's shape checks run after the device check; call it on meta tensors
    q = torch.empty(2, 6, 8, 64, dtype=torch.bfloat16, device="meta")
    k = torch.empty(2, 4, 8, 64, dtype=torch.bfloat16, device="meta")
    with pytest.raises(ValueError):
        _layout(q, k, k)   # meta tensors are not on the GPU
