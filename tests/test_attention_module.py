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


def test_v_with_other_strides_than_k_is_rejected():
    # K a transposed view, V contiguous: same shape, different strides; the
    # library would read V with K's strides, so the module refuses
    q = _t(2, 4, 8, 64)
    k = _t(2, 8, 2, 64).transpose(1, 2)
    v = _t(2, 2, 8, 64)
    assert k.shape == v.shape and k.stride() != v.stride()
    with pytest.raises(ValueError, match="strides"):
        BlockFilteredAttention()(q, k, v)


def test_kv_descriptor_checks():
    from paper_2605_12193_amd import bfla
    k = _t(2, 8, 64)
    with pytest.raises(ValueError, match="same shape and strides"):
        bfla.KV(k, _t(8, 2, 64).transpose(0, 1))
    pages = _t(4, 16, 2, 64)
    for table in (torch.zeros(1, 4, dtype=torch.int64),
                  torch.zeros(4, 2, dtype=torch.int32).t(),
                  None):
        with pytest.raises(ValueError, match="block_table"):
            bfla.KV(pages, pages, paged=True, block_table=table)


def test_varlen_length_rules():
    from paper_2605_12193_amd.attention import _host_ints, _lengths
    assert _lengths([0, 3, 10], 10, "cu") == [3, 7]
    assert _host_ints(torch.tensor([0, 5]), "cu") == [0, 5]
    for cu, total in (([1, 3], 3), ([0, 3], 4), ([0, 3, 3], 3), ([0], 0)):
        with pytest.raises(ValueError, match="cu"):
            _lengths(cu, total, "cu")


def test_varlen_and_paged_reject_host_tensors():
    q = _t(10, 4, 64)
    with pytest.raises(ValueError, match="GPU tensor"):
        BlockFilteredAttention().forward_varlen(q, _t(10, 2, 64), _t(10, 2, 64), [0, 10], [0, 10])
    with pytest.raises(ValueError, match="GPU tensor"):
        BlockFilteredAttention().forward_paged(q, _t(4, 16, 2, 64), _t(4, 16, 2, 64),
                                               torch.zeros(1, 4, dtype=torch.int32), [10], [0, 10])
