"""Python binding checks that need no GPU: host tensors are refused before any
library call (the kernels would dereference their addresses on the GPU)."""
import pytest
import torch

import paper_2603_18815_amd as ra


def test_host_pools_are_refused():
    k = torch.zeros((4, 2, 16, 128), dtype=torch.bfloat16)
    v = torch.zeros((4, 2, 128, 16), dtype=torch.bfloat16)
    bt = torch.zeros((1, 4), dtype=torch.int32)
    with pytest.raises(ValueError, match="GPU tensor"):
        ra.PagedKV(k, v, bt)


def test_host_logprob_inputs_are_refused():
    h = torch.zeros((2, 64), dtype=torch.bfloat16)
    W = torch.zeros((10, 64), dtype=torch.bfloat16)
    t = torch.zeros((2,), dtype=torch.int32)
    with pytest.raises(ValueError, match="GPU tensor"):
        ra.token_logprob(h, W, t)
    with pytest.raises(ValueError, match="GPU tensor"):
        ra.token_logprob_pack_weight(W)
