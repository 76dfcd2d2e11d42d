"""The stable embedding layer (Section 3.3) on the CPU: Xavier-uniform init, a
layer norm on the output, and the flag that gives its weight 32-bit states."""
from __future__ import annotations

import math

import pytest
import torch

from paper_2110_02861_amd import nn, optim


def test_init_is_xavier_uniform_and_flagged():
    torch.manual_seed(0)
    emb = nn.StableEmbedding(5000, 256)
    bound = math.sqrt(6.0 / (5000 + 256))
    w = emb.weight.detach()
    assert float(w.abs().max()) <= bound
    # a uniform distribution on [-bound, bound] has variance bound^2 / 3
    assert abs(float(w.var()) / (bound ** 2 / 3) - 1.0) < 0.02
    assert emb.weight.bq_32bit_state is True


def test_output_is_layer_normed():
    torch.manual_seed(1)
    emb = nn.StableEmbedding(100, 64, padding_idx=0)
    assert torch.all(emb.weight.detach()[0] == 0)
    y = emb(torch.randint(1, 100, (8, 12)))  # not the padding index (its row is 0)
    assert y.shape == (8, 12, 64)
    assert torch.allclose(y.mean(-1), torch.zeros(8, 12), atol=1e-5)
    # unit variance up to the norm's eps (1e-5) against row variances near 0.01
    assert torch.allclose(y.var(-1, unbiased=False), torch.ones(8, 12), atol=2e-3)
    y.sum().backward()
    assert emb.weight.grad is not None and not emb.weight.grad.is_sparse


def test_optimizers_keep_its_weight_in_32_bit():
    emb = nn.StableEmbedding(10, 4)
    lin = torch.nn.Linear(4, 4)
    opt = optim.Adam8bit(list(emb.parameters()) + list(lin.parameters()))
    assert not opt._is_8bit(emb.weight)
    assert opt._is_8bit(lin.weight)
    with pytest.raises(ValueError):
        nn.StableEmbedding(10, 4, sparse=True)
