"""The stable embedding layer of Section 3.3, for use with the 8-bit optimizers.

A word embedding initialized with Xavier-uniform values whose output goes
through a layer norm (add position embeddings after it).  Its weight carries
the attribute ``bq_32bit_state = True``, which makes every 8-bit optimizer of
``paper_2110_02861_amd.optim`` keep that weight's optimizer states in 32 bit
(the paper keeps only this layer's states in 32 bit); the weight and its
gradient keep their own dtype.
"""
from __future__ import annotations

import torch
import torch.nn.functional as F


class StableEmbedding(torch.nn.Embedding):
    def __init__(self, num_embeddings: int, embedding_dim: int, padding_idx=None,
                 max_norm=None, norm_type: float = 2.0, scale_grad_by_freq: bool = False,
                 sparse: bool = False, device=None, dtype=None):
        if sparse:
            raise ValueError("the 8-bit optimizers take dense gradients only")
        super().__init__(num_embeddings, embedding_dim, padding_idx, max_norm, norm_type,
                         scale_grad_by_freq, sparse=False, device=device, dtype=dtype)
        self.norm = torch.nn.LayerNorm(embedding_dim, device=device, dtype=dtype)
        self.weight.bq_32bit_state = True

    def reset_parameters(self) -> None:
        torch.nn.init.xavier_uniform_(self.weight)
        self._fill_padding_idx_with_zero()

    def forward(self, input: torch.Tensor) -> torch.Tensor:
        emb = F.embedding(input, self.weight, self.padding_idx, self.max_norm, self.norm_type,
                          self.scale_grad_by_freq, self.sparse)
        return self.norm(emb)
