"""CPU oracle (test infrastructure only; never used by the product path)."""
from .upr_oracle import (cache_index, cache_shape, encode, full_sequence, gelu_tanh,
                         layer_norm, linear, masked_softmax_attention, mfalcon_mask,
                         rank, score_head, unpack_weights)

__all__ = ["cache_index", "cache_shape", "encode", "full_sequence", "gelu_tanh",
           "layer_norm", "linear", "masked_softmax_attention", "mfalcon_mask",
           "rank", "score_head", "unpack_weights"]
