"""CPU oracle (test infrastructure only; never used by the product path)."""
from .upr_oracle import (cache_index, cache_shape, encode, full_sequence, gelu_tanh,
                         layer_norm, linear, masked_softmax_attention, mfalcon_mask,
                         rank, rank_hidden, score_head, unpack_weights)
from .upr_heads import (action_logits, heads_blob_size, sigmoid, topk_by_utility,
                        unpack_heads, utility)
from .upr_mx import (e4m3_round_codes, e4m3_value, linear_mx, mx_block_exponent,
                     mx_dequantize, mx_quantize, mx_round)

__all__ = ["cache_index", "cache_shape", "encode", "full_sequence", "gelu_tanh",
           "layer_norm", "linear", "masked_softmax_attention", "mfalcon_mask",
           "rank", "rank_hidden", "score_head", "unpack_weights",
           "action_logits", "heads_blob_size", "sigmoid", "topk_by_utility", "unpack_heads",
           "utility", "e4m3_round_codes", "e4m3_value", "linear_mx",
           "mx_block_exponent", "mx_dequantize", "mx_quantize", "mx_round"]
