"""fp64 CPU oracle for the Kraken prefill (test infrastructure only; see kraken_oracle)."""

from .kraken_oracle import (LN_EPS, PARAM_NAMES, causal_attention, feed_forward, gelu,
                            kraken_param_count, kraken_prefill, layer_norm,
                            multi_head_attention, sub_layer_forward)

__all__ = ["LN_EPS", "PARAM_NAMES", "causal_attention", "feed_forward", "gelu",
           "kraken_param_count", "kraken_prefill", "layer_norm", "multi_head_attention",
           "sub_layer_forward"]
