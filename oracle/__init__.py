"""CPU oracle (test infrastructure only; see mzoracle's header)."""
from .mzoracle import *  # noqa: F401,F403
from .mzoracle import (Hyper, Weights, OracleContext, q4_0_decode, rmsnorm, rope, silu,
                       causal_gqa_attention, clean_prefill, restore_rows, argmax_first,
                       layer_forward, output_logits, RES, SWAP, DROP)  # noqa: F401
