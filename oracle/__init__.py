"""CPU oracle (test infrastructure only; never imported by the product path).

Only tests, the smoke check and the benchmark's CPU-baseline leg use it.
"""
from .lstm import (bf16_round, sigmoid, lstm_forward_literal, lstm_forward,
                   lstm_backward, stacked_forward, stacked_backward,
                   matmul_chain_grad)

__all__ = ["bf16_round", "sigmoid", "lstm_forward_literal", "lstm_forward",
           "lstm_backward", "stacked_forward", "stacked_backward",
           "matmul_chain_grad"]
