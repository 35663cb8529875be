"""CPU oracle (test infrastructure only; never imported by the product path).

Only tests, the smoke check and the benchmark's CPU-baseline leg use it.
"""
from .lstm import (bf16_round, sigmoid, lstm_forward_literal, lstm_forward,
                   lstm_backward, stacked_forward, stacked_backward,
                   matmul_chain_grad)
from .rnn import (rnn_forward_literal, rnn_forward, rnn_backward,
                  stacked_rnn_forward, stacked_rnn_backward)
from .gru import (gru_forward_literal, gru_forward, gru_backward,
                  stacked_gru_forward, stacked_gru_backward)
from .skip import (skip_forward_literal, skip_forward, skip_backward,
                   stacked_skip_forward, stacked_skip_backward)
from .act import (act_forward_literal, act_forward, act_backward,
                  stacked_act_forward, stacked_act_backward, ACT_EPS)

__all__ = ["bf16_round", "sigmoid", "lstm_forward_literal", "lstm_forward",
           "lstm_backward", "stacked_forward", "stacked_backward",
           "matmul_chain_grad", "rnn_forward_literal", "rnn_forward", "rnn_backward",
           "stacked_rnn_forward", "stacked_rnn_backward", "gru_forward_literal",
           "gru_forward", "gru_backward", "stacked_gru_forward", "stacked_gru_backward",
           "skip_forward_literal", "skip_forward", "skip_backward", "stacked_skip_forward",
           "stacked_skip_backward", "act_forward_literal", "act_forward", "act_backward",
           "stacked_act_forward", "stacked_act_backward", "ACT_EPS"]
