"""CPU oracle for TransAct V2's lifelong-sequence NN-select + encode path.

TEST INFRASTRUCTURE ONLY.  This package is the slow, plain, obviously correct
statement of what the GPU path computes, written from the paper: the
candidate-anchored nearest-neighbour search of Eq. 3 (Sec. 3.2.2), the token
set of Eq. 2 (lifelong, real-time and impression sources; rows stored as the
int8 codes of Sec. 3.2.1 enter the encoder dequantised), the feature
encoding with early fusion of Eq. 4, the causal transformer encoder and the
linear + max-pool head (Sec. 3.2.2, 'Transformer Encoder').  Only the tests,
the package's smoke check and the benchmark's CPU-baseline leg may import it;
the GPU library never does, and this package imports nothing from it.

Arithmetic: scores are exact (integer arithmetic on the inputs' dyadic grid);
the encoder runs in float64 on the same (bf16-rounded where applicable) values
the GPU receives.

Pins (tests/test_oracle_*.py): brute-force exact sort of tiny score vectors,
selection invariants, the encoder against torch's own post-LN
TransformerEncoderLayer in float64, the single-token closed form, causal prefix
invariance, head-permutation invariance and the Eq. 4 special case.
"""
from .nn_select import (exact_scores, nn_select, nn_select_batch, token_positions, gather_tokens,
                        normalised_scores, nn_select_i8, eq2_tokens, dequantise)
from .encoder import (feature_encode, encoder_layer, pool, encode, encode_states, select_encode,
                      select_encode_eq2)

__all__ = ["exact_scores", "nn_select", "nn_select_batch", "token_positions", "gather_tokens",
           "normalised_scores", "nn_select_i8", "eq2_tokens", "dequantise",
           "feature_encode", "encoder_layer", "pool", "encode", "encode_states",
           "select_encode", "select_encode_eq2"]
