"""Seeded synthetic workloads shared by the oracle's tests and the GPU path's tests.

Holds no arithmetic of the method: shapes, random draws and layout only.
"""
from .configs import (WORKLOADS, BY_NAME, Workload, TINY, SINGLE, RAGGED, MIXED, STRESS,
                      SELECT_I8, EQ2, PAPER, PAPER_I8, scaled)
from .generate import (Inputs, SeqBatch, Weights, Layer, make_inputs, make_weights,
                       round_to_bf16, to_padded, subset_candidates, int8_codes, N_ACT, N_TIME,
                       TokenBatch, make_tokens)
