"""GPU parity of tav2_nn_select over int8 sequence codes, whose rows are
dequantised and L2-normalised inside the score kernel (Sec. 3.4.2, fused
sequence dequantisation), against the oracle: indices and scores bit for bit
(the dot products and sums of squares are exact, the square root and the
division rounded to nearest on both sides).  Cases: the 16k-row single-request
workload with all of its candidates (the launch the benchmark times), ragged
batches over several candidate tiles with ragged tails, k past the row count,
the narrowest and widest embeddings, all-zero and duplicated rows."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_select_equal, upload
from paper_2506_02267_amd import tav2 as T

pytestmark = pytest.mark.gpu


def check(w, seed=None, zero_every=0):
    inp = synth.make_inputs(w, seed=seed)
    if zero_every:
        inp.seq.emb[::zero_every] = 0
    print(f"select_i8 R={w.R} L={w.L or w.L_range} d={w.d} N={w.N} k={w.k}", flush=True)
    seq, _, cands = upload(inp)
    assert seq.emb.dtype == torch.int8 and cands.emb.dtype == torch.bfloat16
    idx, score = T.nn_select(seq, cands, w.k)
    torch.cuda.synchronize()
    ref_i, ref_s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, w.k)
    assert_select_equal(idx, score, ref_i, ref_s)


def test_full_size_all_candidates():
    check(synth.SELECT_I8, zero_every=1021)


def test_several_long_requests_large_k():
    """Four 16k-row requests with 2000 candidates each and k = 512."""
    w = synth.scaled(synth.SELECT_I8, R=4, N=2000, k=512)
    check(w, seed=25, zero_every=2003)


@pytest.mark.parametrize("d,R,Lr,N,k,seed", [
    (32, 3, (1, 700), 130, 64, 21),       # 2 candidate tiles, ragged tails, short rows
    (256, 2, (300, 2100), 40, 256, 22),   # wide codes, k above some row counts
    (16, 2, (37, 37), 1, 100, 23),        # narrowest rows, k > L (padding)
    (512, 1, (5000, 5000), 9, 33, 24),    # widest rows, long-row top-k
])
def test_ragged_batches(d, R, Lr, N, k, seed):
    w = synth.scaled(synth.SELECT_I8, R=R, L=None, L_range=Lr, d=d, N=N, k=k, tie_frac=0.05)
    check(w, seed=seed, zero_every=13)
