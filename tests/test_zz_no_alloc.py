"""tav2_nn_select_noalloc (the NN search on the library's static scratch, for
callers that cannot allocate) against tav2_nn_select with a caller workspace:
indices and scores bit for bit on two calls in a row (the second smaller), on
the on-chip-score search for long rows and on the materialised score rows for
short ones, and against the oracle; a request too large for the scratch is
refused before anything runs."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_select_equal, upload
from paper_2506_02267_amd import tav2 as T

pytestmark = pytest.mark.gpu


def both(inp, k):
    seq, _, cands = upload(inp)
    ref_i, ref_s = T.nn_select(seq, cands, k)
    idx = torch.full((cands.total, k), 7, dtype=torch.int32, device="cuda")
    score = torch.full((cands.total, k), 7.0, dtype=torch.float32, device="cuda")
    T.nn_select_noalloc(seq, cands, k, idx, score)
    torch.cuda.synchronize()
    assert torch.equal(idx, ref_i)
    assert torch.equal(score.view(torch.int32), ref_s.view(torch.int32))
    return idx, score


@pytest.mark.parametrize("dtype", ["bf16", "i8"])
def test_two_calls_in_a_row_second_smaller(dtype):
    base = synth.SINGLE if dtype == "bf16" else synth.SELECT_I8
    big = synth.scaled(base, R=2, L=16384, N=300, k=256)
    small = synth.scaled(base, R=1, L=9000, N=40, k=64)
    print(f"no-alloc {dtype}: {big.R}x{big.N} at L={big.L}, then {small.R}x{small.N} at "
          f"L={small.L}", flush=True)
    inp1 = synth.make_inputs(big, seed=61)
    i1, s1 = both(inp1, big.k)
    inp2 = synth.make_inputs(small, seed=62)
    i2, s2 = both(inp2, small.k)
    ref_i, ref_s = oracle.nn_select_batch(inp2.seq, inp2.cand, inp2.cand_offset, small.k)
    assert_select_equal(i2, s2, ref_i, ref_s)


def test_short_rows_materialised_path():
    w = synth.scaled(synth.RAGGED, R=3, L_range=(500, 4000), N=64, k=128)
    inp = synth.make_inputs(w, seed=63)
    print("no-alloc short rows", flush=True)
    i, s = both(inp, w.k)
    ref_i, ref_s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, w.k)
    assert_select_equal(i, s, ref_i, ref_s)


def test_too_large_for_the_scratch_is_refused():
    lib = T.load_library()
    assert lib.tav2_scratch_bytes() == 64 << 20
    w = synth.scaled(synth.SINGLE, R=1, L=16384, N=8, k=1024)
    inp = synth.make_inputs(w, seed=64)
    seq, _, cands = upload(inp)
    c = cands.struct()
    c.total, c.max_count = 40000, 40000   # host-side sizing only: refused before any launch
    st = lib.tav2_nn_select_noalloc(ctypes.byref(seq.struct()), ctypes.byref(c), 1024,
                                    ctypes.c_void_p(0x10000), ctypes.c_void_p(0x10000), None)
    assert st == -7
