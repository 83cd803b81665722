"""tav2_select_encode captured into a HIP graph (the paper's serving engine
replays its GPU work as graphs, Sec. 3.4.2): the library issues only kernel
launches on the caller's stream (no allocation, no memset, no synchronisation),
so one call captures whole.  Every replay, with eager work and synchronisations
between replays, must give the eager call's outputs bit for bit."""
import numpy as np
import pytest
import torch

import synth
from helpers import upload
from paper_2506_02267_amd import tav2 as T

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("k", [64, 256])   # one encoder block; two blocks (cached keys)
def test_select_encode_graph_replays_match_eager(k):
    w = synth.scaled(synth.SINGLE, L=3000, N=70, k=k)
    inp = synth.make_inputs(w, seed=31)
    print(f"graph capture L={w.L} N={w.N} k={k}", flush=True)
    seq, rt, cands = upload(inp)
    call = T.SelectEncode(seq, rt, cands, w.k, T.DeviceWeights(synth.make_weights(w)))
    call()                                   # eager (also sets per-device kernel attributes)
    torch.cuda.synchronize()
    want = [t.clone() for t in (call.idx, call.score, call.out)]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (call.idx, call.score, call.out):
            t.fill_(-7)                      # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for got, ref in zip((call.idx, call.score, call.out), want):
            assert torch.equal(got, ref), f"replay {rep}"
    call()                                   # eager again after the replays
    torch.cuda.synchronize()
    for got, ref in zip((call.idx, call.score, call.out), want):
        assert torch.equal(got, ref)
