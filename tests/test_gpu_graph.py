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


CASES = {
    # d_model 256: one encoder block; two blocks (cached keys)
    "single_k64": dict(base=synth.SINGLE, L=3000, N=70, k=64),
    "single_k256": dict(base=synth.SINGLE, L=3000, N=70, k=256),
    # the paper's encoder shape (d_model 64) behind the fused search (rows > 4096),
    # with a real-time tail: three 64-position blocks
    "paper": dict(base=synth.PAPER, L=6000, N=40),
    # fp32 (the LDS-resident fp32 encoder)
    "tiny_f32": dict(base=synth.TINY, L=900, N=12),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_select_encode_graph_replays_match_eager(case):
    kw = dict(CASES[case])
    w = synth.scaled(kw.pop("base"), **kw)
    inp = synth.make_inputs(w, seed=31)
    print(f"graph capture {case}: L={w.L} N={w.N} k={w.k} T={w.T}", flush=True)
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
