"""GPU parity of the gather and encoder (Eq. 2 order, Eq. 4, causal encoder,
linear + max-pool head) against the oracle: tokens bit for bit, pooled outputs
within max-abs 1e-4 (fp32) / 2e-2 (bf16)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import (BF16_TOL, F32_TOL, assert_select_equal, max_abs, oracle_select_encode,
                     strided_ids, upload)
from paper_2506_02267_amd import tav2 as T

pytestmark = pytest.mark.gpu


def run_path(inp, W, flags=T.MASK_CAUSAL, pack=False):
    seq, rt, cands = upload(inp)
    dw = T.DeviceWeights(W, pack=pack)
    idx, score, out = T.select_encode(seq, rt, cands, inp.w.k, dw, flags=flags)
    torch.cuda.synchronize()
    return idx, score, out


def check_workload(w, ids=None, W=None, inp=None, gpu=None, flags=T.MASK_CAUSAL):
    """The whole path against the oracle on the candidates in ids (all by default);
    gpu: outputs of an earlier run of the same inputs, reused."""
    inp = inp if inp is not None else synth.make_inputs(w)
    W = W if W is not None else synth.make_weights(w)
    n_ids = inp.total if ids is None else len(ids)
    print(f"select_encode workload {w.name} R={w.R} N={w.N} T={w.T}: {n_ids} of {inp.total} "
          f"candidates, flags {flags}", flush=True)
    idx, score, out = gpu if gpu is not None else run_path(inp, W, flags)
    ref_i, ref_s, ref_out = oracle_select_encode(inp, W, w.k, ids=ids,
                                                 causal=flags == T.MASK_CAUSAL)
    assert_select_equal(idx, score, ref_i, ref_s, ids=ids)
    err = max_abs(out, ref_out, ids=ids)
    tol = F32_TOL if w.dtype == "f32" else BF16_TOL
    print(f"  max abs error {err:.3e} (bound {tol})", flush=True)
    assert err <= tol
    return err


def test_tiny_fp32_all_candidates():
    check_workload(synth.TINY)


@pytest.mark.parametrize("shape,flags", [
    # the whole fp32 envelope: T 64, d_model 128, FFN 512 (four hidden chunks), d 256
    (dict(d=256, d_model=128, n_heads=4, d_ffn=512, n_layers=2, k=64, has_time=True),
     T.MASK_CAUSAL),
    # 3 heads of 32, FFN 200 (a partial hidden chunk), a 48-wide embedding
    (dict(d=48, d_model=96, n_heads=3, d_ffn=200, n_layers=1, k=40, has_time=False),
     T.MASK_CAUSAL),
    # one head of 128, three layers, T = 61 (keys padded to 64 in the P V product)
    (dict(d=256, d_model=128, n_heads=1, d_ffn=64, n_layers=3, k=61, has_time=True),
     T.MASK_CAUSAL),
    (dict(d=256, d_model=128, n_heads=1, d_ffn=64, n_layers=3, k=61, has_time=True),
     T.MASK_NONE),
    # eight heads of 4, T = 17
    (dict(d=16, d_model=32, n_heads=8, d_ffn=36, n_layers=1, k=17, has_time=False),
     T.MASK_CAUSAL),
])
def test_fp32_encoder_shapes(shape, flags):
    w = synth.scaled(synth.TINY, R=2, L=700, N=10, **shape)
    check_workload(w, flags=flags)


def test_small_bf16_all_candidates():
    w = synth.scaled(synth.SINGLE, R=2, L=3000, N=24, k=64)
    check_workload(w)


@pytest.mark.parametrize("d", [64, 128])
def test_small_bf16_narrow_embedding(d):
    # token / candidate embeddings narrower than d_model: the input projection's
    # token half is zero-padded to 256 columns, its candidate half is a shorter
    # contraction
    w = synth.scaled(synth.SINGLE, R=2, L=1500, N=20, k=64, d=d)
    check_workload(w)


def test_small_bf16_eight_heads_ragged_tail():
    # T = 40 + 0 (not a multiple of 32), 8 heads of 32
    w = synth.scaled(synth.STRESS, R=3, L=900, N=10, k=40, tie_frac=0.01)
    check_workload(w)


def test_small_mixed_realtime_tail():
    w = synth.scaled(synth.MIXED, L=2000, N=16, k=64, rt_len=37)
    check_workload(w)


@pytest.mark.parametrize("cid", [2, 4])
def test_full_workload_all_candidates(cid):
    """Every candidate of the single-request workloads (1000 each)."""
    check_workload(synth.WORKLOADS[cid])


def test_ragged_workload_every_8th_candidate():
    """Every 8th candidate of each of the 64 requests (4,000 of 32,000) and the
    last one of each; T = 128 is one encoder block, one launch."""
    w = synth.RAGGED
    inp = synth.make_inputs(w)
    check_workload(w, ids=strided_ids(inp, 8), inp=inp)


_STRESS = {}


@pytest.mark.parametrize("part", range(4))
def test_stress_workload_every_8th_candidate(part):
    """Every 8th candidate of each request (8,000 of 64,000), the last one of each,
    and both candidates at every edge of the encoder's 2048-candidate launches
    (T = 512 positions: four blocks joined by a K/V cache of 1 MB per candidate,
    2 GB per launch), checked four requests at a time; the GPU runs once."""
    w = synth.STRESS
    if "run" not in _STRESS:
        inp = synth.make_inputs(w)
        W = synth.make_weights(w)
        _STRESS["run"] = (inp, W, run_path(inp, W))
    inp, W, gpu = _STRESS["run"]
    ids = strided_ids(inp, 8, boundaries=range(2048, inp.total, 2048))
    lo, hi = int(inp.cand_offset[4 * part]), int(inp.cand_offset[4 * part + 4])
    check_workload(w, ids=ids[(ids >= lo) & (ids < hi)], W=W, inp=inp, gpu=gpu)


def test_large_mean_layernorm_inputs():
    """Every LayerNorm input shifted by about +8 to +16 on all of its features
    (b_in, b_o and b_2 raised by 8) against a spread of about 0.2: the d_model-256
    kernel's one-pass statistics (E[x^2] - mean^2 in fp32) stay within the bf16
    bound.  T = 200: two encoder blocks joined by the K/V cache."""
    w = synth.scaled(synth.SINGLE, R=1, L=3000, N=16, k=200)
    W = synth.make_weights(w)
    W.b_in = (W.b_in + 8.0).astype(np.float32)
    for L in W.layers:
        L.b_o = (L.b_o + 8.0).astype(np.float32)
        L.b_2 = (L.b_2 + 8.0).astype(np.float32)
    check_workload(w, W=W)


def test_short_and_empty_requests_pad_and_zero():
    w = synth.scaled(synth.MIXED, R=3, L=None, L_range=(1, 1), N=4, k=32, rt_len=5, d=256)
    inp = synth.make_inputs(w)
    # lengths 0, 10 and 500: valid prefixes 5, 15 and 37 of T = 37
    lengths = [0, 10, 500]
    rng = np.random.default_rng(9)
    off = np.zeros(3, dtype=np.int64)
    off[1:] = np.cumsum(lengths)[:-1]
    rows = sum(lengths)
    inp.seq = synth.SeqBatch(emb=rng.integers(-8, 9, (rows, 256)).astype(np.float32) / 8,
                             act=rng.integers(0, 8, rows).astype(np.uint8),
                             time=np.sort(rng.integers(0, 64, rows)).astype(np.uint8),
                             offset=off, length=np.asarray(lengths, dtype=np.int32))
    check_workload(w, inp=inp)
    # no real-time tail and an empty request: all-zero output rows
    w2 = synth.scaled(w, rt_len=0)
    inp2 = synth.Inputs(w=w2, seq=inp.seq, cand=inp.cand, cand_offset=inp.cand_offset)
    idx, score, out = run_path(inp2, synth.make_weights(w2))
    assert torch.all(out[:4] == 0)
    check_workload(w2, inp=inp2)


def test_gather_matches_oracle_bitwise():
    w = synth.scaled(synth.MIXED, R=2, L=1500, N=9, k=48, rt_len=11)
    inp = synth.make_inputs(w)
    seq, rt, cands = upload(inp)
    idx, _ = T.nn_select(seq, cands, w.k)
    tok = T.gather(seq, rt, cands, idx, w.k)
    torch.cuda.synchronize()
    ref = oracle.gather_tokens(inp.seq, inp.rt, inp.cand_request(), idx.cpu().numpy(), w.T)
    np.testing.assert_array_equal(tok.emb.float().cpu().numpy(), ref[0])
    np.testing.assert_array_equal(tok.act.cpu().numpy(), ref[1])
    np.testing.assert_array_equal(tok.time.cpu().numpy(), ref[2])
    np.testing.assert_array_equal(tok.valid_len.cpu().numpy(), ref[3])


@pytest.mark.parametrize("cid", [1, 3])
def test_explicit_tokens_equal_fused_gather(cid):
    w = synth.WORKLOADS[cid]
    if cid == 3:
        w = synth.scaled(w, R=4, N=20)
    inp = synth.make_inputs(w)
    W = synth.make_weights(w)
    seq, rt, cands = upload(inp)
    dw = T.DeviceWeights(W)
    idx, score, out = T.select_encode(seq, rt, cands, w.k, dw)
    tok = T.gather(seq, rt, cands, idx, w.k)
    out2 = T.encode(tok, cands.emb, dw)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)


def test_repeated_runs_bitwise_identical():
    w = synth.scaled(synth.SINGLE, R=1, L=4000, N=40, k=256)
    inp = synth.make_inputs(w)
    W = synth.make_weights(w)
    seq, rt, cands = upload(inp)
    call = T.SelectEncode(seq, rt, cands, w.k, T.DeviceWeights(W))
    first = [t.clone() for t in call()]
    for _ in range(2):
        again = call()
        for a, b in zip(first, again):
            assert torch.equal(a, b)


@pytest.mark.parametrize("case", ["bf16_4heads", "bf16_8heads_ragged", "bf16_rt_tail_128",
                                  "f32_tiny"])
def test_unmasked_encoder(case):
    """TAV2_MASK_NONE: every valid position attends to every valid position (the
    oracle's causal=False), with padding keys excluded; bf16 within one block of
    128 positions."""
    if case == "bf16_4heads":
        w = synth.scaled(synth.SINGLE, R=2, L=3000, N=24, k=64)
    elif case == "bf16_8heads_ragged":   # k past some row counts: valid lengths 40 and 17
        w = synth.scaled(synth.STRESS, R=2, L=None, L_range=(17, 45), N=12, k=40, tie_frac=0.0)
    elif case == "bf16_rt_tail_128":     # T = 100 + 28 = 128 exactly
        w = synth.scaled(synth.MIXED, L=2000, N=16, k=100, rt_len=28)
    else:
        w = synth.TINY
    check_workload(w, flags=T.MASK_NONE)


def test_unmasked_differs_from_causal():
    w = synth.scaled(synth.SINGLE, R=1, L=2000, N=8, k=64)
    inp = synth.make_inputs(w)
    W = synth.make_weights(w)
    _, _, causal = run_path(inp, W)
    _, _, unmasked = run_path(inp, W, flags=T.MASK_NONE)
    assert float((causal - unmasked).abs().max()) > 1e-3


@pytest.mark.parametrize("k", [64, 256])   # one block; two blocks joined by the K/V cache
def test_packed_weights_equal_per_call_packing(k):
    """Weights packed once (tav2_pack_weights) give the outputs of the per-call
    packing bit for bit."""
    w = synth.scaled(synth.MIXED, L=3000, N=40, k=k, rt_len=20)
    inp = synth.make_inputs(w, seed=55)
    W = synth.make_weights(w)
    a = run_path(inp, W)
    b = run_path(inp, W, pack=True)
    for x, y in zip(a, b):
        assert torch.equal(x, y)
