"""GPU parity of the gather and encoder (Eq. 2 order, Eq. 4, causal encoder,
linear + max-pool head) against the oracle: tokens bit for bit, pooled outputs
within max-abs 1e-4 (fp32) / 2e-2 (bf16)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import BF16_TOL, F32_TOL, assert_select_equal, max_abs, sample_ids, upload
from paper_2506_02267_amd import tav2 as T

pytestmark = pytest.mark.gpu


def run_path(inp, W):
    seq, rt, cands = upload(inp)
    dw = T.DeviceWeights(W)
    idx, score, out = T.select_encode(seq, rt, cands, inp.w.k, dw)
    torch.cuda.synchronize()
    return idx, score, out


def check_workload(w, per_request=None, W=None, inp=None):
    inp = inp if inp is not None else synth.make_inputs(w)
    W = W if W is not None else synth.make_weights(w)
    print(f"select_encode workload {w.name} R={w.R} N={w.N} T={w.T}", flush=True)
    idx, score, out = run_path(inp, W)
    ids = None if per_request is None else sample_ids(inp, per_request)
    ref_i, ref_s, ref_out = oracle.select_encode(inp, W, w.k, only=ids)
    assert_select_equal(idx, score, ref_i, ref_s, ids=ids)
    err = max_abs(out, ref_out, ids=ids)
    tol = F32_TOL if w.dtype == "f32" else BF16_TOL
    print(f"  max abs error {err:.3e} (bound {tol})", flush=True)
    assert err <= tol
    return err


def test_tiny_fp32_all_candidates():
    check_workload(synth.TINY)


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


@pytest.mark.parametrize("cid,per", [(2, 40), (3, 2), (4, 24), (5, 2)])
def test_full_workload_sampled(cid, per):
    check_workload(synth.WORKLOADS[cid], per_request=per)


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
