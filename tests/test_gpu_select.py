"""GPU parity of tav2_nn_select (Eq. 3) against the oracle: indices and scores
bit for bit, on the five workloads (every candidate of each) and on edge cases
(ragged, empty and short requests, k = 1 and k = K_MAX, heavy ties, padded
layout, every register-tile size of the short-row top-k, the fused search for
long rows with short rows in its batch, ties inside its survivor lists, inputs
that send it to its exhaustive fallback, and the float32 streaming top-k)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_select_equal, oracle_select, upload
from paper_2506_02267_amd import tav2 as T

pytestmark = pytest.mark.gpu


def run_select(inp, k):
    seq, _, cands = upload(inp)
    idx, score = T.nn_select(seq, cands, k)
    torch.cuda.synchronize()
    return idx, score


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_full_workload_all_candidates(cid):
    """Every candidate of every workload (32,000 at ragged, 64,000 at stress)."""
    w = synth.WORKLOADS[cid]
    inp = synth.make_inputs(w)
    print(f"select workload {w.name}: all {inp.total} candidates", flush=True)
    idx, score = run_select(inp, w.k)
    ref_i, ref_s = oracle_select(inp, w.k)
    assert_select_equal(idx, score, ref_i, ref_s)


def custom_inputs(lengths, counts, d=64, dtype="bf16", levels=8, seed=0):
    """Requests with the given lengths and candidate counts (grid values)."""
    rng = np.random.default_rng(seed)
    w = synth.scaled(synth.SINGLE, R=len(lengths), d=d, dtype=dtype, N=max(counts) if counts else 0)
    off = np.zeros(len(lengths), dtype=np.int64)
    off[1:] = np.cumsum(lengths)[:-1]
    rows = int(np.sum(lengths))
    seq = synth.SeqBatch(emb=rng.integers(-levels, levels + 1, (rows, d)).astype(np.float32) / 8,
                         act=rng.integers(0, 8, rows).astype(np.uint8),
                         time=np.sort(rng.integers(0, 64, rows)).astype(np.uint8),
                         offset=off, length=np.asarray(lengths, dtype=np.int32))
    coff = np.zeros(len(counts) + 1, dtype=np.int64)
    coff[1:] = np.cumsum(counts)
    cand = rng.integers(-levels, levels + 1, (int(coff[-1]), d)).astype(np.float32) / 8
    return synth.Inputs(w=w, seq=seq, cand=cand, cand_offset=coff)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_ragged_short_and_empty_requests(dtype):
    inp = custom_inputs([0, 5, 300, 2000, 64], [3, 4, 7, 5, 2], dtype=dtype)
    for k in (1, 64, 301):
        idx, score = run_select(inp, k)
        ref_i, ref_s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, k)
        assert_select_equal(idx, score, ref_i, ref_s)


def test_short_rows_in_a_long_batch():
    # the batch's longest request selects the streaming top-k kernel; its shorter
    # requests take that kernel's other branches (every row kept at <= 2048 rows,
    # sampled threshold just above)
    inp = custom_inputs([5000, 100, 3000, 0, 2048, 2049], [3, 4, 5, 2, 3, 3], seed=7)
    for k in (1, 64, 301, 1024):
        idx, score = run_select(inp, k)
        ref_i, ref_s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, k)
        assert_select_equal(idx, score, ref_i, ref_s)


def test_request_without_candidates():
    inp = custom_inputs([100, 200, 300], [4, 0, 3])
    idx, score = run_select(inp, 16)
    ref_i, ref_s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, 16)
    assert_select_equal(idx, score, ref_i, ref_s)


@pytest.mark.parametrize("L", [100, 3000, 6000, 16384, 20000, 32768])
def test_each_register_tile_size(L):
    inp = custom_inputs([L], [9], d=32, levels=2, seed=L)
    k = min(1024, L)
    idx, score = run_select(inp, k)
    ref_i, ref_s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, k)
    assert_select_equal(idx, score, ref_i, ref_s)


def test_heavy_ties_and_k_max():
    inp = custom_inputs([4096, 3000], [6, 6], d=16, levels=1, seed=3)   # values in {-1/8, 0, 1/8}
    for k in (1, 2, 1024):
        idx, score = run_select(inp, k)
        ref_i, ref_s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, k)
        assert_select_equal(idx, score, ref_i, ref_s)


@pytest.mark.parametrize("k", [1, 256, 1024])
def test_sampled_threshold_with_tied_rows(k):
    # long rows (the top-k takes its threshold from a sample of the keys): every
    # embedding row appears three times in a row, so ties fall inside the
    # compacted candidate set and are resolved by row in the radix select
    inp = custom_inputs([16384, 9000], [5, 4], d=64, levels=8, seed=11)
    for r0, n in zip(inp.seq.offset, inp.seq.length):
        e = inp.seq.emb[r0:r0 + n]
        e[:] = np.repeat(e[0::3], 3, axis=0)[:n]
    idx, score = run_select(inp, k)
    ref_i, ref_s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, k)
    assert_select_equal(idx, score, ref_i, ref_s)


@pytest.mark.parametrize("case", ["all_equal", "sample_misses_top"])
def test_sampled_threshold_falls_back(case):
    # inputs for which the sample gives no usable threshold, so every candidate
    # takes the exhaustive fallback: all scores equal (16384 survivors, far above
    # the list capacity), or the largest scores only on rows the sample never
    # looks at (the sample of a 16384-row request is the 32-row blocks starting at
    # multiples of 512: big scores on rows = 2 mod 4 outside those blocks, about
    # 3600 of them, again above the capacity)
    inp = custom_inputs([16384], [4], d=32, levels=8, seed=5)
    e = inp.seq.emb
    if case == "all_equal":
        e[:] = e[0]
    else:
        rows = np.arange(e.shape[0])
        big = (rows % 4 == 2) & (rows % 512 >= 64)
        e[:] = -np.abs(e)
        e[big] = np.abs(e[big]) + 1.0
        inp.cand[:] = np.abs(inp.cand) + 0.125
    idx, score = run_select(inp, 512)
    ref_i, ref_s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, 512)
    assert_select_equal(idx, score, ref_i, ref_s)


@pytest.mark.parametrize("lengths", [[4096, 300], [4097, 5], [6000, 4000, 0, 1]])
def test_materialised_and_fused_paths_meet(lengths):
    # the longest request decides the path: at most 4096 rows keep the score rows
    # in memory (register top-k), beyond it the scores stay on chip
    inp = custom_inputs(lengths, [3] * len(lengths), d=48, seed=sum(lengths))
    for k in (1, 100, 1024):
        idx, score = run_select(inp, k)
        ref_i, ref_s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, k)
        assert_select_equal(idx, score, ref_i, ref_s)


def test_many_candidate_tiles_with_a_ragged_tail():
    # 3 requests x 300 candidates: three 128-candidate tiles, the last one partial
    inp = custom_inputs([9000, 16384, 5000], [300, 300, 300], d=64, seed=41)
    idx, score = run_select(inp, 256)
    ref_i, ref_s = oracle_select(inp, 256)
    assert_select_equal(idx, score, ref_i, ref_s)


@pytest.mark.parametrize("L", [5000, 20000])
def test_f32_long_rows_stream_topk(L):
    # float32 sequences keep the materialised score rows at every length: rows of
    # more than 4096 keys take the streaming top-k
    inp = custom_inputs([L, 700], [5, 3], d=32, dtype="f32", seed=L + 1)
    for k in (1, 256, 1024):
        idx, score = run_select(inp, k)
        ref_i, ref_s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, k)
        assert_select_equal(idx, score, ref_i, ref_s)


def test_zero_scores_are_positive_zero():
    inp = custom_inputs([50], [3], d=16)
    inp.seq.emb[:] = 0.0
    inp.cand[0] = -1.0
    idx, score = run_select(inp, 10)
    s = score.cpu().numpy()
    assert np.all(s == 0) and not np.any(np.signbit(s))
    np.testing.assert_array_equal(idx.cpu().numpy(), np.tile(np.arange(10), (3, 1)))


def test_padded_layout_equals_packed_and_batch_equals_single():
    w = synth.scaled(synth.RAGGED, R=5, L_range=(700, 3000), N=11, k=128)
    inp = synth.make_inputs(w)
    idx, score = run_select(inp, 128)
    padded = synth.Inputs(w=w, seq=synth.to_padded(inp.seq, pad_to=3072), cand=inp.cand,
                          cand_offset=inp.cand_offset)
    i2, s2 = run_select(padded, 128)
    assert torch.equal(idx, i2) and torch.equal(score.view(torch.int32), s2.view(torch.int32))
    for r in range(w.R):
        a, b = int(inp.cand_offset[r]), int(inp.cand_offset[r + 1])
        one = synth.Inputs(w=w, seq=synth.SeqBatch(
            emb=inp.seq.emb[inp.seq.rows(r)], act=inp.seq.act[inp.seq.rows(r)],
            time=inp.seq.time[inp.seq.rows(r)], offset=np.zeros(1, np.int64),
            length=inp.seq.length[r:r + 1].copy()), cand=inp.cand[a:b],
            cand_offset=np.array([0, b - a], dtype=np.int64))
        i1, s1 = run_select(one, 128)
        assert torch.equal(i1, idx[a:b]) and torch.equal(s1, score[a:b])


def test_repeated_runs_and_streams_are_bitwise_identical():
    w = synth.scaled(synth.STRESS, R=2, N=300, k=512)
    inp = synth.make_inputs(w)
    seq, _, cands = upload(inp)
    outs = []
    for i in range(3):
        st = torch.cuda.Stream()
        with torch.cuda.stream(st):
            outs.append(T.nn_select(seq, cands, 512, stream=st))
        st.synchronize()
    for i, s in outs[1:]:
        assert torch.equal(i, outs[0][0]) and torch.equal(s, outs[0][1])
