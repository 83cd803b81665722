"""Pins for the oracle's NN select (Eq. 3) and token assembly (Eq. 2 / Eq. 3 order).

Every check here is independent of the oracle's own arithmetic: a hand-worked
example, brute force with pure-Python integer dot products and Python's sort,
and invariants that any correct top-k under the (score desc, index asc) order
must satisfy.
"""
import json
import os
import random
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth

HERE = os.path.dirname(os.path.abspath(__file__))


def brute_force(E, c, k):
    """Exact scores with Python Fractions, then Python's sort by (-score, index)."""
    s = [sum(Fraction(float(a)) * Fraction(float(b)) for a, b in zip(row, c)) for row in E]
    order = sorted(range(len(E)), key=lambda i: (-s[i], i))[:k]
    return order, [s[i] for i in order]


def test_hand_worked_example():
    g = json.load(open(os.path.join(HERE, "golden", "select_hand.json")))
    E = np.array(g["E"], dtype=np.float32)
    C = np.array(g["c"], dtype=np.float32)
    s = oracle.exact_scores(E, C)
    np.testing.assert_array_equal(s, np.array(g["scores_by_hand"]))
    idx, score = oracle.nn_select(E, C, g["k"])
    np.testing.assert_array_equal(idx, np.array(g["idx"]))
    np.testing.assert_array_equal(score, np.array(g["score"], dtype=np.float32))
    # a zero score is reported as +0.0 (row 3 of candidate 1 is a -0.0 product sum)
    assert not np.any(np.signbit(score[1]))
    for n in range(2):
        np.testing.assert_array_equal(oracle.token_positions(idx[n]), g["encoder_order"][n])
    idx7, score7 = oracle.nn_select(E, C, g["k_over_L"])
    np.testing.assert_array_equal(idx7, np.array(g["idx_k_over_L"]))
    assert np.all(np.isneginf(score7[:, 5:]))


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_tiny(seed):
    rng = random.Random(seed)
    L = rng.randint(1, 48)
    d = rng.randint(1, 6)
    n = rng.randint(1, 4)
    # a small value set forces many ties
    vals = [-1.0, -0.5, -0.125, 0.0, 0.125, 0.5, 1.0] if seed % 2 else [-0.125, 0.0, 0.125]
    E = np.array([[rng.choice(vals) for _ in range(d)] for _ in range(L)], dtype=np.float32)
    C = np.array([[rng.choice(vals) for _ in range(d)] for _ in range(n)], dtype=np.float32)
    for k in sorted({1, max(1, L // 3), L, L + 3}):
        idx, score = oracle.nn_select(E, C, k)
        for j in range(n):
            want_i, want_s = brute_force(E, C[j], k)
            m = len(want_i)
            assert list(idx[j, :m]) == want_i
            assert [Fraction(float(x)) for x in score[j, :m]] == want_s
            assert np.all(idx[j, m:] == -1) and np.all(np.isneginf(score[j, m:]))


def test_exact_scores_match_integer_dot_products():
    rng = np.random.default_rng(7)
    E = synth.generate.grid_values(rng, (300, 256))
    C = synth.generate.grid_values(rng, (5, 256))
    s = oracle.exact_scores(E, C)
    Ei = (E * 8).astype(np.int64).tolist()
    Ci = (C * 8).astype(np.int64).tolist()
    for j in range(5):
        for i in range(0, 300, 7):
            want = sum(a * b for a, b in zip(Ei[i], Ci[j]))
            assert s[j, i] * 64 == want


def _grid_case(seed, L=600, d=32, n=6, levels=3):
    rng = np.random.default_rng(seed)
    E = rng.integers(-levels, levels + 1, size=(L, d)).astype(np.float32) / 8
    C = rng.integers(-levels, levels + 1, size=(n, d)).astype(np.float32) / 8
    return E, C


@pytest.mark.parametrize("seed", range(6))
def test_permuting_unselected_rows_keeps_selection(seed):
    E, C = _grid_case(seed)
    k = 40
    idx, score = oracle.nn_select(E, C, k)
    s = oracle.exact_scores(E, C)
    rng = np.random.default_rng(100 + seed)
    for j in range(C.shape[0]):
        kth = score[j, k - 1]
        below = np.where(s[j] < kth)[0]            # strictly below the k-th score
        perm = below.copy()
        rng.shuffle(perm)
        E2 = E.copy()
        E2[below] = E[perm]
        i2, s2 = oracle.nn_select(E2, C[j:j + 1], k)
        np.testing.assert_array_equal(i2[0], idx[j])
        np.testing.assert_array_equal(s2[0], score[j])


@pytest.mark.parametrize("m", [-3, -1, 1, 2])
def test_candidate_power_of_two_scaling(m):
    E, C = _grid_case(11)
    k = 50
    idx, score = oracle.nn_select(E, C, k)
    i2, s2 = oracle.nn_select(E, C * np.float32(2.0 ** m), k)
    np.testing.assert_array_equal(i2, idx)
    np.testing.assert_array_equal(s2, score * np.float32(2.0 ** m))


def test_k_equals_L_is_full_order_and_k1_is_first_argmax():
    E, C = _grid_case(3, L=200)
    idx, score = oracle.nn_select(E, C, 200)
    s = oracle.exact_scores(E, C)
    for j in range(C.shape[0]):
        assert sorted(idx[j].tolist()) == list(range(200))
        # non-increasing scores, index ascending within equal scores
        for a, b in zip(idx[j][:-1], idx[j][1:]):
            assert s[j, a] > s[j, b] or (s[j, a] == s[j, b] and a < b)
    i1, _ = oracle.nn_select(E, C, 1)
    for j in range(C.shape[0]):
        assert i1[j, 0] == int(np.flatnonzero(s[j] == s[j].max())[0])


def test_duplicated_rows_come_out_in_ascending_index_order():
    w = synth.scaled(synth.STRESS, R=1, L=2048, N=8, k=512)
    inp = synth.make_inputs(w)
    E = inp.seq.emb
    idx, score = oracle.nn_select(E, inp.cand, 512)
    # find duplicated rows (tie injection) and check their relative order
    _, first, inv = np.unique(E, axis=0, return_index=True, return_inverse=True)
    inv = inv.reshape(-1)
    dup_groups = [np.flatnonzero(inv == g) for g in np.flatnonzero(np.bincount(inv) > 1)]
    assert len(dup_groups) > 5
    for j in range(idx.shape[0]):
        pos = {int(r): p for p, r in enumerate(idx[j])}
        for g in dup_groups:
            present = [pos[int(r)] for r in g if int(r) in pos]
            assert present == sorted(present)   # lower row (more recent) first


def test_batch_equals_per_request_and_padded_equals_packed():
    w = synth.scaled(synth.RAGGED, R=4, L_range=(50, 400), N=5, k=64)
    inp = synth.make_inputs(w)
    idx, score = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, 64)
    for r in range(w.R):
        a, b = inp.cand_offset[r], inp.cand_offset[r + 1]
        i1, s1 = oracle.nn_select(inp.seq.emb[inp.seq.rows(r)], inp.cand[a:b], 64)
        np.testing.assert_array_equal(idx[a:b], i1)
        np.testing.assert_array_equal(score[a:b], s1)
    padded = synth.to_padded(inp.seq, pad_to=512)
    i2, s2 = oracle.nn_select_batch(padded, inp.cand, inp.cand_offset, 64)
    np.testing.assert_array_equal(i2, idx)
    np.testing.assert_array_equal(s2, score)


def test_gather_places_rank_order_reversed_then_realtime_oldest_first():
    w = synth.scaled(synth.MIXED, L=300, N=3, k=16, rt_len=5, d=32)
    inp = synth.make_inputs(w)
    idx, _ = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, 16)
    tok_emb, tok_act, tok_time, valid = oracle.gather_tokens(
        inp.seq, inp.rt, inp.cand_request(), idx, 21)
    assert np.all(valid == 21)
    for n in range(3):
        for p in range(16):
            row = idx[n, 15 - p]
            np.testing.assert_array_equal(tok_emb[n, p], inp.seq.emb[row])
            assert tok_act[n, p] == inp.seq.act[row] and tok_time[n, p] == inp.seq.time[row]
        for q in range(5):
            row = 4 - q                   # oldest real-time action first
            np.testing.assert_array_equal(tok_emb[n, 16 + q], inp.rt.emb[row])
            assert tok_act[n, 16 + q] == inp.rt.act[row]


def test_short_request_pads_and_realtime_follows_valid_prefix():
    w = synth.scaled(synth.MIXED, L=10, N=2, k=16, rt_len=4, d=16)
    inp = synth.make_inputs(w)
    idx, score = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, 16)
    assert np.all(idx[:, 10:] == -1) and np.all(np.isneginf(score[:, 10:]))
    tok_emb, tok_act, _, valid = oracle.gather_tokens(inp.seq, inp.rt, inp.cand_request(), idx, 20)
    assert np.all(valid == 14)
    np.testing.assert_array_equal(tok_emb[:, 10], np.broadcast_to(inp.rt.emb[3], (2, 16)))
    assert np.all(tok_emb[:, 14:] == 0)


def test_empty_request_and_no_candidates():
    E = np.zeros((0, 8), dtype=np.float32)
    C = np.ones((3, 8), dtype=np.float32)
    idx, score = oracle.nn_select(E, C, 4)
    assert np.all(idx == -1) and np.all(np.isneginf(score))
    idx, score = oracle.nn_select(np.ones((5, 8), np.float32), np.zeros((0, 8), np.float32), 4)
    assert idx.shape == (0, 4)


# ---------------------------------------------------------------- int8 storage
# Scores over int8 codes with dequantisation and L2 normalisation (Sec. 3.4.2,
# fused sequence dequantisation; the codes of Sec. 3.2.1).

def test_normalised_closed_forms():
    """Hand-computed values: <q, c> / |q| with |q| a perfect square root."""
    Q = np.zeros((5, 16), dtype=np.int8)
    Q[0, :2] = [3, 4]                 # |q| = 5
    Q[1, :4] = [1, 1, 1, 1]           # |q| = 2
    Q[2, 0] = -127                    # |q| = 127
    Q[4, :2] = [-4, 3]                # |q| = 5; row 3 stays zero
    C = np.zeros((1, 16), dtype=np.float32)
    C[0, :4] = [1.0, 1.0, 0.5, 0.5]
    s = oracle.normalised_scores(Q, C)
    assert s.dtype == np.float32
    assert s[0, 0] == np.float32(7.0) / np.float32(5.0)      # 1.4 rounded once
    assert s[0, 1] == np.float32(1.5)                          # (1 + 1 + .5 + .5) / 2
    assert s[0, 2] == np.float32(-1.0)
    assert s[0, 3] == 0.0                                      # all-zero row
    assert s[0, 4] == np.float32(-0.2)                         # (-4 + 3) / 5


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_normalised_scores_match_the_dequantised_definition(seed):
    """Against Sec. 3.4.2 written out in float64: dequantise with the 0.65 / 127
    scale, divide each row by its length, dot with the candidate.  Two roundings
    to float32 bound the difference by about 2 ulp of the score."""
    rng = np.random.default_rng(seed)
    Q = synth.int8_codes(rng, (300, 32))
    C = synth.generate.grid_values(rng, (7, 32))
    s = oracle.normalised_scores(Q, C).astype(np.float64)
    E = Q.astype(np.float64) * (0.65 / 127.0)
    Eh = E / np.linalg.norm(E, axis=1, keepdims=True)
    ref = C.astype(np.float64) @ Eh.T
    assert np.all(np.abs(s - ref) <= 2.5 * 2.0 ** -24 * np.abs(ref) + 1e-12)
    # the normalisation is what ranks: the raw dot product ranks differently
    raw = oracle.exact_scores(Q.astype(np.float64), C)
    assert not np.array_equal(np.argsort(-raw, axis=1), np.argsort(-ref, axis=1))


@pytest.mark.parametrize("seed", [3, 4])
def test_i8_select_is_brute_force_order_of_normalised_scores(seed):
    rng = np.random.default_rng(seed)
    Q = synth.int8_codes(rng, (40, 16))
    Q[[5, 17]] = Q[9]                      # ties: equal rows rank by index
    Q[11] = 0
    C = synth.generate.grid_values(rng, (6, 16))
    s = oracle.normalised_scores(Q, C)
    for k in (1, 7, 40, 45):
        idx, sc = oracle.nn_select_i8(Q, C, k)
        for n in range(C.shape[0]):
            want = sorted(range(40), key=lambda i: (-float(s[n, i]), i))[:k]
            got = [int(i) for i in idx[n] if i >= 0]
            assert got == want
            assert np.array_equal(sc[n, :len(want)], s[n, want] + np.float32(0.0))
            assert np.all(sc[n, len(want):] == -np.inf)


def test_i8_batch_uses_each_requests_rows():
    w = synth.scaled(synth.SELECT_I8, R=3, L=None, L_range=(5, 60), N=4, k=8)
    inp = synth.make_inputs(w, seed=11)
    assert inp.seq.emb.dtype == np.int8
    idx, sc = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, w.k)
    for r in range(w.R):
        a, b = int(inp.cand_offset[r]), int(inp.cand_offset[r + 1])
        i1, s1 = oracle.nn_select_i8(inp.seq.emb[inp.seq.rows(r)], inp.cand[a:b], w.k)
        assert np.array_equal(idx[a:b], i1) and np.array_equal(sc[a:b], s1)
