"""Pins for the oracle's token set of Eq. 2 (Sec. 3.2.2): a hand-worked
example (tests/golden/eq2_hand.json), the reduction to the lifelong + kept
real-time assembly when the other searches are off, per-part invariants on
random inputs, and the search over S_RT[r:] as a search over the sliced rows."""
import json
import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "eq2_hand.json")


def seqbatch(rows, act_base):
    E = np.asarray(rows, dtype=np.float32)
    L = E.shape[0]
    return synth.SeqBatch(emb=E, act=(act_base + np.arange(L)).astype(np.uint8) % 8,
                          time=np.arange(L, dtype=np.uint8), offset=np.zeros(1, np.int64),
                          length=np.array([L], np.int32))


def test_hand_worked_example():
    g = json.load(open(GOLDEN))
    c = np.asarray([g["c"]], dtype=np.float32)
    ll, rt, imp = seqbatch(g["S_LL"], 0), seqbatch(g["S_RT"], 3), seqbatch(g["S_imp"], 5)
    for name, sq in (("S_LL", ll), ("S_RT", rt), ("S_imp", imp)):
        np.testing.assert_array_equal(oracle.exact_scores(sq.emb, c)[0], g[name + "_scores_by_hand"])
    off = np.array([0, 1], np.int64)
    for case in g["cases"]:
        k, r, k_rt, k_imp = case["k"], case["r"], case["k_rt"], case["k_imp"]
        i_ll, _ = oracle.nn_select_batch(ll, c, off, k)
        i_rt, _ = oracle.nn_select_batch(rt, c, off, k_rt, skip=r)
        i_imp, _ = oracle.nn_select_batch(imp, c, off, k_imp)
        assert i_ll[0].tolist() == case["idx_ll"]
        assert i_rt[0].tolist() == case["idx_rt_from_r"]
        assert i_imp[0].tolist() == case["idx_imp"]
        T = k + r + k_rt + k_imp
        emb, act, tim, valid, prov = oracle.eq2_tokens(ll, rt, imp, np.zeros(1, np.int32), i_ll,
                                                       r, i_rt, i_imp, T)
        want = case["tokens"]
        assert int(valid[0]) == len(want)
        assert prov[0, :len(want)].tolist() == want
        assert np.all(prov[0, len(want):] == -1) and np.all(emb[0, len(want):] == 0)
        src = {0: ll, 1: rt, 2: imp}
        for p, (s_id, row) in enumerate(want):
            np.testing.assert_array_equal(emb[0, p], src[s_id].emb[row])
            assert act[0, p] == src[s_id].act[row] and tim[0, p] == src[s_id].time[row]


def test_reduces_to_lifelong_plus_kept_realtime():
    """No search over S_RT[r:] or S_imp and r at least the real-time length: the
    pinned lifelong + kept real-time assembly."""
    w = synth.scaled(synth.MIXED, R=3, L=None, L_range=(50, 400), N=5, k=64, rt_len=37)
    inp = synth.make_inputs(w, seed=3)
    idx, _ = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, w.k)
    creq = inp.cand_request()
    a = oracle.gather_tokens(inp.seq, inp.rt, creq, idx, w.T)
    b = oracle.eq2_tokens(inp.seq, inp.rt, None, creq, idx, 10 ** 6, None, None, w.T)
    for x, y in zip(a, b[:4]):
        np.testing.assert_array_equal(x, y)


def test_rest_search_is_a_search_over_the_sliced_rows():
    w = synth.scaled(synth.EQ2, R=2, L=300, N=6, rt_len=90, rt_keep=17, k_rt=20)
    inp = synth.make_inputs(w, seed=4)
    got, gs = oracle.nn_select_batch(inp.rt, inp.cand, inp.cand_offset, w.k_rt, skip=w.r)
    for q in range(inp.rt.R):
        rows = inp.rt.emb[inp.rt.rows(q)][w.r:]
        a, b = int(inp.cand_offset[q]), int(inp.cand_offset[q + 1])
        want, ws = oracle.nn_select(rows, inp.cand[a:b], w.k_rt)
        np.testing.assert_array_equal(got[a:b], want)
        np.testing.assert_array_equal(gs[a:b], ws)


@pytest.mark.parametrize("lens", [(300, 90, 120), (40, 10, 5), (0, 0, 0)])
def test_part_lengths_and_contents(lens):
    L, Lrt, Limp = lens
    w = synth.scaled(synth.EQ2, R=1, L=max(L, 1), N=7, k=64, rt_len=max(Lrt, 1), rt_keep=16,
                     k_rt=24, imp_len=max(Limp, 1), k_imp=32)
    inp = synth.make_inputs(w, seed=5)
    for sq, n in ((inp.seq, L), (inp.rt, Lrt), (inp.imp, Limp)):   # shorten to the case's lengths
        sq.length[:] = n
    idx, score, out = oracle.select_encode_eq2(inp, synth.make_weights(w))
    k, r = w.k, w.r
    t_ll, t_keep = min(k, L), min(r, Lrt)
    t_rt, t_imp = min(w.k_rt, max(Lrt - r, 0)), min(w.k_imp, Limp)
    i_ll, i_rt, i_imp = idx[:, :k], idx[:, k:k + w.k_rt], idx[:, k + w.k_rt:]
    _, _, _, valid, prov = oracle.eq2_tokens(inp.seq, inp.rt, inp.imp, inp.cand_request(),
                                             i_ll, r, i_rt, i_imp, w.T)
    assert np.all(valid == t_ll + t_keep + t_rt + t_imp)
    for n in range(inp.total):
        p = prov[n]
        np.testing.assert_array_equal(p[:t_ll, 1], i_ll[n, :t_ll][::-1])
        np.testing.assert_array_equal(p[t_ll:t_ll + t_keep, 1], np.arange(t_keep)[::-1])
        seg = p[t_ll + t_keep:t_ll + t_keep + t_rt, 1]
        np.testing.assert_array_equal(seg, t_keep + i_rt[n, :t_rt][::-1])
        seg = p[t_ll + t_keep + t_rt:valid[n], 1]
        np.testing.assert_array_equal(seg, i_imp[n, :t_imp][::-1])
        assert list(p[:valid[n], 0]) == [0] * t_ll + [1] * (t_keep + t_rt) + [2] * t_imp
    if valid.max() == 0:
        assert np.all(out == 0)


def test_eq2_path_without_extra_searches_equals_the_mixed_path():
    w = synth.scaled(synth.MIXED, R=2, L=500, N=4, k=32, rt_len=12)
    inp = synth.make_inputs(w, seed=6)
    W = synth.make_weights(w)
    i1, s1, o1 = oracle.select_encode(inp, W, w.k)
    i2, s2, o2 = oracle.select_encode_eq2(inp, W)
    np.testing.assert_array_equal(i1, i2)
    np.testing.assert_array_equal(s1, s2)
    np.testing.assert_array_equal(o1, o2)
