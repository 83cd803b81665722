"""GPU parity of tav2_select_encode_eq2, the whole of Eq. 2 (Sec. 3.2.2):
NN(S_LL, c) + S_RT[:r] + NN(S_RT[r:], c) + NN(S_imp, c), against the oracle:
the three searches' rows and scores bit for bit, pooled outputs within 2e-2
(bf16) / 1e-4 (fp32).  Cases: the full Eq. 2 workload (every candidate), ragged
requests whose real-time or impression rows run out before r, k_rt or k_imp
(down to none), the unmasked mode, float32, and the reduction to the lifelong
+ real-time call."""
import numpy as np
import pytest
import torch

import synth
from helpers import BF16_TOL, F32_TOL, assert_select_equal, max_abs, oracle_select_encode_eq2, upload
from paper_2506_02267_amd import tav2 as T

pytestmark = pytest.mark.gpu


def device(inp):
    seq, rt, cands = upload(inp)
    dt = {"bf16": T.BF16, "i8": T.I8}.get(inp.w.dtype, T.F32)
    imp = T.DeviceSeq.from_host(inp.imp, dt) if inp.imp is not None else None
    return seq, rt, imp, cands


def run_eq2(inp, W, flags=T.MASK_CAUSAL):
    w = inp.w
    seq, rt, imp, cands = device(inp)
    call = T.SelectEncodeEq2(seq, rt, w.r, w.k_rt if rt is not None else 0, imp,
                             w.k_imp if imp is not None else 0, cands, w.k,
                             T.DeviceWeights(W), flags)
    out = call()
    torch.cuda.synchronize()
    return out


def check(inp, W, flags=T.MASK_CAUSAL, ids=None):
    w = inp.w
    print(f"eq2 R={w.R} N={w.N} k={w.k} r={w.r} k_rt={w.k_rt} k_imp={w.k_imp} T={w.T} "
          f"flags={flags}", flush=True)
    idx, score, out = run_eq2(inp, W, flags)
    ref_i, ref_s, ref_out = oracle_select_encode_eq2(inp, W, ids=ids,
                                                     causal=flags == T.MASK_CAUSAL)
    assert_select_equal(idx, score, ref_i, ref_s, ids=ids)
    err = max_abs(out, ref_out, ids=ids)
    tol = F32_TOL if w.dtype == "f32" else BF16_TOL
    print(f"  max abs error {err:.3e} (bound {tol})", flush=True)
    assert err <= tol


def test_full_eq2_workload_all_candidates():
    w = synth.EQ2
    check(synth.make_inputs(w), synth.make_weights(w))


def shorten(inp, lengths_ll=None, lengths_rt=None, lengths_imp=None):
    for sq, ln in ((inp.seq, lengths_ll), (inp.rt, lengths_rt), (inp.imp, lengths_imp)):
        if ln is not None:
            sq.length[:] = np.minimum(np.asarray(ln, np.int32), sq.length)
    return inp


def test_ragged_sources_run_out():
    # request 0: everything long enough; 1: real-time rows fewer than r; 2: the
    # real-time rest shorter than k_rt and impressions shorter than k_imp; 3: no
    # impressions and a lifelong sequence shorter than k
    w = synth.scaled(synth.EQ2, R=4, L=3000, N=9, k=64, rt_len=80, rt_keep=20, k_rt=24,
                     imp_len=60, k_imp=40)
    inp = shorten(synth.make_inputs(w, seed=71), lengths_ll=[3000, 3000, 3000, 30],
                  lengths_rt=[80, 11, 35, 80], lengths_imp=[60, 60, 7, 0])
    check(inp, synth.make_weights(w))


def test_long_lifelong_rows_and_several_tiles():
    # 16k-row lifelong sequences (the on-chip-score search) with 300 candidates
    # per request (three 128-candidate tiles)
    w = synth.scaled(synth.EQ2, R=2, L=16384, N=300, k=128, rt_len=120, rt_keep=16, k_rt=48,
                     imp_len=200, k_imp=32)
    check(synth.make_inputs(w, seed=72), synth.make_weights(w))


def test_unmasked_within_one_block():
    w = synth.scaled(synth.EQ2, R=2, L=2000, N=12, k=64, rt_len=40, rt_keep=8, k_rt=16,
                     imp_len=50, k_imp=32)   # T = 120
    check(synth.make_inputs(w, seed=73), synth.make_weights(w), flags=T.MASK_NONE)


def test_float32():
    w = synth.scaled(synth.TINY, R=2, L=300, N=6, k=16, rt_len=20, rt_keep=4, k_rt=8,
                     imp_len=25, k_imp=8, has_time=False)   # T = 36
    check(synth.make_inputs(w, seed=74), synth.make_weights(w))


def test_reduces_to_the_lifelong_plus_realtime_call():
    w = synth.scaled(synth.MIXED, R=2, L=5000, N=40, k=128, rt_len=37)
    inp = synth.make_inputs(w, seed=75)
    W = synth.make_weights(w)
    seq, rt, cands = upload(inp)
    dw = T.DeviceWeights(W)
    a = T.SelectEncode(seq, rt, cands, w.k, dw)()
    b = T.SelectEncodeEq2(seq, rt, 37, 0, None, 0, cands, w.k, dw)()
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
