"""GPU parity of the d_model-64 encoder (the paper's production shape, Sec.
3.2.2, run as one kernel with every weight on chip, Sec. 3.4.2) against the
oracle: explicit tokens at 64 to 2048 positions with ragged valid lengths, one
and two heads, one and two layers, the causal and the unmasked mode, and the
whole select + encode path on the paper workload.  Pooled outputs within
max-abs 2e-2 (bf16 operands, fp32 accumulation)."""
import numpy as np
import pytest
import torch

import synth
from helpers import (BF16_TOL, max_abs, oracle_encode_tokens, upload_tokens)
from test_gpu_encode import check_workload
from paper_2506_02267_amd import tav2 as T

pytestmark = pytest.mark.gpu


def weights_for(T_, d=32, n_heads=1, d_ffn=32, n_layers=2, has_time=True, seed=None):
    """Encoder weights of the paper workload's shape, sized for T_ positions."""
    w = synth.scaled(synth.PAPER, k=T_, rt_len=0, d=d, n_heads=n_heads, d_ffn=d_ffn,
                     n_layers=n_layers, has_time=has_time)
    return synth.make_weights(w, seed=seed)


def ragged_lengths(total, T_, rng):
    """Valid lengths over [0, T_] with the edges of 64-position steps (63, 64, 65,
    127, 128, 129, ...: the encoder's blocks are 64 positions, its key pairs 32)
    and the extremes (0, 1, T_) present."""
    edges = [0, 1, T_]
    for e in range(64, T_ + 1, 64):
        edges += [e - 1, e, e + 1]
    edges = [e for e in edges if 0 <= e <= T_]
    vl = rng.integers(0, T_ + 1, size=total)
    vl[:len(edges)] = edges[:total]
    return vl.astype(np.int32)


def run_and_check(tb, W, flags=T.MASK_CAUSAL, ids=None, tol=BF16_TOL):
    tok, cand = upload_tokens(tb)
    out = T.encode(tok, cand, T.DeviceWeights(W), flags=flags)
    torch.cuda.synchronize()
    ref = oracle_encode_tokens(tb, W, ids=ids, causal=flags == T.MASK_CAUSAL)
    err = max_abs(out, ref, ids=ids)
    print(f"  max abs error {err:.3e} (bound {tol})", flush=True)
    assert err <= tol
    if ids is None:
        empty = np.flatnonzero(tb.valid_len == 0)
        assert torch.all(out[torch.from_numpy(empty).to(out.device)] == 0)
    return out


@pytest.mark.parametrize("T_,total", [(64, 48), (192, 64), (256, 40), (1000, 12), (2048, 8)])
def test_paper_shape_ragged(T_, total):
    """d 32, one head, FFN 32, two layers; positions spanning 1 to 32 blocks of
    64, every block edge among the valid lengths."""
    print(f"encode_small T={T_} total={total}", flush=True)
    rng = np.random.default_rng(T_)
    tb = synth.make_tokens(total, T_, 32, seed=T_, valid_len=ragged_lengths(total, T_, rng))
    run_and_check(tb, weights_for(T_))


@pytest.mark.parametrize("case", ["two_heads", "one_layer_ffn96", "no_time_d64",
                                  "two_heads_one_layer_d256"])
def test_other_shapes(case):
    """Two heads of 32; an FFN wider than 64 (its hidden rows in a region of their
    own); d 64 without the time feature; d 256."""
    T_ = 300
    kw = {"two_heads": dict(n_heads=2),
          "one_layer_ffn96": dict(n_layers=1, d_ffn=96),
          "no_time_d64": dict(d=64, has_time=False),
          "two_heads_one_layer_d256": dict(n_heads=2, n_layers=1, d=256)}[case]
    print(f"encode_small {case}", flush=True)
    rng = np.random.default_rng(7)
    d = kw.get("d", 32)
    tb = synth.make_tokens(24, T_, d, has_time=kw.get("has_time", True), seed=11,
                           valid_len=ragged_lengths(24, T_, rng))
    run_and_check(tb, weights_for(T_, **kw))


def test_many_candidates_persistent_loop():
    """2,500 candidates at 192 positions: about ten candidates per workgroup, each
    reusing the workgroup's K/V cache; every 16th candidate and the last checked."""
    total, T_ = 2500, 192
    print(f"encode_small persistent total={total}", flush=True)
    rng = np.random.default_rng(3)
    tb = synth.make_tokens(total, T_, 32, seed=5, valid_len=rng.integers(1, T_ + 1, total))
    ids = np.unique(np.r_[np.arange(0, total, 16), total - 1])
    run_and_check(tb, weights_for(T_), ids=ids)


@pytest.mark.parametrize("n_heads", [1, 2])
def test_unmasked_one_block(n_heads):
    """TAV2_MASK_NONE within one block of 64: every valid token sees every valid
    token, padding excluded."""
    print(f"encode_small unmasked heads={n_heads}", flush=True)
    rng = np.random.default_rng(n_heads)
    tb = synth.make_tokens(40, 64, 32, seed=21, valid_len=ragged_lengths(40, 64, rng))
    run_and_check(tb, weights_for(64, n_heads=n_heads), flags=T.MASK_NONE)


def test_unmasked_past_one_block_is_unsupported():
    tb = synth.make_tokens(2, 65, 32, seed=1)
    tok, cand = upload_tokens(tb)
    with pytest.raises(T.Tav2Error) as e:
        T.encode(tok, cand, T.DeviceWeights(weights_for(65)), flags=T.MASK_NONE)
    assert e.value.status == -4   # TAV2_ERR_UNSUPPORTED


def test_paper_workload_select_encode():
    """The whole path on the paper workload: NN top-128 over a 16k lifelong
    sequence of 32-d embeddings plus 64 real-time actions (192 positions), 256
    candidates, every candidate checked."""
    check_workload(synth.PAPER)


@pytest.mark.parametrize("kw", [dict(), dict(n_heads=2, d=64)])
def test_packed_weights_equal_unpacked(kw):
    """Weights packed once (the kernel's LDS image, loaded by one contiguous copy)
    give the outputs of the weights read as given, bit for bit."""
    d = kw.get("d", 32)
    tb = synth.make_tokens(64, 192, d, seed=4, valid_len=np.random.default_rng(4).integers(0, 193, 64))
    tok, cand = upload_tokens(tb)
    W = weights_for(192, **kw)
    a = T.encode(tok, cand, T.DeviceWeights(W))
    b = T.encode(tok, cand, T.DeviceWeights(W, pack=True))
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_int8_code_tokens():
    """Explicit tokens stored as int8 codes (Sec. 3.2.1): the encoder takes their
    dequantised values (the oracle: codes x 0.65 / 127 in float64)."""
    rng = np.random.default_rng(8)
    tb = synth.make_tokens(48, 192, 32, seed=8, valid_len=ragged_lengths(48, 192, rng), codes=True)
    run_and_check(tb, weights_for(192))


def test_paper_int8_workload_select_encode():
    """The paper's production path on its int8 storage: NN top-128 with fused
    dequantisation and L2 normalisation over 16k codes, the 64 real-time code
    rows kept, the encoder on the dequantised rows; every candidate checked."""
    check_workload(synth.PAPER_I8)


def test_repeated_runs_bitwise_identical():
    tb = synth.make_tokens(300, 192, 32, seed=2)
    tok, cand = upload_tokens(tb)
    dw = T.DeviceWeights(weights_for(192))
    first = T.encode(tok, cand, dw).clone()
    for _ in range(2):
        assert torch.equal(T.encode(tok, cand, dw), first)
