"""Pins of the oracle's dequantisation of the int8 sequence codes (Sec. 3.2.1):
the affine quantisation q = clamp(round(e / 0.65 * 127), -127, 127) is written
out here from the paper's formula, and a code must stand for a value within half
a quantisation step of every value that maps to it."""
import numpy as np

import oracle
import synth


def quantise(e):
    return np.clip(np.rint(np.asarray(e, dtype=np.float64) / 0.65 * 127.0), -127, 127).astype(np.int8)


def test_end_points_and_zero():
    q = np.array([127, -127, 0, 1, -64], dtype=np.int8)
    np.testing.assert_allclose(oracle.dequantise(q), [0.65, -0.65, 0.0, 0.65 / 127, -64 * 0.65 / 127],
                               rtol=0, atol=1e-15)


def test_round_trip_within_half_a_step():
    e = np.linspace(-0.65, 0.65, 100001)
    err = np.abs(oracle.dequantise(quantise(e)) - e)
    assert err.max() <= 0.65 / 254 + 1e-12
    # and every code is its own fixed point
    q = np.arange(-127, 128, dtype=np.int8)
    np.testing.assert_array_equal(quantise(oracle.dequantise(q)), q)


def test_clamped_values_map_to_the_end_codes():
    np.testing.assert_array_equal(quantise([0.9, -3.0]), [127, -127])
    np.testing.assert_allclose(oracle.dequantise(quantise([0.9, -3.0])), [0.65, -0.65])


def test_select_encode_on_codes_equals_the_encoder_on_dequantised_rows():
    """The whole oracle path over int8 storage: its encoder output is the encoder
    applied to the dequantised values of the rows its search selected (and the
    kept real-time rows), not to the raw codes."""
    w = synth.scaled(synth.PAPER_I8, L=300, N=3, k=16, rt_len=5)
    inp = synth.make_inputs(w)
    W = synth.make_weights(w)
    idx, _, out = oracle.select_encode(inp, W, w.k)
    creq = np.zeros(inp.total, dtype=np.int32)
    emb, act, tim, valid = oracle.gather_tokens(inp.seq, inp.rt, creq, idx, w.T)
    ref = oracle.encode(oracle.dequantise(emb.astype(np.int8)), act, tim, valid, inp.cand, W)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    raw = oracle.encode(emb, act, tim, valid, inp.cand, W)
    assert np.abs(raw - out).max() > 1e-3
