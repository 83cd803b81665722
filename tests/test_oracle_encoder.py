"""Pins for the oracle's feature encoding (Eq. 4), encoder layers and head.

Independent references: torch's own post-LN nn.TransformerEncoderLayer run in
float64 on the CPU (the textbook layer, with a causal mask and without one), the
Eq. 4 special case d_model = 2 d / identity projection, the single-token closed
form, and invariants (causal prefix, head permutation, W_q/W_k independence at
one token, token-permutation equivariance of the unmasked encoder).
"""
import copy

import numpy as np
import pytest
import torch

import oracle
import synth


def small_weights(d=8, dm=16, heads=2, ffn=24, layers=2, T=12, seed=0, has_time=True):
    w = synth.scaled(synth.TINY, d=d, d_model=dm, n_heads=heads, d_ffn=ffn, n_layers=layers,
                     k=T, has_time=has_time)
    W = synth.make_weights(w, seed=seed, scale=0.3)
    return w, W


def random_tokens(n, T, d, seed=1):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((n, T, d)), rng.integers(0, 8, (n, T)),
            rng.integers(0, 64, (n, T)), rng.standard_normal((n, d)))


def torch_layer(Lw, dm, heads, ffn):
    layer = torch.nn.TransformerEncoderLayer(dm, heads, ffn, dropout=0.0, activation="relu",
                                             layer_norm_eps=1e-5, batch_first=True,
                                             norm_first=False, dtype=torch.float64)
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))
    with torch.no_grad():
        layer.self_attn.in_proj_weight.copy_(t(Lw.W_qkv))
        layer.self_attn.in_proj_bias.copy_(t(Lw.b_qkv))
        layer.self_attn.out_proj.weight.copy_(t(Lw.W_o))
        layer.self_attn.out_proj.bias.copy_(t(Lw.b_o))
        layer.linear1.weight.copy_(t(Lw.W_1))
        layer.linear1.bias.copy_(t(Lw.b_1))
        layer.linear2.weight.copy_(t(Lw.W_2))
        layer.linear2.bias.copy_(t(Lw.b_2))
        layer.norm1.weight.copy_(t(Lw.ln1_g))
        layer.norm1.bias.copy_(t(Lw.ln1_b))
        layer.norm2.weight.copy_(t(Lw.ln2_g))
        layer.norm2.bias.copy_(t(Lw.ln2_b))
    layer.eval()
    return layer


@pytest.mark.parametrize("heads,T", [(1, 1), (2, 12), (4, 12), (2, 33)])
def test_layers_match_torch_transformer_encoder_layer(heads, T):
    w, W = small_weights(heads=heads, T=T)
    tok, act, tim, cand = random_tokens(3, T, w.d)
    xs = oracle.encode_states(tok, act, tim, cand, W)
    mask = torch.nn.Transformer.generate_square_subsequent_mask(T, dtype=torch.float64)
    x = torch.tensor(xs[0])
    for li, Lw in enumerate(W.layers):
        layer = torch_layer(Lw, w.d_model, heads, w.d_ffn)
        with torch.no_grad():
            x = layer(x, src_mask=mask, is_causal=True)
        np.testing.assert_allclose(xs[li + 1], x.numpy(), rtol=0, atol=1e-10)


def test_feature_encoding_reduces_to_eq4_with_identity_projection():
    d = 8
    w, W = small_weights(d=d, dm=2 * d, T=10)
    W.W_in = np.eye(2 * d, dtype=np.float32)
    W.b_in = np.zeros(2 * d, dtype=np.float32)
    tok, act, tim, cand = random_tokens(2, 10, d)
    x = oracle.feature_encode(tok, act, tim, cand, W)
    for n in range(2):
        for p in range(10):
            eq4 = (np.concatenate([tok[n, p], cand[n]]) + W.E_act[act[n, p]]
                   + W.E_time[tim[n, p]] + W.E_pos[p])
            np.testing.assert_allclose(x[n, p], eq4, rtol=0, atol=1e-12)


def test_feature_encoding_without_time_table():
    d = 8
    w, W = small_weights(d=d, dm=2 * d, T=6, has_time=False)
    assert W.E_time is None
    W.W_in = np.eye(2 * d, dtype=np.float32)
    W.b_in = np.zeros(2 * d, dtype=np.float32)
    tok, act, tim, cand = random_tokens(1, 6, d)
    x = oracle.feature_encode(tok, act, tim, cand, W)
    eq4 = np.concatenate([tok[0, 3], cand[0]]) + W.E_act[act[0, 3]] + W.E_pos[3]
    np.testing.assert_allclose(x[0, 3], eq4, rtol=0, atol=1e-12)


def test_single_token_closed_form_and_qk_independence():
    """At T = 1 softmax over one key is 1, so attention is x W_v^T + b_v."""
    w, W = small_weights(heads=1, T=1, layers=1)
    tok, act, tim, cand = random_tokens(4, 1, w.d)
    x0 = oracle.feature_encode(tok, act, tim, cand, W)[:, 0]
    Lw = W.layers[0]
    dm = w.d_model
    Wq, Wk, Wv = Lw.W_qkv[:dm], Lw.W_qkv[dm:2 * dm], Lw.W_qkv[2 * dm:]
    bv = Lw.b_qkv[2 * dm:]

    def ln(v, g, b):
        mu = v.mean(-1, keepdims=True)
        var = ((v - mu) ** 2).mean(-1, keepdims=True)
        return (v - mu) / np.sqrt(var + 1e-5) * g + b

    a = x0 @ Wv.T.astype(np.float64) + bv
    h1 = ln(x0 + a @ Lw.W_o.T + Lw.b_o, Lw.ln1_g, Lw.ln1_b)
    h2 = ln(h1 + np.maximum(h1 @ Lw.W_1.T + Lw.b_1, 0) @ Lw.W_2.T + Lw.b_2, Lw.ln2_g, Lw.ln2_b)
    xs = oracle.encode_states(tok, act, tim, cand, W)
    np.testing.assert_allclose(xs[1][:, 0], h2, rtol=0, atol=1e-12)
    # the pooled output is then fixed: max over one token, and that token itself
    out = oracle.encode(tok, act, tim, np.ones(4, np.int32), cand, W)
    np.testing.assert_allclose(out[:, :dm], h2 @ W.W_pool.T + W.b_pool, atol=1e-12)
    np.testing.assert_allclose(out[:, dm:], h2, atol=1e-12)
    # W_q, W_k and their biases cannot matter with one token
    W2 = copy.deepcopy(W)
    W2.layers[0].W_qkv[:2 * dm] = np.random.default_rng(5).standard_normal((2 * dm, dm))
    W2.layers[0].b_qkv[:2 * dm] += 3.0
    np.testing.assert_array_equal(oracle.encode(tok, act, tim, np.ones(4, np.int32), cand, W2), out)


def test_causal_prefix_invariance():
    w, W = small_weights(heads=2, T=16)
    tok, act, tim, cand = random_tokens(2, 16, w.d)
    xs = oracle.encode_states(tok, act, tim, cand, W)
    p = 9
    tok2, act2, tim2 = tok.copy(), act.copy(), tim.copy()
    tok2[:, p + 1:] += 5.0
    act2[:, p + 1:] = (act2[:, p + 1:] + 3) % 8
    tim2[:, p + 1:] = (tim2[:, p + 1:] + 7) % 64
    ys = oracle.encode_states(tok2, act2, tim2, cand, W)
    for x, y in zip(xs, ys):
        np.testing.assert_allclose(x[:, :p + 1], y[:, :p + 1], rtol=0, atol=1e-12)
        assert np.abs(x[:, p + 1:] - y[:, p + 1:]).max() > 1e-3


def test_head_permutation_invariance():
    heads = 4
    w, W = small_weights(dm=16, heads=heads, T=10)
    tok, act, tim, cand = random_tokens(2, 10, w.d)
    out = oracle.encode(tok, act, tim, np.full(2, 10), cand, W)
    dm, dh = 16, 4
    perm = [2, 0, 3, 1]
    cols = np.concatenate([np.arange(h * dh, (h + 1) * dh) for h in perm])
    W2 = copy.deepcopy(W)
    for Lw in W2.layers:
        for part in range(3):
            blk = slice(part * dm, (part + 1) * dm)
            Lw.W_qkv[blk] = Lw.W_qkv[blk][cols]
            Lw.b_qkv[blk] = Lw.b_qkv[blk][cols]
        Lw.W_o = Lw.W_o[:, cols]
    out2 = oracle.encode(tok, act, tim, np.full(2, 10), cand, W2)
    np.testing.assert_allclose(out2, out, rtol=0, atol=1e-12)


def test_pool_properties_and_valid_length_groups():
    w, W = small_weights(heads=2, T=12)
    tok, act, tim, cand = random_tokens(5, 12, w.d)
    valid = np.array([12, 7, 1, 0, 12])
    out = oracle.encode(tok, act, tim, valid, cand, W)
    dm = w.d_model
    assert np.all(out[3] == 0)
    for n in (0, 1, 2, 4):
        t = valid[n]
        xs = oracle.encode_states(tok[n:n + 1, :t], act[n:n + 1, :t], tim[n:n + 1, :t],
                                  cand[n:n + 1], W)
        y = xs[-1][0] @ W.W_pool.T + W.b_pool
        assert np.all(out[n, :dm] >= y - 1e-12)
        np.testing.assert_allclose(out[n, :dm], y.max(axis=0), atol=1e-12)
        np.testing.assert_allclose(out[n, dm:], xs[-1][0, t - 1], atol=1e-12)
    # padding positions never influence valid output
    tok2 = tok.copy()
    tok2[1, 7:] = 100.0
    out2 = oracle.encode(tok2, act, tim, valid, cand, W)
    np.testing.assert_array_equal(out2[1], out[1])


def test_layer_norm_matches_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((4, 7, 32))
    g, b = rng.standard_normal(32), rng.standard_normal(32)
    want = torch.nn.functional.layer_norm(torch.tensor(x), (32,), torch.tensor(g),
                                          torch.tensor(b), eps=1e-5).numpy()
    np.testing.assert_allclose(oracle.encoder.layer_norm(x, g, b), want, rtol=0, atol=1e-12)


@pytest.mark.parametrize("heads,T", [(1, 7), (2, 12), (4, 33)])
def test_unmasked_layers_match_torch_transformer_encoder_layer(heads, T):
    """causal=False is the textbook layer with no attention mask at all."""
    w, W = small_weights(heads=heads, T=T)
    tok, act, tim, cand = random_tokens(3, T, w.d)
    xs = oracle.encode_states(tok, act, tim, cand, W, causal=False)
    x = torch.tensor(xs[0])
    for li, Lw in enumerate(W.layers):
        layer = torch_layer(Lw, w.d_model, heads, w.d_ffn)
        with torch.no_grad():
            x = layer(x)
        np.testing.assert_allclose(xs[li + 1], x.numpy(), rtol=0, atol=1e-10)


def test_unmasked_encoder_is_permutation_equivariant_without_positions():
    """With E_pos = 0 and no mask, permuting the tokens permutes every layer's
    output the same way, so the max-pooled half of the head is unchanged and the
    last-token half is the output of whichever token lands last."""
    T = 11
    w, W = small_weights(heads=2, T=T)
    W.E_pos = np.zeros_like(W.E_pos)
    tok, act, tim, cand = random_tokens(2, T, w.d, seed=4)
    perm = np.random.default_rng(8).permutation(T)
    xs = oracle.encode_states(tok, act, tim, cand, W, causal=False)
    ys = oracle.encode_states(tok[:, perm], act[:, perm], tim[:, perm], cand, W, causal=False)
    for x, y in zip(xs, ys):
        np.testing.assert_allclose(y, x[:, perm], rtol=0, atol=1e-12)
    valid = np.full(2, T)
    out = oracle.encode(tok, act, tim, valid, cand, W, causal=False)
    out_p = oracle.encode(tok[:, perm], act[:, perm], tim[:, perm], valid, cand, W, causal=False)
    dm = w.d_model
    np.testing.assert_allclose(out_p[:, :dm], out[:, :dm], rtol=0, atol=1e-12)
    np.testing.assert_allclose(out_p[:, dm:], xs[-1][:, perm[-1]], rtol=0, atol=1e-12)
    # the causal encoder is not equivariant (a check that the permutation matters)
    c = oracle.encode(tok, act, tim, valid, cand, W)
    c_p = oracle.encode(tok[:, perm], act[:, perm], tim[:, perm], valid, cand, W)
    assert np.abs(c_p[:, :dm] - c[:, :dm]).max() > 1e-6


def test_unmasked_equals_causal_at_one_token_and_differs_after():
    w, W = small_weights(heads=2, T=6)
    tok, act, tim, cand = random_tokens(3, 6, w.d, seed=6)
    one = np.ones(3, np.int32)
    np.testing.assert_array_equal(oracle.encode(tok, act, tim, one, cand, W, causal=False),
                                  oracle.encode(tok, act, tim, one, cand, W))
    six = np.full(3, 6)
    a = oracle.encode(tok, act, tim, six, cand, W, causal=False)
    b = oracle.encode(tok, act, tim, six, cand, W)
    assert np.abs(a - b).max() > 1e-6
