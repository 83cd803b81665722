"""Oracle for feature encoding (Eq. 4), the causal transformer encoder and the
linear + max-pool head (Sec. 3.2.2), in float64.

Test infrastructure only (see the package docstring).

Readings taken where the paper is silent or its widths disagree:
  * Eq. 4 concatenates the token's PinSage embedding with the candidate's
    (early fusion) and adds action, surface and position embeddings of the
    same width.  Here the concatenation [e_p ; e_c] is projected to d_model by
    a learned W_in, b_in (this is Eq. 4 exactly when d_model = 2 d, W_in = I,
    b_in = 0), and the side features are an action-type table, a time-bucket
    table in place of surface, and a learned position table.
  * Encoder layer: post-LayerNorm (add & norm after each sublayer), ReLU FFN,
    biases on every linear map, scaled dot-product attention with scale
    1/sqrt(d_head), LayerNorm with population variance and eps = 1e-5.
  * Mask: causal over encoder positions (Sec. 3.2.2 and Sec. 3.3.2: a token sees
    itself and earlier tokens only).  Positions at or past a candidate's valid
    length are padding; no valid position may see them, so the oracle simply
    runs on the valid prefix.  `causal=False` drops the causal mask (every valid
    token sees every valid token), the unmasked setting of the paper's appendix
    comparison of its fused transformer (Appendix B).
  * Head: out = [max over valid positions of (X W_pool^T + b_pool) ; X at the
    last valid position], width 2 d_model.  A candidate with no valid token
    gets zeros.
"""
from __future__ import annotations

import numpy as np

LN_EPS = 1e-5


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def feature_encode(tok_emb, tok_act, tok_time, cand, W):
    """X0 for a group of candidates sharing one valid length T.

    tok_emb [n, T, d], tok_act/tok_time [n, T], cand [n, d] -> [n, T, d_model].
    """
    e = _f64(tok_emb)
    n, T, d = e.shape
    c = np.broadcast_to(_f64(cand)[:, None, :], (n, T, d))
    fused = np.concatenate([e, c], axis=-1)                  # early fusion: [e_p ; e_c]
    x = fused @ _f64(W.W_in).T + _f64(W.b_in)
    x = x + _f64(W.E_act)[np.asarray(tok_act, dtype=np.int64)]
    if W.E_time is not None:
        x = x + _f64(W.E_time)[np.asarray(tok_time, dtype=np.int64)]
    x = x + _f64(W.E_pos)[:T][None, :, :]
    return x


def layer_norm(x, g, b, eps=LN_EPS):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * _f64(g) + _f64(b)


def attention(q, k, v, causal=True):
    """q, k, v: [n, heads, T, d_head] -> [n, heads, T, d_head]; scaled dot-product
    attention over all T positions, causal unless causal=False."""
    T, dh = q.shape[-2], q.shape[-1]
    s = q @ np.swapaxes(k, -1, -2) / np.sqrt(dh)
    if causal:
        future = np.triu(np.ones((T, T), dtype=bool), k=1)  # key j > query p
        s = np.where(future, -np.inf, s)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    return p @ v


def encoder_layer(X, Lw, n_heads, causal=True):
    """One post-LN encoder layer on X [n, T, d_model]."""
    n, T, dm = X.shape
    dh = dm // n_heads
    qkv = X @ _f64(Lw.W_qkv).T + _f64(Lw.b_qkv)
    q, k, v = qkv[..., :dm], qkv[..., dm:2 * dm], qkv[..., 2 * dm:]

    def heads(t):
        return t.reshape(n, T, n_heads, dh).transpose(0, 2, 1, 3)

    o = attention(heads(q), heads(k), heads(v), causal)
    o = o.transpose(0, 2, 1, 3).reshape(n, T, dm)
    X = layer_norm(X + o @ _f64(Lw.W_o).T + _f64(Lw.b_o), Lw.ln1_g, Lw.ln1_b)
    h = np.maximum(X @ _f64(Lw.W_1).T + _f64(Lw.b_1), 0.0)
    X = layer_norm(X + h @ _f64(Lw.W_2).T + _f64(Lw.b_2), Lw.ln2_g, Lw.ln2_b)
    return X


def pool(X, W):
    """[n, T, d_model] (all valid) -> [n, 2 d_model]: max of the linear map, last token."""
    n, T, dm = X.shape
    if T == 0:
        return np.zeros((n, 2 * dm), dtype=np.float64)
    y = X @ _f64(W.W_pool).T + _f64(W.b_pool)
    return np.concatenate([y.max(axis=1), X[:, T - 1, :]], axis=-1)


def encode_states(tok_emb, tok_act, tok_time, cand, W, causal=True):
    """All hidden states [X0, X1, ...] for a group with one valid length (pins use it)."""
    xs = [feature_encode(tok_emb, tok_act, tok_time, cand, W)]
    for Lw in W.layers:
        xs.append(encoder_layer(xs[-1], Lw, W.n_heads, causal))
    return xs


def encode(tok_emb, tok_act, tok_time, valid_len, cand, W, chunk=32, only=None, causal=True):
    """Pooled encoder output for every candidate (or the ids in `only`).

    tok_emb [total, T, d], tok_act/tok_time [total, T], valid_len [total],
    cand [total, d] -> out [total, 2 d_model] float64 (rows outside `only` are 0).
    """
    total = tok_emb.shape[0]
    dm = W.d_model
    out = np.zeros((total, 2 * dm), dtype=np.float64)
    ids = np.arange(total) if only is None else np.asarray(only, dtype=np.int64)
    valid_len = np.asarray(valid_len)
    for t in np.unique(valid_len[ids]):
        group = ids[valid_len[ids] == t]
        if t == 0:
            continue
        for s in range(0, group.size, chunk):
            g = group[s:s + chunk]
            xs = encode_states(tok_emb[g, :t], tok_act[g, :t], tok_time[g, :t], cand[g], W,
                               causal)
            out[g] = pool(xs[-1], W)
    return out


def select_encode(inputs, W, k, only=None, chunk=32, causal=True):
    """The whole path: NN select (Eq. 3), token assembly (Eq. 2 with the kept
    real-time tail), feature encoding (Eq. 4), encoder and head.

    Returns idx, score (as nn_select_batch) and out [total, 2 d_model] float64.
    """
    from .nn_select import nn_select_batch, gather_tokens, dequantise
    idx, score = nn_select_batch(inputs.seq, inputs.cand, inputs.cand_offset, k, only=only)
    T = k + (0 if inputs.rt is None else int(inputs.rt.length.max()))
    creq = np.empty(inputs.cand.shape[0], dtype=np.int32)
    for r in range(inputs.seq.R):
        creq[inputs.cand_offset[r]:inputs.cand_offset[r + 1]] = r
    ids = np.arange(inputs.cand.shape[0]) if only is None else np.asarray(only, dtype=np.int64)
    tok_emb, tok_act, tok_time, valid = gather_tokens(inputs.seq, inputs.rt, creq[ids],
                                                      idx[ids], T)
    if inputs.seq.emb.dtype == np.int8:   # int8 storage: the encoder takes the values
        tok_emb = dequantise(tok_emb)
    out_ids = encode(tok_emb, tok_act, tok_time, valid, inputs.cand[ids], W, chunk=chunk,
                     causal=causal)
    out = np.zeros((inputs.cand.shape[0], 2 * W.d_model), dtype=np.float64)
    out[ids] = out_ids
    return idx, score, out


def select_encode_eq2(inputs, W, only=None, chunk=32, causal=True):
    """The whole path with every source of Eq. 2: NN(S_LL, c) with k rows,
    S_RT[:r], NN(S_RT[r:], c) with k_rt rows and NN(S_imp, c) with k_imp rows
    (the workload's fields), token assembly, Eq. 4, encoder and head.

    Returns idx [total, k + k_rt + k_imp] int32 (the three searches' rows in
    rank order side by side: S_LL rows, then S_RT[r:] rows counted from S_RT[r],
    then S_imp rows; -1 padded), score of the same shape (float32, -inf padded)
    and out [total, 2 d_model] float64.
    """
    from .nn_select import nn_select_batch, eq2_tokens, dequantise
    w = inputs.w
    k, r = w.k, w.r
    k_rt = w.k_rt if inputs.rt is not None else 0
    k_imp = w.k_imp if inputs.imp is not None else 0
    total = inputs.cand.shape[0]
    idx_ll, s_ll = nn_select_batch(inputs.seq, inputs.cand, inputs.cand_offset, k, only=only)
    idx_rt = s_rt = idx_imp = s_imp = None
    if k_rt > 0:
        idx_rt, s_rt = nn_select_batch(inputs.rt, inputs.cand, inputs.cand_offset, k_rt,
                                       only=only, skip=r)
    if k_imp > 0:
        idx_imp, s_imp = nn_select_batch(inputs.imp, inputs.cand, inputs.cand_offset, k_imp,
                                         only=only)
    creq = np.empty(total, dtype=np.int32)
    for q in range(inputs.seq.R):
        creq[inputs.cand_offset[q]:inputs.cand_offset[q + 1]] = q
    ids = np.arange(total) if only is None else np.asarray(only, dtype=np.int64)
    pick = lambda a: None if a is None else a[ids]
    tok_emb, tok_act, tok_time, valid, _ = eq2_tokens(
        inputs.seq, inputs.rt, inputs.imp, creq[ids], idx_ll[ids], r, pick(idx_rt),
        pick(idx_imp), w.T)
    if inputs.seq.emb.dtype == np.int8:
        tok_emb = dequantise(tok_emb)
    out = np.zeros((total, 2 * W.d_model), dtype=np.float64)
    out[ids] = encode(tok_emb, tok_act, tok_time, valid, inputs.cand[ids], W, chunk=chunk,
                      causal=causal)
    idx = np.concatenate([a for a in (idx_ll, idx_rt, idx_imp) if a is not None], axis=1)
    score = np.concatenate([a for a in (s_ll, s_rt, s_imp) if a is not None], axis=1)
    return idx, score, out
