"""The oracle's pins must fail on plausible mistakes.

Each test plants one mistake in the oracle (on the CPU, by patching the oracle's
module for the duration of the test) and checks that a pin from
test_oracle_select.py / test_oracle_encoder.py then fails.
"""
import sys

import numpy as np
import pytest

import oracle
import oracle.encoder  # noqa: F401  (registers the submodules)

enc = sys.modules["oracle.encoder"]
sel = sys.modules["oracle.nn_select"]

import test_oracle_encoder as te  # noqa: E402
import test_oracle_eq2 as t2  # noqa: E402
import test_oracle_select as ts  # noqa: E402


def _fails(fn, *args, **kw):
    with pytest.raises(AssertionError):
        fn(*args, **kw)


def test_reversed_tie_break_is_caught(monkeypatch):
    def newest_first_among_ties(s):
        # ties ordered by descending index instead of ascending
        flipped = np.argsort(-s[:, ::-1], axis=1, kind="stable")
        return s.shape[1] - 1 - flipped

    monkeypatch.setattr(sel, "rank_order", newest_first_among_ties)
    _fails(ts.test_hand_worked_example)


def test_wrong_token_order_is_caught(monkeypatch):
    monkeypatch.setattr(sel, "token_positions", lambda idx_row: idx_row[idx_row >= 0].copy())
    _fails(ts.test_gather_places_rank_order_reversed_then_realtime_oldest_first)


def test_wrong_layer_norm_eps_is_caught(monkeypatch):
    monkeypatch.setattr(enc, "LN_EPS", 1e-6)
    monkeypatch.setattr(enc.layer_norm, "__defaults__", (1e-6,))
    _fails(te.test_layers_match_torch_transformer_encoder_layer, 2, 12)


def test_mask_off_by_one_is_caught(monkeypatch):
    def leaky(q, k, v, causal=True):
        T, dh = q.shape[-2], q.shape[-1]
        s = q @ np.swapaxes(k, -1, -2) / np.sqrt(dh)
        s = np.where(np.triu(np.ones((T, T), dtype=bool), k=2), -np.inf, s)  # sees one future key
        s = s - s.max(axis=-1, keepdims=True)
        p = np.exp(s)
        return (p / p.sum(axis=-1, keepdims=True)) @ v

    monkeypatch.setattr(enc, "attention", leaky)
    _fails(te.test_causal_prefix_invariance)
    _fails(te.test_layers_match_torch_transformer_encoder_layer, 2, 12)


def test_missing_output_bias_is_caught(monkeypatch):
    real = enc.encoder_layer

    def no_bo(X, Lw, n_heads, causal=True):
        import copy
        L2 = copy.copy(Lw)
        L2.b_o = np.zeros_like(Lw.b_o)
        return real(X, L2, n_heads, causal)

    monkeypatch.setattr(enc, "encoder_layer", no_bo)
    _fails(te.test_layers_match_torch_transformer_encoder_layer, 2, 12)


def test_swapped_concat_is_caught(monkeypatch):
    real = enc.feature_encode

    def swapped(tok_emb, tok_act, tok_time, cand, W):
        import copy
        d = np.asarray(tok_emb).shape[-1]
        W2 = copy.copy(W)
        W2.W_in = np.concatenate([W.W_in[:, d:], W.W_in[:, :d]], axis=1)
        return real(tok_emb, tok_act, tok_time, cand, W2)

    monkeypatch.setattr(enc, "feature_encode", swapped)
    monkeypatch.setattr(oracle, "feature_encode", swapped)
    _fails(te.test_feature_encoding_reduces_to_eq4_with_identity_projection)


def test_transposed_ffn_weight_is_caught(monkeypatch):
    real = enc.encoder_layer

    def transposed(X, Lw, n_heads, causal=True):
        import copy
        L2 = copy.copy(Lw)
        L2.W_o = Lw.W_o.T.copy()
        return real(X, L2, n_heads, causal)

    monkeypatch.setattr(enc, "encoder_layer", transposed)
    _fails(te.test_layers_match_torch_transformer_encoder_layer, 2, 12)


def test_pool_on_wrong_token_is_caught(monkeypatch):
    def first_token(X, W):
        y = X @ np.asarray(W.W_pool, np.float64).T + W.b_pool
        return np.concatenate([y.max(axis=1), X[:, 0, :]], axis=-1)

    monkeypatch.setattr(enc, "pool", first_token)
    _fails(te.test_pool_properties_and_valid_length_groups)


def _score_mutant(kind):
    """normalised_scores with one plausible mistake."""
    def scores(Q, C):
        Q = np.asarray(Q)
        dot = sel.exact_scores(Q.astype(np.float64), C)
        sq = np.sum(Q.astype(np.int64) ** 2, axis=1).astype(np.float64)
        if kind == "no_normalisation":
            s = dot
        elif kind == "no_square_root":
            s = dot / np.where(sq > 0, sq, 1.0)[None, :]
        else:   # "candidate_normalised": the wrong operand's length
            s = dot / np.linalg.norm(np.asarray(C, dtype=np.float64), axis=1, keepdims=True)
        return s.astype(np.float32)
    return scores


@pytest.mark.parametrize("kind", ["no_normalisation", "no_square_root", "candidate_normalised"])
def test_int8_score_mistakes_are_caught(monkeypatch, kind):
    bad = _score_mutant(kind)
    monkeypatch.setattr(sel, "normalised_scores", bad)
    monkeypatch.setattr(oracle, "normalised_scores", bad)
    _fails(ts.test_normalised_closed_forms)
    _fails(ts.test_normalised_scores_match_the_dequantised_definition, 0)


def test_unmasked_mode_that_keeps_the_causal_mask_is_caught(monkeypatch):
    real = enc.attention
    monkeypatch.setattr(enc, "attention", lambda q, k, v, causal=True: real(q, k, v, True))
    _fails(te.test_unmasked_layers_match_torch_transformer_encoder_layer, 2, 12)
    _fails(te.test_unmasked_encoder_is_permutation_equivariant_without_positions)


def _eq2_mutant(kind):
    """eq2_tokens with one plausible mistake in the order of Eq. 2's parts."""
    real = sel.eq2_tokens

    def tokens(seq, rt, imp, cand_request, idx_ll, r, idx_rt, idx_imp, T):
        if kind == "imp_before_rt_rest":   # S_imp's part ahead of S_RT[r:]'s
            out = real(seq, rt, None, cand_request, idx_ll, r, idx_rt, None, T)
            if imp is None or idx_imp is None:
                return out
            emb, act, tim, valid, prov = real(seq, rt, imp, cand_request, idx_ll, r, None,
                                              idx_imp, T)
            e2, a2, t2_, v2, p2 = real(seq, rt, imp, cand_request, idx_ll, r, idx_rt, idx_imp, T)
            for n in range(valid.shape[0]):
                q = int(cand_request[n])
                keep = min(r, int(rt.length[q])) if rt is not None else 0
                start = int((prov[n, :, 0] == 0).sum()) + keep
                rest = v2[n] - valid[n]                  # S_RT[r:] tokens
                n_imp = valid[n] - start
                order = list(range(start + rest, v2[n])) + list(range(start, start + rest))
                for arr in (e2, a2, t2_, p2):
                    arr[n, start:v2[n]] = arr[n, order]
            return e2, a2, t2_, v2, p2
        # "kept_newest_first": S_RT[:r] in stored order instead of oldest first
        emb, act, tim, valid, prov = real(seq, rt, imp, cand_request, idx_ll, r, idx_rt, idx_imp, T)
        for n in range(valid.shape[0]):
            if rt is None:
                break
            q = int(cand_request[n])
            keep = min(r, int(rt.length[q]))
            start = int((prov[n, :, 0] == 0).sum())
            for arr in (emb, act, tim, prov):
                arr[n, start:start + keep] = arr[n, start:start + keep][::-1].copy()
        return emb, act, tim, valid, prov
    return tokens


@pytest.mark.parametrize("kind", ["imp_before_rt_rest", "kept_newest_first"])
def test_eq2_part_order_mistakes_are_caught(monkeypatch, kind):
    bad = _eq2_mutant(kind)
    monkeypatch.setattr(sel, "eq2_tokens", bad)
    monkeypatch.setattr(oracle, "eq2_tokens", bad)
    _fails(t2.test_hand_worked_example)


def test_eq2_rest_search_over_all_rows_is_caught(monkeypatch):
    real = sel.nn_select_batch

    def no_skip(seq, cand, cand_offset, k, only=None, skip=0):
        return real(seq, cand, cand_offset, k, only=only, skip=0)

    monkeypatch.setattr(sel, "nn_select_batch", no_skip)
    monkeypatch.setattr(oracle, "nn_select_batch", no_skip)
    _fails(t2.test_hand_worked_example)
