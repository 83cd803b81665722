"""Oracle for the candidate-anchored nearest-neighbour search (Eq. 3, Sec. 3.2.2).

Test infrastructure only (see the package docstring).

Eq. 3 keeps the K sequence rows with the largest dot product against the
candidate embedding e_c.  Readings taken where the paper is silent:
  * ties: the total order is (score descending, row index ascending); rows are
    stored most-recent-first (the notation table defines S_RT[:r] as the most
    recent r tokens), so among equal scores the more recent action wins;
  * -0.0 and +0.0 are the same score, and a reported zero score is +0.0;
  * when K exceeds the sequence length, the tail is padded with index -1 and
    score -inf;
  * tokens enter the encoder in the order Eq. 3's ascending argsort returns
    them: the selected rows by ascending score, so the best match sits last;
    the kept real-time actions (Eq. 2, S_RT[:r]) follow, oldest first.
"""
from __future__ import annotations

from typing import Optional, Tuple

import numpy as np


def _dyadic_scale(x: np.ndarray, max_bits: int = 24) -> int:
    """Smallest power of two 2^b such that x * 2^b is integral (b <= max_bits)."""
    x64 = np.asarray(x, dtype=np.float64)
    for b in range(max_bits + 1):
        y = x64 * (2.0 ** b)
        if np.all(y == np.round(y)):
            return b
    raise ValueError("oracle scores need dyadic inputs (multiples of 2^-%d)" % max_bits)


def exact_scores(E: np.ndarray, C: np.ndarray) -> np.ndarray:
    """s[n, i] = sum_j E[i, j] * C[n, j], computed exactly (Eq. 3's dot product).

    Both operands are scaled to integers; the integer product is formed with a
    float64 matrix product, which is exact because every partial sum is an
    integer below 2^53 (checked).  Returns float64 [n, L].
    """
    E = np.asarray(E, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    if E.shape[0] == 0 or C.shape[0] == 0:
        return np.zeros((C.shape[0], E.shape[0]), dtype=np.float64)
    be, bc = _dyadic_scale(E), _dyadic_scale(C)
    Ei = np.round(E * 2.0 ** be)
    Ci = np.round(C * 2.0 ** bc)
    bound = np.abs(Ci).sum(axis=1).max() * np.abs(Ei).max()
    if bound >= 2.0 ** 53:
        raise ValueError("integer dot products would exceed float64's exact range")
    s = Ci @ Ei.T
    return s / 2.0 ** (be + bc)


def rank_order(s: np.ndarray) -> np.ndarray:
    """Row indices of each score row in the total order (score desc, index asc).

    A stable sort of the negated scores orders by score descending and keeps
    equal scores in ascending row order; -0.0 and +0.0 compare equal.
    """
    return np.argsort(-s, axis=1, kind="stable")


def dequantise(Q: np.ndarray) -> np.ndarray:
    """Embedding values of int8 codes (Sec. 3.2.1): the affine quantisation maps e
    to round(e / 0.65 * 127) clamped to [-127, 127], so a code q stands for
    q * 0.65 / 127.  float64.  (The paper dequantises into fp16; the encoder
    here takes the value in exact arithmetic.)"""
    return np.asarray(Q, dtype=np.float64) * (0.65 / 127.0)


def normalised_scores(Q: np.ndarray, C: np.ndarray) -> np.ndarray:
    """Scores over the int8 sequence storage with dequantisation and L2
    normalisation (Sec. 3.4.2, fused sequence dequantisation; codes of Sec. 3.2.1).

    Row i dequantises to e_i = (0.65 / 127) q_i and is normalised to unit length
    before the dot product of Eq. 3, so s[n, i] = <e_i / |e_i|, c_n>; the scale
    cancels and s[n, i] = <q_i, c_n> / |q_i|.  An all-zero row scores 0.
    Precision (the paper gives none for this step): the dot product and the sum
    of squares exactly, then one float32 square root and one float32 division,
    each rounded to nearest.  Returns float32 [n, L].
    """
    Q = np.asarray(Q)
    n, L = C.shape[0], Q.shape[0]
    if n == 0 or L == 0:
        return np.zeros((n, L), dtype=np.float32)
    dot = exact_scores(Q.astype(np.float64), C)
    dot32 = dot.astype(np.float32)
    if not np.array_equal(dot32.astype(np.float64), dot):
        raise ValueError("dot products not exact in float32: the rounding order would matter")
    sq = np.sum(Q.astype(np.int64) ** 2, axis=1)
    if sq.max() >= 2 ** 24:
        raise ValueError("sum of squares not exact in float32")
    norm = np.sqrt(sq.astype(np.float32))                  # one rounding
    safe = np.where(sq > 0, norm, np.float32(1.0)).astype(np.float32)
    s = (dot32 / safe[None, :]).astype(np.float32)         # one rounding
    return np.where(sq[None, :] > 0, s, np.float32(0.0)).astype(np.float32)


def _select(s: np.ndarray, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """The first k rows of each score row in the total order, padded."""
    if k < 1:
        raise ValueError("k must be >= 1")
    n, L = s.shape
    idx = np.full((n, k), -1, dtype=np.int32)
    score = np.full((n, k), -np.inf, dtype=np.float32)
    if n == 0 or L == 0:
        return idx, score
    order = rank_order(s)[:, :min(k, L)]
    m = order.shape[1]
    idx[:, :m] = order
    top = np.take_along_axis(s, order, axis=1) + 0.0   # -0.0 -> +0.0
    score[:, :m] = top.astype(np.float32)
    return idx, score


def nn_select(E: np.ndarray, C: np.ndarray, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """Top-k rows of one request's sequence for each of its candidates.

    Returns idx [n, k] int32 (row within the request, -1 padding) and
    score [n, k] float32 (-inf padding), both in the total order
    (score desc, index asc).
    """
    if k < 1:
        raise ValueError("k must be >= 1")
    return _select(exact_scores(E, C), k)


def nn_select_i8(Q: np.ndarray, C: np.ndarray, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """nn_select over int8 codes, ranked by normalised_scores (float32 values,
    compared exactly)."""
    if k < 1:
        raise ValueError("k must be >= 1")
    return _select(normalised_scores(Q, C).astype(np.float64), k)


def nn_select_batch(seq, cand: np.ndarray, cand_offset: np.ndarray, k: int,
                    only: Optional[np.ndarray] = None, skip: int = 0):
    """nn_select over a de-duplicated batch: candidates of request r are
    cand[cand_offset[r]:cand_offset[r+1]] and see only request r's rows.

    `only`, if given, restricts the work to those candidate ids (sampling);
    the rows of other candidates are left as padding.  `skip` searches only the
    rows from skip on of each request (Eq. 2's S_RT[r:]); the indices are then
    relative to that row.
    """
    total = cand.shape[0]
    idx = np.full((total, k), -1, dtype=np.int32)
    score = np.full((total, k), -np.inf, dtype=np.float32)
    want = None if only is None else np.zeros(total, dtype=bool)
    if want is not None:
        want[np.asarray(only, dtype=np.int64)] = True
    for r in range(seq.R):
        a, b = int(cand_offset[r]), int(cand_offset[r + 1])
        ids = np.arange(a, b)
        if want is not None:
            ids = ids[want[a:b]]
        if ids.size == 0:
            continue
        E = seq.emb[seq.rows(r)][skip:]
        i, s = (nn_select_i8 if E.dtype == np.int8 else nn_select)(E, cand[ids], k)
        idx[ids], score[ids] = i, s
    return idx, score


def token_positions(idx_row: np.ndarray) -> np.ndarray:
    """Encoder order of one candidate's selected rows.

    idx_row is in rank order (best first, -1 padded).  Position p of the
    encoder holds rank T_LL - 1 - p, so the selected rows appear by ascending
    score.  Returns the row indices in encoder order (length T_LL).
    """
    valid = idx_row[idx_row >= 0]
    return valid[::-1].copy()


def gather_tokens(seq, rt, cand_request: np.ndarray, idx: np.ndarray, T: int):
    """Selected (and, when present, real-time) rows of every candidate in encoder order.

    Returns tok_emb [total, T, d] float32, tok_act [total, T] uint8,
    tok_time [total, T] uint8 (zeros without a time feature) and
    valid_len [total] int32.  Positions >= valid_len are zero.
    """
    total = idx.shape[0]
    d = seq.emb.shape[1]
    tok_emb = np.zeros((total, T, d), dtype=np.float32)
    tok_act = np.zeros((total, T), dtype=np.uint8)
    tok_time = np.zeros((total, T), dtype=np.uint8)
    valid = np.zeros(total, dtype=np.int32)
    for n in range(total):
        r = int(cand_request[n])
        base = int(seq.offset[r])
        rows = token_positions(idx[n])
        m = rows.size
        src = base + rows
        tok_emb[n, :m] = seq.emb[src]
        tok_act[n, :m] = seq.act[src]
        if seq.time is not None:
            tok_time[n, :m] = seq.time[src]
        p = m
        if rt is not None:
            Lrt = int(rt.length[r])
            # real-time rows are most-recent-first; the encoder takes them oldest first
            rsrc = int(rt.offset[r]) + np.arange(Lrt - 1, -1, -1)
            tok_emb[n, p:p + Lrt] = rt.emb[rsrc]
            tok_act[n, p:p + Lrt] = rt.act[rsrc]
            if rt.time is not None:
                tok_time[n, p:p + Lrt] = rt.time[rsrc]
            p += Lrt
        valid[n] = p
    return tok_emb, tok_act, tok_time, valid


def eq2_tokens(seq, rt, imp, cand_request: np.ndarray, idx_ll: np.ndarray, r: int,
               idx_rt: Optional[np.ndarray], idx_imp: Optional[np.ndarray], T: int):
    """S_all of Eq. 2 for every candidate, in encoder order:

        NN(S_LL, c) + S_RT[:r] + NN(S_RT[r:], c) + NN(S_imp, c)

    idx_ll, idx_rt, idx_imp are the three searches' rows in rank order (best
    first, -1 padded); idx_rt counts rows from S_RT[r]; None (or an absent
    sequence) contributes nothing.  Each NN part enters in ascending score (as
    Eq. 3's argsort returns it) and the kept real-time rows oldest first; the
    valid tokens of all parts are packed from position 0.  Returns tok_emb
    [total, T, d] float32, tok_act / tok_time [total, T] uint8, valid_len
    [total] int32 and prov [total, T, 2] int32: the (source, row) of every
    token, source 0 = S_LL, 1 = S_RT, 2 = S_imp (-1 for padding).
    """
    total = idx_ll.shape[0]
    d = seq.emb.shape[1]
    tok_emb = np.zeros((total, T, d), dtype=np.float32)
    tok_act = np.zeros((total, T), dtype=np.uint8)
    tok_time = np.zeros((total, T), dtype=np.uint8)
    valid = np.zeros(total, dtype=np.int32)
    prov = np.full((total, T, 2), -1, dtype=np.int32)
    for n in range(total):
        q = int(cand_request[n])
        parts = [(0, seq, token_positions(idx_ll[n]))]
        if rt is not None:
            Lrt = int(rt.length[q])
            keep = min(r, Lrt)
            parts.append((1, rt, np.arange(keep - 1, -1, -1)))          # oldest first
            if idx_rt is not None:
                parts.append((1, rt, keep + token_positions(idx_rt[n])))  # S_RT[r:] rows
        if imp is not None and idx_imp is not None:
            parts.append((2, imp, token_positions(idx_imp[n])))
        p = 0
        for src_id, src, rows in parts:
            m = rows.size
            at = int(src.offset[q]) + rows
            tok_emb[n, p:p + m] = src.emb[at]
            tok_act[n, p:p + m] = src.act[at]
            if src.time is not None:
                tok_time[n, p:p + m] = src.time[at]
            prov[n, p:p + m, 0] = src_id
            prov[n, p:p + m, 1] = rows
            p += m
        valid[n] = p
    return tok_emb, tok_act, tok_time, valid, prov
