"""Seeded synthetic inputs and weights for the NN-select + encode path.

Both the CPU oracle's tests and the GPU path's tests draw their inputs here, so
this module holds no arithmetic of the method itself: only random draws, the
exact 1/8 grid, bf16 rounding of the drawn weights, and layout bookkeeping.

Recipe (every draw from one numpy PCG64 stream):
  data seed = workload id, weight seed = 100 + workload id.
  * lengths: fixed, or uniform integers in [lo, hi] per request (ragged);
  * action embeddings and candidate embeddings: integers in [-8, 8] / 8, i.e.
    uniform on the 17 multiples of 1/8 in [-1, 1] (every dot product of such
    rows is a multiple of 1/64 and exact in fp32 accumulation);
  * action type: integers in [0, 8); time bucket: sorted integers in [0, 64)
    (row 0 is the most recent action, so its age bucket is the smallest);
  * tie injection: a fraction of rows per request is overwritten by a copy of
    another uniformly chosen row, so the pair ties for every candidate;
  * int8 workloads: every sequence (lifelong, real-time, impression) holds the
    int8 codes of random unit rows (int8_codes); candidates stay on the grid;
  * weights: N(0, 0.02) for every matrix, table and bias; LayerNorm gains
    1 + N(0, 0.02) and offsets N(0, 0.02).  For bf16 and int8 workloads matrices
    and embedding tables are rounded to bf16 (round to nearest even); biases and
    LayerNorm parameters stay fp32.

Matrices use the [out_features, in_features] layout: y = x W^T + b.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from .configs import Workload

N_ACT = 8      # action types
N_TIME = 64    # time buckets


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32)


def grid_values(rng: np.random.Generator, shape) -> np.ndarray:
    """Uniform on {-1, -7/8, ..., 7/8, 1} as float32."""
    return (rng.integers(-8, 9, size=shape).astype(np.float32) / np.float32(8.0))


def int8_codes(rng: np.random.Generator, shape) -> np.ndarray:
    """Codes of the int8 embedding storage (the quantisation formula of Sec. 3.2.1):
    rows drawn as random unit vectors, scaled by 127 / 0.65, rounded half to even
    and clamped to [-127, 127].  Returns int8."""
    e = rng.standard_normal(shape)
    e /= np.maximum(np.linalg.norm(e, axis=-1, keepdims=True), 1e-30)
    return np.clip(np.rint(e * (127.0 / 0.65)), -127, 127).astype(np.int8)


@dataclass
class SeqBatch:
    """A de-duplicated request-level sequence batch: rows of all requests stored once.

    Request r owns rows [offset[r], offset[r] + len[r]); within it row 0 is the
    most recent action.
    """
    emb: np.ndarray                 # [rows, d] float32 (bf16-exact when dtype is bf16)
    act: np.ndarray                 # [rows] uint8
    time: Optional[np.ndarray]      # [rows] uint8 or None
    offset: np.ndarray              # [R] int64
    length: np.ndarray              # [R] int32

    @property
    def R(self) -> int:
        return int(self.offset.shape[0])

    @property
    def max_len(self) -> int:
        return int(self.length.max()) if self.length.size else 0

    def rows(self, r: int) -> slice:
        o = int(self.offset[r])
        return slice(o, o + int(self.length[r]))


@dataclass
class Inputs:
    w: Workload
    seq: SeqBatch
    cand: np.ndarray                # [total, d] float32
    cand_offset: np.ndarray         # [R+1] int64
    rt: Optional[SeqBatch] = None   # real-time sequence per request (mixed workload)
    imp: Optional[SeqBatch] = None  # impression sequence per request (Eq. 2 workload)

    @property
    def total(self) -> int:
        return int(self.cand.shape[0])

    def cand_request(self) -> np.ndarray:
        """Request id of every candidate, [total] int32."""
        out = np.empty(self.total, dtype=np.int32)
        for r in range(self.seq.R):
            out[self.cand_offset[r]:self.cand_offset[r + 1]] = r
        return out


@dataclass
class Layer:
    W_qkv: np.ndarray   # [3*d_model, d_model] rows: q | k | v
    b_qkv: np.ndarray   # [3*d_model]
    W_o: np.ndarray     # [d_model, d_model]
    b_o: np.ndarray
    ln1_g: np.ndarray
    ln1_b: np.ndarray
    W_1: np.ndarray     # [d_ffn, d_model]
    b_1: np.ndarray
    W_2: np.ndarray     # [d_model, d_ffn]
    b_2: np.ndarray
    ln2_g: np.ndarray
    ln2_b: np.ndarray


@dataclass
class Weights:
    d_in: int
    d_model: int
    n_heads: int
    d_ffn: int
    max_pos: int
    dtype: str
    W_in: np.ndarray    # [d_model, 2*d_in]: columns [0, d_in) token, [d_in, 2 d_in) candidate
    b_in: np.ndarray    # [d_model]
    E_act: np.ndarray   # [8, d_model]
    E_time: Optional[np.ndarray]  # [64, d_model] or None
    E_pos: np.ndarray   # [max_pos, d_model]
    layers: List[Layer] = field(default_factory=list)
    W_pool: np.ndarray = None   # [d_model, d_model]
    b_pool: np.ndarray = None   # [d_model]

    @property
    def n_layers(self) -> int:
        return len(self.layers)


def _draw_seq(rng, lengths, d, has_time, tie_frac, codes=False) -> SeqBatch:
    R = len(lengths)
    offset = np.zeros(R, dtype=np.int64)
    if R > 1:
        offset[1:] = np.cumsum(np.asarray(lengths, dtype=np.int64))[:-1]
    rows = int(np.sum(lengths))
    emb = np.empty((rows, d), dtype=np.int8 if codes else np.float32)
    act = np.empty(rows, dtype=np.uint8)
    time = np.empty(rows, dtype=np.uint8) if has_time else None
    for r, L in enumerate(lengths):
        o = int(offset[r])
        e = int8_codes(rng, (L, d)) if codes else grid_values(rng, (L, d))
        if tie_frac > 0.0 and L > 1:
            n_dup = max(1, int(L * tie_frac))
            dst = rng.choice(L, size=n_dup, replace=False)
            src = rng.integers(0, L, size=n_dup)
            src = np.where(src == dst, (src + 1) % L, src)
            e[dst] = e[src]
        emb[o:o + L] = e
        act[o:o + L] = rng.integers(0, N_ACT, size=L).astype(np.uint8)
        if has_time:
            time[o:o + L] = np.sort(rng.integers(0, N_TIME, size=L)).astype(np.uint8)
    return SeqBatch(emb=emb, act=act, time=time, offset=offset,
                    length=np.asarray(lengths, dtype=np.int32))


def make_inputs(w: Workload, seed: Optional[int] = None) -> Inputs:
    rng = np.random.Generator(np.random.PCG64(w.data_seed if seed is None else seed))
    if w.L_range is not None:
        lo, hi = w.L_range
        lengths = [int(x) for x in rng.integers(lo, hi + 1, size=w.R)]
    else:
        lengths = [w.L] * w.R
    seq = _draw_seq(rng, lengths, w.d, w.has_time, w.tie_frac, codes=(w.dtype == "i8"))
    cand = grid_values(rng, (w.R * w.N, w.d))
    cand_offset = np.arange(w.R + 1, dtype=np.int64) * w.N
    rt = None
    if w.rt_len > 0:
        rt = _draw_seq(rng, [w.rt_len] * w.R, w.d, w.has_time, 0.0, codes=(w.dtype == "i8"))
    imp = None
    if w.imp_len > 0:
        imp = _draw_seq(rng, [w.imp_len] * w.R, w.d, w.has_time, 0.0, codes=(w.dtype == "i8"))
    return Inputs(w=w, seq=seq, cand=cand, cand_offset=cand_offset, rt=rt, imp=imp)


def make_weights(w: Workload, seed: Optional[int] = None, scale: float = 0.02) -> Weights:
    rng = np.random.Generator(np.random.PCG64(w.weight_seed if seed is None else seed))
    dm, ff = w.d_model, w.d_ffn
    # int8 sequences feed a bf16 encoder
    wdtype = "bf16" if w.dtype in ("bf16", "i8") else w.dtype
    mat = (lambda a: round_to_bf16(a)) if wdtype == "bf16" else (lambda a: a)

    def n(*shape):
        return (rng.standard_normal(shape) * scale).astype(np.float32)

    W_in = mat(n(dm, 2 * w.d))
    b_in = n(dm)
    E_act = mat(n(N_ACT, dm))
    E_time = mat(n(N_TIME, dm)) if w.has_time else None
    E_pos = mat(n(w.T, dm))
    layers = []
    for _ in range(w.n_layers):
        W_qkv = mat(n(3 * dm, dm))
        b_qkv = n(3 * dm)
        W_o = mat(n(dm, dm))
        b_o = n(dm)
        ln1_g = (1.0 + n(dm)).astype(np.float32)
        ln1_b = n(dm)
        W_1 = mat(n(ff, dm))
        b_1 = n(ff)
        W_2 = mat(n(dm, ff))
        b_2 = n(dm)
        ln2_g = (1.0 + n(dm)).astype(np.float32)
        ln2_b = n(dm)
        layers.append(Layer(W_qkv, b_qkv, W_o, b_o, ln1_g, ln1_b, W_1, b_1, W_2, b_2,
                            ln2_g, ln2_b))
    W_pool = mat(n(dm, dm))
    b_pool = n(dm)
    return Weights(d_in=w.d, d_model=dm, n_heads=w.n_heads, d_ffn=ff, max_pos=w.T,
                   dtype=wdtype, W_in=W_in, b_in=b_in, E_act=E_act, E_time=E_time,
                   E_pos=E_pos, layers=layers, W_pool=W_pool, b_pool=b_pool)


@dataclass
class TokenBatch:
    """Explicit encoder inputs (the encoder run on its own): per candidate T token
    rows with their action types, time buckets and valid length, and the
    candidate's embedding.  Rows at or past a valid length hold grid values too."""
    emb: np.ndarray                 # [total, T, d] float32 on the 1/8 grid, or int8 codes
    act: np.ndarray                 # [total, T] uint8
    time: Optional[np.ndarray]      # [total, T] uint8 or None
    valid_len: np.ndarray           # [total] int32
    cand: np.ndarray                # [total, d] float32 on the 1/8 grid

    @property
    def total(self) -> int:
        return int(self.emb.shape[0])


def make_tokens(total: int, T: int, d: int, has_time: bool = True, seed: int = 0,
                valid_len=None, codes: bool = False) -> TokenBatch:
    """Seeded explicit tokens: grid rows (codes: int8 codes of random unit rows),
    uniform action types, sorted time buckets; valid_len defaults to T for every
    candidate."""
    rng = np.random.Generator(np.random.PCG64(seed))
    emb = int8_codes(rng, (total, T, d)) if codes else grid_values(rng, (total, T, d))
    act = rng.integers(0, N_ACT, size=(total, T)).astype(np.uint8)
    time = np.sort(rng.integers(0, N_TIME, size=(total, T)), axis=1).astype(np.uint8) \
        if has_time else None
    cand = grid_values(rng, (total, d))
    vl = np.full(total, T, dtype=np.int32) if valid_len is None else \
        np.asarray(valid_len, dtype=np.int32)
    return TokenBatch(emb=emb, act=act, time=time, valid_len=vl, cand=cand)


def to_padded(seq: SeqBatch, pad_to: Optional[int] = None) -> SeqBatch:
    """Same requests laid out with a fixed stride (offset[r] = r * stride).

    Rows past a request's length hold arbitrary filler (here: +1 grid rows) that a
    correct consumer never reads.
    """
    stride = pad_to if pad_to is not None else max(seq.max_len, 1)
    R, d = seq.R, seq.emb.shape[1]
    emb = np.ones((R * stride, d), dtype=np.float32)
    act = np.full(R * stride, 7, dtype=np.uint8)
    time = np.full(R * stride, 63, dtype=np.uint8) if seq.time is not None else None
    for r in range(R):
        src = seq.rows(r)
        L = int(seq.length[r])
        emb[r * stride:r * stride + L] = seq.emb[src]
        act[r * stride:r * stride + L] = seq.act[src]
        if time is not None:
            time[r * stride:r * stride + L] = seq.time[src]
    return SeqBatch(emb=emb, act=act, time=time,
                    offset=np.arange(R, dtype=np.int64) * stride, length=seq.length.copy())


def subset_candidates(inp: Inputs, per_request: int) -> Inputs:
    """Keep the first `per_request` candidates of every request (smaller parity runs)."""
    keep = []
    offs = [0]
    for r in range(inp.seq.R):
        a, b = int(inp.cand_offset[r]), int(inp.cand_offset[r + 1])
        sel = np.arange(a, min(b, a + per_request))
        keep.append(sel)
        offs.append(offs[-1] + sel.size)
    idx = np.concatenate(keep) if keep else np.zeros(0, dtype=np.int64)
    return Inputs(w=inp.w, seq=inp.seq, cand=inp.cand[idx].copy(),
                  cand_offset=np.asarray(offs, dtype=np.int64), rt=inp.rt, imp=inp.imp)
