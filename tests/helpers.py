"""Shared plumbing for the GPU parity tests (device upload, oracle sampling,
the oracle spread over the host's cores)."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

import oracle
import synth
from paper_2506_02267_amd import tav2 as T

BF16_TOL = 2e-2   # max-abs error bound for bf16 encoder outputs
F32_TOL = 1e-4    # max-abs error bound for fp32 encoder outputs


def dtype_code(w):
    return {"bf16": T.BF16, "i8": T.I8}.get(w.dtype, T.F32)


def upload(inp, device="cuda"):
    dt = dtype_code(inp.w)
    seq = T.DeviceSeq.from_host(inp.seq, dt, device)
    rt = T.DeviceSeq.from_host(inp.rt, dt, device) if inp.rt is not None else None
    cands = T.DeviceCands.from_host(inp.cand, inp.cand_offset, dt, device)
    return seq, rt, cands


def assert_select_equal(idx_gpu, score_gpu, idx_ref, score_ref, ids=None):
    ig = idx_gpu.cpu().numpy()
    sg = score_gpu.cpu().numpy()
    if ids is not None:
        ig, sg, idx_ref, score_ref = ig[ids], sg[ids], idx_ref[ids], score_ref[ids]
    bad = np.argwhere(ig != idx_ref)
    assert bad.size == 0, f"{len(bad)} idx mismatches, first at {bad[:5].tolist()}"
    # scores compared bit for bit (+0.0 canonical, -inf padding)
    assert np.array_equal(sg.view(np.uint32), score_ref.astype(np.float32).view(np.uint32))


def max_abs(out_gpu, out_ref, ids=None):
    og = out_gpu.cpu().numpy().astype(np.float64)
    if ids is not None:
        og, out_ref = og[ids], out_ref[ids]
    assert np.all(np.isfinite(og))
    return float(np.abs(og - out_ref).max()) if og.size else 0.0


def host_workers():
    """Threads for oracle work: the host's cores, at most 16 (one GPU's share)."""
    return max(1, min(16, os.cpu_count() or 1))


def parallel_map(fn, parts):
    """fn over parts on host_workers() threads with single-threaded BLAS (numpy
    releases the GIL in its array loops and BLAS calls, so the oracle's pieces
    run side by side)."""
    from threadpoolctl import threadpool_limits
    with threadpool_limits(1):
        with ThreadPoolExecutor(host_workers()) as ex:
            return list(ex.map(fn, parts))


def chunks(ids, size):
    ids = np.asarray(ids, dtype=np.int64)
    return [ids[i:i + size] for i in range(0, ids.size, size)]


def oracle_select(inp, k, ids=None, chunk=64):
    """oracle.nn_select_batch for the candidates in ids (all by default), split
    into chunks computed in parallel; rows outside ids are padding."""
    total = inp.total
    ids = np.arange(total) if ids is None else np.asarray(ids, dtype=np.int64)
    idx = np.full((total, k), -1, dtype=np.int32)
    score = np.full((total, k), -np.inf, dtype=np.float32)

    def one(part):
        i, s = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, k, only=part)
        return part, i[part], s[part]

    for part, i, s in parallel_map(one, chunks(ids, chunk)):
        idx[part], score[part] = i, s
    return idx, score


def oracle_select_encode(inp, W, k, ids=None, chunk=16, causal=True):
    """oracle.select_encode for the candidates in ids (all by default), in
    parallel chunks.  Returns idx, score, out as oracle.select_encode does."""
    total = inp.total
    ids = np.arange(total) if ids is None else np.asarray(ids, dtype=np.int64)
    idx = np.full((total, k), -1, dtype=np.int32)
    score = np.full((total, k), -np.inf, dtype=np.float32)
    out = np.zeros((total, 2 * W.d_model), dtype=np.float64)

    def one(part):
        i, s, o = oracle.select_encode(inp, W, k, only=part, causal=causal)
        return part, i[part], s[part], o[part]

    for part, i, s, o in parallel_map(one, chunks(ids, chunk)):
        idx[part], score[part], out[part] = i, s, o
    return idx, score, out


def strided_ids(inp, stride, boundaries=()):
    """Every stride-th candidate of every request (from its first), the last
    candidate of each request, and both candidates on each side of every global
    index in boundaries (launch chunk edges)."""
    ids = set()
    for r in range(inp.seq.R):
        a, b = int(inp.cand_offset[r]), int(inp.cand_offset[r + 1])
        ids.update(range(a, b, stride))
        if b > a:
            ids.add(b - 1)
    for e in boundaries:
        ids.update(x for x in (e - 1, e) if 0 <= x < inp.total)
    return np.array(sorted(ids), dtype=np.int64)


def oracle_select_encode_eq2(inp, W, ids=None, chunk=16, causal=True):
    """oracle.select_encode_eq2 for the candidates in ids (all by default), in
    parallel chunks."""
    w = inp.w
    total = inp.total
    K = w.k + (w.k_rt if inp.rt is not None else 0) + (w.k_imp if inp.imp is not None else 0)
    ids = np.arange(total) if ids is None else np.asarray(ids, dtype=np.int64)
    idx = np.full((total, K), -1, dtype=np.int32)
    score = np.full((total, K), -np.inf, dtype=np.float32)
    out = np.zeros((total, 2 * W.d_model), dtype=np.float64)

    def one(part):
        i, s, o = oracle.select_encode_eq2(inp, W, only=part, causal=causal)
        return part, i[part], s[part], o[part]

    for part, i, s, o in parallel_map(one, chunks(ids, chunk)):
        idx[part], score[part], out[part] = i, s, o
    return idx, score, out


def upload_tokens(tb, dtype=T.BF16, device="cuda"):
    """A synth.TokenBatch as explicit device tokens and candidate embeddings (int8
    codes stay codes, with bf16 candidates)."""
    if tb.emb.dtype == np.int8:
        dtype = T.I8
    td = T.torch_dtype(dtype)
    tok = T.DeviceTokens(
        emb=torch.from_numpy(tb.emb).to(device=device, dtype=td).contiguous(),
        act=torch.from_numpy(tb.act).to(device).contiguous(),
        time=None if tb.time is None else torch.from_numpy(tb.time).to(device).contiguous(),
        valid_len=torch.from_numpy(tb.valid_len).to(device).contiguous(), dtype=dtype)
    cand = torch.from_numpy(tb.cand).to(device=device, dtype=T.cand_dtype(dtype)).contiguous()
    return tok, cand


def oracle_encode_tokens(tb, W, ids=None, causal=True, chunk=4):
    """oracle.encode on explicit tokens for the candidates in ids (all by
    default), in parallel chunks; rows outside ids are 0."""
    ids = np.arange(tb.total) if ids is None else np.asarray(ids, dtype=np.int64)
    out = np.zeros((tb.total, 2 * W.d_model), dtype=np.float64)
    time = tb.time if tb.time is not None else np.zeros_like(tb.act)
    emb = oracle.dequantise(tb.emb) if tb.emb.dtype == np.int8 else tb.emb

    def one(part):
        o = oracle.encode(emb, tb.act, time, tb.valid_len, tb.cand, W, only=part,
                          chunk=chunk, causal=causal)
        return part, o[part]

    for part, o in parallel_map(one, chunks(ids, chunk)):
        out[part] = o
    return out
