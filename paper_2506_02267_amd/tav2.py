"""Thin Python binding of libtav2 (the C ABI in include/tav2.h).

Argument marshalling only: every step of the NN-select + encode path runs in
the library's HIP kernels.  torch supplies device memory and the stream.  The
binding refuses to run when the library is not built (no CPU fallback).
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_int32, c_int64, c_size_t, c_void_p
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np
import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtav2.so")

F32, BF16, I8 = 0, 1, 2
MASK_CAUSAL, MASK_NONE = 0, 1
K_MAX, T_MAX = 1024, 2048
STATUS = {0: "ok", -1: "null", -2: "shape", -3: "dtype", -4: "unsupported", -5: "workspace",
          -6: "hip", -7: "too_large"}


class Seq(ctypes.Structure):
    _fields_ = [("emb", c_void_p), ("action_type", c_void_p), ("time_bucket", c_void_p),
                ("offset", c_void_p), ("len", c_void_p), ("num_requests", c_int32),
                ("d", c_int32), ("dtype", c_int32), ("max_len", c_int32)]


class Cands(ctypes.Structure):
    _fields_ = [("emb", c_void_p), ("offset", c_void_p), ("total", c_int64),
                ("max_count", c_int32), ("reserved", c_int32)]


class Tokens(ctypes.Structure):
    _fields_ = [("emb", c_void_p), ("action_type", c_void_p), ("time_bucket", c_void_p),
                ("valid_len", c_void_p), ("total", c_int64), ("T", c_int32), ("d", c_int32),
                ("dtype", c_int32), ("reserved", c_int32)]


class Eq2(ctypes.Structure):
    _fields_ = [("rt", POINTER(Seq)), ("r", c_int32), ("k_rt", c_int32), ("imp", POINTER(Seq)),
                ("k_imp", c_int32), ("reserved", c_int32)]


class Layer(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("W_qkv", "b_qkv", "W_o", "b_o", "ln1_g", "ln1_b",
                                        "W_1", "b_1", "W_2", "b_2", "ln2_g", "ln2_b")]


class Weights(ctypes.Structure):
    _fields_ = [("d_in", c_int32), ("d_model", c_int32), ("n_heads", c_int32),
                ("d_ffn", c_int32), ("n_layers", c_int32), ("max_pos", c_int32),
                ("dtype", c_int32), ("reserved", c_int32), ("W_in", c_void_p),
                ("b_in", c_void_p), ("E_act", c_void_p), ("E_time", c_void_p),
                ("E_pos", c_void_p), ("layers", POINTER(Layer)), ("W_pool", c_void_p),
                ("b_pool", c_void_p), ("packed", c_void_p), ("packed_bytes", ctypes.c_uint64)]


class BatcherConfig(ctypes.Structure):
    _fields_ = [("dtype", c_int32), ("d", c_int32), ("has_time", c_int32),
                ("max_requests", c_int32), ("max_rows", ctypes.c_int64),
                ("max_rt_rows", ctypes.c_int64), ("max_cands", ctypes.c_int64)]


class Request(ctypes.Structure):
    _fields_ = [("emb", c_void_p), ("action_type", c_void_p), ("time_bucket", c_void_p),
                ("len", c_int32), ("rt_len", c_int32), ("rt_emb", c_void_p),
                ("rt_action_type", c_void_p), ("rt_time_bucket", c_void_p),
                ("cand_emb", c_void_p), ("n_cands", c_int32), ("reserved", c_int32)]


FUNCTIONS = {
    "tav2_status_string": (ctypes.c_char_p, [c_int32]),
    "tav2_abi_version": (c_int32, []),
    "tav2_nn_select_workspace": (c_size_t, [POINTER(Seq), POINTER(Cands), c_int32]),
    "tav2_nn_select": (c_int32, [POINTER(Seq), POINTER(Cands), c_int32, c_void_p, c_void_p,
                                 c_void_p, c_size_t, c_void_p]),
    "tav2_scratch_bytes": (c_size_t, []),
    "tav2_nn_select_noalloc": (c_int32, [POINTER(Seq), POINTER(Cands), c_int32, c_void_p,
                                         c_void_p, c_void_p]),
    "tav2_gather": (c_int32, [POINTER(Seq), POINTER(Seq), POINTER(Cands), c_void_p, c_int32,
                              c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]),
    "tav2_encode_workspace": (c_size_t, [POINTER(Tokens), POINTER(Weights)]),
    "tav2_pack_weights_bytes": (c_size_t, [POINTER(Weights)]),
    "tav2_pack_weights": (c_int32, [POINTER(Weights), c_void_p, c_size_t, c_void_p]),
    "tav2_encode": (c_int32, [POINTER(Tokens), c_void_p, POINTER(Weights), ctypes.c_uint32,
                              c_void_p, c_void_p, c_size_t, c_void_p]),
    "tav2_select_encode_workspace": (c_size_t, [POINTER(Seq), POINTER(Seq), POINTER(Cands),
                                                c_int32, POINTER(Weights)]),
    "tav2_select_encode": (c_int32, [POINTER(Seq), POINTER(Seq), POINTER(Cands), c_int32,
                                     POINTER(Weights), ctypes.c_uint32, c_void_p, c_void_p,
                                     c_void_p, c_void_p, c_size_t, c_void_p]),
    "tav2_select_encode_eq2_workspace": (c_size_t, [POINTER(Seq), POINTER(Eq2), POINTER(Cands),
                                                    c_int32, POINTER(Weights)]),
    "tav2_select_encode_eq2": (c_int32, [POINTER(Seq), POINTER(Eq2), POINTER(Cands), c_int32,
                                         POINTER(Weights), ctypes.c_uint32, c_void_p, c_void_p,
                                         c_void_p, c_void_p, c_size_t, c_void_p]),
    "tav2_batcher_create": (c_int32, [POINTER(BatcherConfig), POINTER(c_void_p)]),
    "tav2_batcher_destroy": (None, [c_void_p]),
    "tav2_batcher_arena_bytes": (c_size_t, [c_void_p]),
    "tav2_batcher_reset": (c_int32, [c_void_p]),
    "tav2_batcher_add": (c_int32, [c_void_p, POINTER(Request)]),
    "tav2_batcher_upload": (c_int32, [c_void_p, c_void_p]),
    "tav2_batcher_views": (c_int32, [c_void_p, POINTER(Seq), POINTER(Seq), POINTER(Cands)]),
    "tav2_profile_enable": (c_int32, [c_int32, ctypes.c_char_p]),
    "tav2_profile_report": (ctypes.c_int64, [ctypes.c_char_p, c_size_t]),
}

_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libtav2.so (built by paper_2506_02267_amd.build); raises if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2506_02267_amd.build` (there is no CPU fallback)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in FUNCTIONS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class Tav2Error(RuntimeError):
    def __init__(self, fn: str, status: int):
        msg = load_library().tav2_status_string(status).decode()
        super().__init__(f"{fn} returned {status} ({msg})")
        self.status = status


def _check(fn: str, status: int):
    if status != 0:
        raise Tav2Error(fn, status)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_handle(stream: Optional[torch.cuda.Stream]):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _used_on(stream: Optional[torch.cuda.Stream], *tensors):
    """Tell torch's caching allocator that tensors allocated on the current stream
    are in use on `stream` (a temporary workspace dropped on return must not be
    handed out again before the kernels reading it on `stream` have finished)."""
    if stream is None or stream == torch.cuda.current_stream():
        return
    for t in tensors:
        if t is not None:
            t.record_stream(stream)


def torch_dtype(dtype: int):
    """Storage type of a sequence of this dtype (int8 codes for I8)."""
    return {BF16: torch.bfloat16, I8: torch.int8}.get(dtype, torch.float32)


def cand_dtype(dtype: int):
    """Storage type of the candidates that go with a sequence of this dtype."""
    return torch.bfloat16 if dtype in (BF16, I8) else torch.float32


def _dev(a, dtype, device) -> torch.Tensor:
    t = torch.as_tensor(np.ascontiguousarray(a))
    return t.to(device=device, dtype=dtype).contiguous()


# ------------------------------------------------------------------ device containers
@dataclass
class DeviceSeq:
    """A de-duplicated request-level sequence batch resident on the GPU."""
    emb: torch.Tensor
    act: torch.Tensor
    time: Optional[torch.Tensor]
    offset: torch.Tensor
    length: torch.Tensor
    max_len: int
    dtype: int

    @classmethod
    def from_host(cls, s, dtype: int, device="cuda"):
        """From any object with emb/act/time/offset/length arrays (host)."""
        length = np.asarray(s.length, dtype=np.int32)
        return cls(emb=_dev(s.emb, torch_dtype(dtype), device),
                   act=_dev(s.act, torch.uint8, device),
                   time=None if s.time is None else _dev(s.time, torch.uint8, device),
                   offset=_dev(s.offset, torch.int64, device),
                   length=_dev(length, torch.int32, device),
                   max_len=int(length.max()) if length.size else 0, dtype=dtype)

    def struct(self) -> Seq:
        return Seq(emb=self.emb.data_ptr() if self.emb.numel() else None,
                   action_type=self.act.data_ptr(),
                   time_bucket=None if self.time is None else self.time.data_ptr(),
                   offset=self.offset.data_ptr(), len=self.length.data_ptr(),
                   num_requests=int(self.offset.shape[0]), d=int(self.emb.shape[1]),
                   dtype=self.dtype, max_len=self.max_len)


@dataclass
class DeviceCands:
    emb: torch.Tensor
    offset: torch.Tensor
    max_count: int

    @classmethod
    def from_host(cls, cand, cand_offset, dtype: int, device="cuda"):
        off = np.asarray(cand_offset, dtype=np.int64)
        counts = np.diff(off)
        return cls(emb=_dev(cand, cand_dtype(dtype), device), offset=_dev(off, torch.int64, device),
                   max_count=int(counts.max()) if counts.size else 0)

    @property
    def total(self) -> int:
        return int(self.emb.shape[0])

    def struct(self) -> Cands:
        return Cands(emb=self.emb.data_ptr() if self.total else None,
                     offset=self.offset.data_ptr(), total=self.total, max_count=self.max_count,
                     reserved=0)


@dataclass
class DeviceTokens:
    emb: torch.Tensor         # [total, T, d]
    act: torch.Tensor         # [total, T] uint8
    time: Optional[torch.Tensor]
    valid_len: torch.Tensor   # [total] int32
    dtype: int

    def struct(self) -> Tokens:
        total, T, d = self.emb.shape
        return Tokens(emb=self.emb.data_ptr(), action_type=self.act.data_ptr(),
                      time_bucket=None if self.time is None else self.time.data_ptr(),
                      valid_len=self.valid_len.data_ptr(), total=total, T=T, d=d,
                      dtype=self.dtype, reserved=0)


class DeviceWeights:
    """Encoder weights on the GPU (matrices/tables in the compute dtype, vectors fp32).

    pack=True also packs them once (tav2_pack_weights) and points the struct at
    the packed copy, so that later calls skip the packing step.
    """

    def __init__(self, w, device="cuda", pack=False):
        self.dtype = BF16 if w.dtype == "bf16" else F32
        md = torch_dtype(self.dtype)
        f32 = torch.float32
        self.keep: List[torch.Tensor] = []

        def m(a):
            t = _dev(a, md, device)
            self.keep.append(t)
            return t.data_ptr()

        def v(a):
            t = _dev(a, f32, device)
            self.keep.append(t)
            return t.data_ptr()

        self.layers = (Layer * len(w.layers))()
        for i, L in enumerate(w.layers):
            self.layers[i] = Layer(W_qkv=m(L.W_qkv), b_qkv=v(L.b_qkv), W_o=m(L.W_o), b_o=v(L.b_o),
                                   ln1_g=v(L.ln1_g), ln1_b=v(L.ln1_b), W_1=m(L.W_1), b_1=v(L.b_1),
                                   W_2=m(L.W_2), b_2=v(L.b_2), ln2_g=v(L.ln2_g), ln2_b=v(L.ln2_b))
        self.s = Weights(d_in=w.d_in, d_model=w.d_model, n_heads=w.n_heads, d_ffn=w.d_ffn,
                         n_layers=len(w.layers), max_pos=w.max_pos, dtype=self.dtype, reserved=0,
                         W_in=m(w.W_in), b_in=v(w.b_in), E_act=m(w.E_act),
                         E_time=None if w.E_time is None else m(w.E_time), E_pos=m(w.E_pos),
                         layers=self.layers, W_pool=m(w.W_pool), b_pool=v(w.b_pool),
                         packed=None, packed_bytes=0)
        self.d_model = w.d_model
        self.packed: Optional[torch.Tensor] = None
        if pack:
            self.pack()

    def pack(self, stream=None):
        """Pack the matrices once into a device buffer the struct then refers to."""
        lib = load_library()
        self.s.packed, self.s.packed_bytes = None, 0
        need = lib.tav2_pack_weights_bytes(ctypes.byref(self.s))
        if need == 0:
            return self
        buf = torch.empty(need + 256, dtype=torch.uint8, device=self.keep[0].device)
        p = buf.data_ptr()
        off = (-p) % 256
        _check("tav2_pack_weights", lib.tav2_pack_weights(ctypes.byref(self.s),
                                                          ctypes.c_void_p(p + off), need,
                                                          _stream_handle(stream)))
        self.packed = buf
        self.s.packed, self.s.packed_bytes = p + off, need
        return self


class Workspace:
    """A reusable, 256-byte-aligned device buffer (allocated outside the hot path)."""

    def __init__(self, device="cuda"):
        self.device = device
        self.buf: Optional[torch.Tensor] = None

    def get(self, nbytes: int):
        if nbytes == 0:
            return None, 0
        if self.buf is None or self.buf.numel() < nbytes + 256:
            self.buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        p = self.buf.data_ptr()
        off = (-p) % 256
        return ctypes.c_void_p(p + off), self.buf.numel() - off


# ------------------------------------------------------------------ entry points
def nn_select_workspace(seq: DeviceSeq, cands: DeviceCands, k: int) -> int:
    lib = load_library()
    return lib.tav2_nn_select_workspace(ctypes.byref(seq.struct()), ctypes.byref(cands.struct()), k)


def nn_select(seq: DeviceSeq, cands: DeviceCands, k: int, out_idx=None, out_score=None,
              ws: Optional[Workspace] = None, stream=None):
    lib = load_library()
    s, c = seq.struct(), cands.struct()
    dev = seq.emb.device
    if out_idx is None:
        out_idx = torch.empty((cands.total, k), dtype=torch.int32, device=dev)
    if out_score is None:
        out_score = torch.empty((cands.total, k), dtype=torch.float32, device=dev)
    ws = ws or Workspace(dev)
    need = lib.tav2_nn_select_workspace(ctypes.byref(s), ctypes.byref(c), k)
    wp, wb = ws.get(need)
    _check("tav2_nn_select", lib.tav2_nn_select(ctypes.byref(s), ctypes.byref(c), k,
                                                _ptr(out_idx), _ptr(out_score), wp, wb,
                                                _stream_handle(stream)))
    _used_on(stream, ws.buf, out_idx, out_score)
    return out_idx, out_score


def nn_select_noalloc(seq: DeviceSeq, cands: DeviceCands, k: int, out_idx: torch.Tensor,
                      out_score: torch.Tensor, stream=None):
    """tav2_nn_select_noalloc: the NN search with the library's static scratch
    (the caller passes the outputs; nothing is allocated)."""
    lib = load_library()
    s, c = seq.struct(), cands.struct()
    _check("tav2_nn_select_noalloc", lib.tav2_nn_select_noalloc(
        ctypes.byref(s), ctypes.byref(c), k, _ptr(out_idx), _ptr(out_score),
        _stream_handle(stream)))
    return out_idx, out_score


def gather(seq: DeviceSeq, rt: Optional[DeviceSeq], cands: DeviceCands, idx: torch.Tensor,
           k: int, stream=None) -> DeviceTokens:
    lib = load_library()
    s, c = seq.struct(), cands.struct()
    r = rt.struct() if rt is not None else None
    T = k + (rt.max_len if rt is not None else 0)
    dev = seq.emb.device
    d = int(seq.emb.shape[1])
    emb = torch.empty((cands.total, T, d), dtype=seq.emb.dtype, device=dev)
    act = torch.empty((cands.total, T), dtype=torch.uint8, device=dev)
    tim = torch.empty((cands.total, T), dtype=torch.uint8, device=dev) if seq.time is not None else None
    valid = torch.empty(cands.total, dtype=torch.int32, device=dev)
    _check("tav2_gather", lib.tav2_gather(ctypes.byref(s), ctypes.byref(r) if r is not None else None,
                                          ctypes.byref(c), _ptr(idx), k, _ptr(emb), _ptr(act),
                                          _ptr(tim), _ptr(valid), _stream_handle(stream)))
    _used_on(stream, emb, act, tim, valid)
    return DeviceTokens(emb=emb, act=act, time=tim, valid_len=valid, dtype=seq.dtype)


def encode(tokens: DeviceTokens, cand_emb: torch.Tensor, w: DeviceWeights, out=None,
           ws: Optional[Workspace] = None, stream=None, flags: int = MASK_CAUSAL) -> torch.Tensor:
    lib = load_library()
    t = tokens.struct()
    dev = tokens.emb.device
    if out is None:
        out = torch.empty((t.total, 2 * w.d_model), dtype=torch.float32, device=dev)
    ws = ws or Workspace(dev)
    need = lib.tav2_encode_workspace(ctypes.byref(t), ctypes.byref(w.s))
    wp, wb = ws.get(need)
    _check("tav2_encode", lib.tav2_encode(ctypes.byref(t), _ptr(cand_emb), ctypes.byref(w.s),
                                          flags, _ptr(out), wp, wb, _stream_handle(stream)))
    _used_on(stream, ws.buf, out)
    return out


def select_encode_workspace(seq: DeviceSeq, rt: Optional[DeviceSeq], cands: DeviceCands, k: int,
                            w: DeviceWeights) -> int:
    lib = load_library()
    r = rt.struct() if rt is not None else None
    return lib.tav2_select_encode_workspace(ctypes.byref(seq.struct()),
                                            ctypes.byref(r) if r is not None else None,
                                            ctypes.byref(cands.struct()), k, ctypes.byref(w.s))


class SelectEncode:
    """Prepared call of tav2_select_encode: structs, outputs and workspace built once."""

    def __init__(self, seq: DeviceSeq, rt: Optional[DeviceSeq], cands: DeviceCands, k: int,
                 w: DeviceWeights, flags: int = MASK_CAUSAL):
        self.lib = load_library()
        self.seq, self.rt, self.cands, self.k, self.w = seq, rt, cands, k, w
        self.flags = flags
        self.s, self.c = seq.struct(), cands.struct()
        self.r = rt.struct() if rt is not None else None
        dev = seq.emb.device
        self.idx = torch.empty((cands.total, k), dtype=torch.int32, device=dev)
        self.score = torch.empty((cands.total, k), dtype=torch.float32, device=dev)
        self.out = torch.empty((cands.total, 2 * w.d_model), dtype=torch.float32, device=dev)
        need = select_encode_workspace(seq, rt, cands, k, w)
        if need == 0 and cands.total > 0:
            # the size query returns 0 for invalid arguments; let the call report why
            need = 1
        self.ws = Workspace(dev)
        self.wp, self.wb = self.ws.get(need)

    def __call__(self, stream=None):
        _check("tav2_select_encode", self.lib.tav2_select_encode(
            ctypes.byref(self.s), ctypes.byref(self.r) if self.r is not None else None,
            ctypes.byref(self.c), self.k, ctypes.byref(self.w.s), self.flags, _ptr(self.idx),
            _ptr(self.score), _ptr(self.out), self.wp, self.wb, _stream_handle(stream)))
        return self.idx, self.score, self.out


class SelectEncodeEq2:
    """Prepared call of tav2_select_encode_eq2 (Eq. 2's four parts): structs,
    outputs [total, k + k_rt + k_imp] and workspace built once."""

    def __init__(self, seq: DeviceSeq, rt: Optional[DeviceSeq], r: int, k_rt: int,
                 imp: Optional[DeviceSeq], k_imp: int, cands: DeviceCands, k: int,
                 w: DeviceWeights, flags: int = MASK_CAUSAL):
        self.lib = load_library()
        self.args = (seq, rt, imp, cands, w)
        self.s, self.c = seq.struct(), cands.struct()
        self.r_s = rt.struct() if rt is not None else None
        self.i_s = imp.struct() if imp is not None else None
        self.e = Eq2(rt=ctypes.pointer(self.r_s) if self.r_s is not None else None, r=r,
                     k_rt=k_rt, imp=ctypes.pointer(self.i_s) if self.i_s is not None else None,
                     k_imp=k_imp, reserved=0)
        self.k, self.w, self.flags = k, w, flags
        dev = seq.emb.device
        K = k + k_rt + k_imp
        self.idx = torch.empty((cands.total, K), dtype=torch.int32, device=dev)
        self.score = torch.empty((cands.total, K), dtype=torch.float32, device=dev)
        self.out = torch.empty((cands.total, 2 * w.d_model), dtype=torch.float32, device=dev)
        need = self.lib.tav2_select_encode_eq2_workspace(ctypes.byref(self.s), ctypes.byref(self.e),
                                                         ctypes.byref(self.c), k,
                                                         ctypes.byref(w.s))
        if need == 0 and cands.total > 0:
            need = 1   # invalid arguments: the call reports why
        self.ws = Workspace(dev)
        self.wp, self.wb = self.ws.get(need)

    def __call__(self, stream=None):
        _check("tav2_select_encode_eq2", self.lib.tav2_select_encode_eq2(
            ctypes.byref(self.s), ctypes.byref(self.e), ctypes.byref(self.c), self.k,
            ctypes.byref(self.w.s), self.flags, _ptr(self.idx), _ptr(self.score), _ptr(self.out),
            self.wp, self.wb, _stream_handle(stream)))
        return self.idx, self.score, self.out


def profile_enable(on: bool, site: Optional[str] = None):
    """Bracket the library's launches (all, or one site) with HIP events."""
    load_library().tav2_profile_enable(1 if on else 0, site.encode() if site else None)


def profile_report() -> dict:
    """{site: (launches, total_ms)} since the last report; call after synchronising."""
    lib = load_library()
    buf = ctypes.create_string_buffer(1 << 16)
    n = lib.tav2_profile_report(buf, len(buf))
    if n >= len(buf):
        raise RuntimeError("profile report truncated")
    out = {}
    for line in buf.value.decode().splitlines():
        name, cnt, ms = line.split()
        out[name] = (int(cnt), float(ms))
    return out


def select_encode(seq, rt, cands, k, w, stream=None, flags: int = MASK_CAUSAL):
    return SelectEncode(seq, rt, cands, k, w, flags)(stream)


class Batcher:
    """A tav2_batcher: pinned host arena + device mirror of one mini-batch.

    add() takes host numpy arrays in the storage layout (bf16 as uint16 bits, int8
    codes, float32) and returns False when the request does not fit the mini-batch."""

    TOO_LARGE = -7

    def __init__(self, dtype: int, d: int, has_time: bool, max_requests: int, max_rows: int,
                 max_rt_rows: int, max_cands: int):
        self.lib = load_library()
        self.cfg = BatcherConfig(dtype=dtype, d=d, has_time=int(has_time),
                                 max_requests=max_requests, max_rows=max_rows,
                                 max_rt_rows=max_rt_rows, max_cands=max_cands)
        h = c_void_p()
        _check("tav2_batcher_create", self.lib.tav2_batcher_create(ctypes.byref(self.cfg),
                                                                   ctypes.byref(h)))
        self.h = h

    @property
    def arena_bytes(self) -> int:
        return int(self.lib.tav2_batcher_arena_bytes(self.h))

    def reset(self):
        _check("tav2_batcher_reset", self.lib.tav2_batcher_reset(self.h))

    def add(self, emb, act, time=None, rt_emb=None, rt_act=None, rt_time=None, cand=None) -> bool:
        a = lambda x: None if x is None else x.ctypes.data
        q = Request(emb=a(emb), action_type=a(act), time_bucket=a(time),
                    len=0 if emb is None else int(emb.shape[0]),
                    rt_len=0 if rt_emb is None else int(rt_emb.shape[0]), rt_emb=a(rt_emb),
                    rt_action_type=a(rt_act), rt_time_bucket=a(rt_time), cand_emb=a(cand),
                    n_cands=0 if cand is None else int(cand.shape[0]), reserved=0)
        st = self.lib.tav2_batcher_add(self.h, ctypes.byref(q))
        if st == self.TOO_LARGE:
            return False
        _check("tav2_batcher_add", st)
        return True

    def upload(self, stream=None):
        _check("tav2_batcher_upload", self.lib.tav2_batcher_upload(self.h, _stream_handle(stream)))

    def views(self):
        """(Seq, Seq, Cands) structs of the uploaded mini-batch on the device."""
        s, r, c = Seq(), Seq(), Cands()
        _check("tav2_batcher_views", self.lib.tav2_batcher_views(self.h, ctypes.byref(s),
                                                                 ctypes.byref(r), ctypes.byref(c)))
        return s, r, c

    def close(self):
        if getattr(self, "h", None):
            self.lib.tav2_batcher_destroy(self.h)
            self.h = None

    def __del__(self):
        self.close()


def select_encode_structs(s: Seq, r: Optional[Seq], c: Cands, k: int, w: DeviceWeights,
                          out_idx: torch.Tensor, out_score: torch.Tensor, out: torch.Tensor,
                          ws: Workspace, stream=None, flags: int = MASK_CAUSAL):
    """tav2_select_encode on raw structs (e.g. a batcher's views); outputs
    preallocated by the caller with at least c.total rows."""
    lib = load_library()
    rp = ctypes.byref(r) if r is not None else None
    need = lib.tav2_select_encode_workspace(ctypes.byref(s), rp, ctypes.byref(c), k,
                                            ctypes.byref(w.s))
    wp, wb = ws.get(max(need, 1))
    _check("tav2_select_encode", lib.tav2_select_encode(
        ctypes.byref(s), rp, ctypes.byref(c), k, ctypes.byref(w.s), flags, _ptr(out_idx),
        _ptr(out_score), _ptr(out), wp, wb, _stream_handle(stream)))
    _used_on(stream, ws.buf, out_idx, out_score, out)
