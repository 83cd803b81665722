"""The serving-side batcher (pinned arena, de-duplicated mini-batches, one
host-to-device copy; Sec. 3.4.2) against the device-resident path: the same
requests collated by the batcher give the same indices, scores and encoder
outputs bit for bit, including across dynamically formed mini-batches."""
import numpy as np
import pytest
import torch

import synth
from helpers import upload
from paper_2506_02267_amd import tav2 as T

pytestmark = pytest.mark.gpu


def host_bytes(a, dtype):
    """A float32 / int8 host array in the storage layout of `dtype`."""
    if dtype == T.BF16:
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).view(
            torch.int16).numpy()
    return np.ascontiguousarray(a)


def requests_of(inp, dt):
    """Per request: (emb, act, time, rt_emb, rt_act, rt_time, cand) host arrays."""
    out = []
    for r in range(inp.seq.R):
        a, L = int(inp.seq.offset[r]), int(inp.seq.length[r])
        s = slice(a, a + L)
        q = dict(emb=host_bytes(inp.seq.emb[s], dt), act=np.ascontiguousarray(inp.seq.act[s]),
                 time=None if inp.seq.time is None else np.ascontiguousarray(inp.seq.time[s]))
        if inp.rt is not None:
            b, m = int(inp.rt.offset[r]), int(inp.rt.length[r])
            t = slice(b, b + m)
            q.update(rt_emb=host_bytes(inp.rt.emb[t], dt), rt_act=np.ascontiguousarray(inp.rt.act[t]),
                     rt_time=None if inp.rt.time is None else np.ascontiguousarray(inp.rt.time[t]))
        c0, c1 = int(inp.cand_offset[r]), int(inp.cand_offset[r + 1])
        q["cand"] = host_bytes(inp.cand[c0:c1], T.BF16 if dt in (T.BF16, T.I8) else T.F32)
        out.append(q)
    return out


def direct(inp, w, dw):
    seq, rt, cands = upload(inp)
    idx, score, out = T.select_encode(seq, rt, cands, w.k, dw)
    torch.cuda.synchronize()
    return idx.cpu(), score.cpu(), out.cpu()


def run_batches(inp, w, dw, dt, cap_rows, cap_cands):
    """Requests in order through one batcher, a new mini-batch whenever the next one
    does not fit; outputs concatenated in request order."""
    b = T.Batcher(dt, w.d, w.has_time, max_requests=64, max_rows=cap_rows,
                  max_rt_rows=max(1, 64 * w.rt_len), max_cands=cap_cands)
    ws = T.Workspace(torch.device("cuda"))
    outs, batches = [], 0

    def flush():
        nonlocal batches
        b.upload()
        s, r, c = b.views()
        n = c.total
        oi = torch.empty((n, w.k), dtype=torch.int32, device="cuda")
        osc = torch.empty((n, w.k), dtype=torch.float32, device="cuda")
        oo = torch.empty((n, 2 * w.d_model), dtype=torch.float32, device="cuda")
        T.select_encode_structs(s, r if w.rt_len else None, c, w.k, dw, oi, osc, oo, ws)
        torch.cuda.synchronize()
        outs.append((oi.cpu(), osc.cpu(), oo.cpu()))
        batches += 1
        b.reset()

    for q in requests_of(inp, dt):
        if not b.add(**q):
            flush()
            assert b.add(**q)
    flush()
    b.close()
    return tuple(torch.cat([o[i] for o in outs]) for i in range(3)), batches


@pytest.mark.parametrize("name", ["paper_i8", "paper_bf16"])
def test_batcher_equals_device_resident_path(name):
    w = synth.scaled(synth.BY_NAME[name], R=6, L=None, L_range=(2000, 9000), N=24)
    inp = synth.make_inputs(w)
    W = synth.make_weights(w)
    dw = T.DeviceWeights(W)
    dt = T.I8 if w.dtype == "i8" else T.BF16
    print(f"batcher {name}: {w.R} requests", flush=True)
    ref = direct(inp, w, dw)
    got, nb = run_batches(inp, w, dw, dt, cap_rows=64 * 9000, cap_cands=64 * 24)
    assert nb == 1
    for a, b in zip(got, ref):
        assert torch.equal(a, b)


def test_dynamic_batches_equal_one_batch():
    """Capacities of about two requests: the six requests go through three or more
    mini-batches of the same batcher (reset and reused), with the same results."""
    w = synth.scaled(synth.PAPER_I8, R=6, L=None, L_range=(2000, 9000), N=24)
    inp = synth.make_inputs(w)
    dw = T.DeviceWeights(synth.make_weights(w))
    ref = direct(inp, w, dw)
    got, nb = run_batches(inp, w, dw, T.I8, cap_rows=18000, cap_cands=48)
    print(f"  {nb} mini-batches", flush=True)
    assert nb >= 3
    for a, b in zip(got, ref):
        assert torch.equal(a, b)


def test_sealed_after_upload_and_reupload():
    w = synth.scaled(synth.PAPER_I8, R=2, L=3000, N=8)
    inp = synth.make_inputs(w)
    qs = requests_of(inp, T.I8)
    b = T.Batcher(T.I8, w.d, True, 4, 10000, 1000, 64)
    assert b.add(**qs[0])
    b.upload()
    with pytest.raises(T.Tav2Error) as e:
        b.add(**qs[1])
    assert e.value.status == -2
    b.upload()   # the same bytes again
    s, r, c = b.views()
    assert (s.num_requests, c.total, s.max_len) == (1, 8, 3000)
    torch.cuda.synchronize()
    b.reset()
    with pytest.raises(T.Tav2Error):
        b.views()   # nothing uploaded since the reset
    assert b.add(**qs[1]) and b.add(**qs[0]) and b.add(**qs[1])
    assert not b.add(**qs[0])   # 10000 rows hold three requests of 3000
    b.close()
