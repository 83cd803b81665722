"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/tav2.h declares, its structs match the binding's
layout, workspace queries are pure host arithmetic, and every argument error
is reported before anything is launched."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2506_02267_amd import tav2 as T

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tav2.h")

FAKE = 0x10000   # an aligned non-null "device" address; never dereferenced on error paths


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b(tav2_\w+)\s*\(",
                                 text, flags=re.M)))


def test_library_exports_every_declared_function():
    lib = T.load_library()
    names = declared_functions()
    assert len(names) >= 9
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(T.FUNCTIONS), "binding and header disagree"
    out = subprocess.run(["nm", "-D", "--defined-only", T.LIB_PATH], capture_output=True,
                         text=True).stdout
    for n in names:
        assert re.search(rf"\bT {n}$", out, flags=re.M), n


def test_struct_layouts_match_header(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "tav2.h"\n'
                   'int main(void){printf("%zu %zu %zu %zu %zu %zu %zu %zu\\n",'
                   'sizeof(tav2_seq), sizeof(tav2_cands), sizeof(tav2_tokens),'
                   'sizeof(tav2_layer), sizeof(tav2_weights), offsetof(tav2_seq, max_len),'
                   'offsetof(tav2_weights, layers), offsetof(tav2_tokens, total));return 0;}\n')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o",
                    str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    want = [ctypes.sizeof(T.Seq), ctypes.sizeof(T.Cands), ctypes.sizeof(T.Tokens),
            ctypes.sizeof(T.Layer), ctypes.sizeof(T.Weights), T.Seq.max_len.offset,
            T.Weights.layers.offset, T.Tokens.total.offset]
    assert got == want


def fake_seq(R=2, d=64, dtype=T.BF16, max_len=100, time=True):
    return T.Seq(emb=FAKE, action_type=FAKE, time_bucket=FAKE if time else None, offset=FAKE,
                 len=FAKE, num_requests=R, d=d, dtype=dtype, max_len=max_len)


def fake_cands(total=10, max_count=5):
    return T.Cands(emb=FAKE, offset=FAKE, total=total, max_count=max_count, reserved=0)


def fake_weights(d=64, dm=256, heads=4, ffn=512, layers=2, max_pos=64, dtype=T.BF16, time=True):
    L = (T.Layer * layers)(*[T.Layer(*([FAKE] * 12)) for _ in range(layers)])
    w = T.Weights(d_in=d, d_model=dm, n_heads=heads, d_ffn=ffn, n_layers=layers,
                  max_pos=max_pos, dtype=dtype, reserved=0, W_in=FAKE, b_in=FAKE, E_act=FAKE,
                  E_time=FAKE if time else None, E_pos=FAKE, layers=L, W_pool=FAKE, b_pool=FAKE,
                  packed=None, packed_bytes=0)
    w._keep = L
    return w


def call_select(seq, cands, k, idx=FAKE, score=FAKE, ws=FAKE, wsb=1 << 40):
    lib = T.load_library()
    return lib.tav2_nn_select(ctypes.byref(seq) if seq is not None else None,
                              ctypes.byref(cands) if cands is not None else None, k, idx, score,
                              ws, wsb, None)


def test_workspace_queries():
    lib = T.load_library()
    s, c = fake_seq(max_len=1000), fake_cands(total=10)
    # scores: total x round_up(max_len, 64) fp32
    assert lib.tav2_nn_select_workspace(ctypes.byref(s), ctypes.byref(c), 16) == 10 * 1024 * 4
    assert lib.tav2_nn_select_workspace(ctypes.byref(s), ctypes.byref(c), 0) == 0
    w = fake_weights()
    tok = T.Tokens(emb=FAKE, action_type=FAKE, time_bucket=FAKE, valid_len=FAKE, total=10, T=64,
                   d=64, dtype=T.BF16, reserved=0)
    # fused bf16 encoder: every matrix in fragment order (W_in's token half padded to
    # 256 columns; each layer matrix followed by a 16-column bias block; the side
    # tables transposed: [E_act | E_time] in 80 columns, E_pos in max_pos rounded up
    # to 128), the candidate half of the input projection (fp32 per candidate) and,
    # past one 128-position block, a K / V cache of layers x 2 x T x d_model bf16
    dm, ff, layers = 256, 512, 2

    def packed(max_pos):
        pos_cols = -(-max_pos // 128) * 128
        per_layer = (3 * dm + dm + ff) * (dm + 16) + dm * (ff + 16)
        return (dm * 256 + dm * dm + layers * per_layer + dm * (80 + pos_cols)) * 2

    cvec = 10 * dm * 4
    assert lib.tav2_encode_workspace(ctypes.byref(tok), ctypes.byref(w)) == packed(64) + cvec
    w256 = fake_weights(max_pos=256)
    tok.T = 256
    assert (lib.tav2_encode_workspace(ctypes.byref(tok), ctypes.byref(w256))
            == packed(256) + cvec + 10 * layers * 2 * 256 * dm * 2)
    tok.T = 64
    wf = fake_weights(dm=64, heads=2, ffn=128, layers=1, max_pos=32, dtype=T.F32, time=False)
    tokf = T.Tokens(emb=FAKE, action_type=FAKE, time_bucket=None, valid_len=FAKE, total=16, T=32,
                    d=64, dtype=T.F32, reserved=0)
    assert lib.tav2_encode_workspace(ctypes.byref(tokf), ctypes.byref(wf)) == 0
    se = lib.tav2_select_encode_workspace(ctypes.byref(s), None, ctypes.byref(c), 64,
                                          ctypes.byref(w))
    assert se > lib.tav2_nn_select_workspace(ctypes.byref(s), ctypes.byref(c), 64)


@pytest.mark.parametrize("case,status", [
    ("null_seq", -1), ("null_cands", -1), ("k0", -2), ("k_big", -2), ("bad_dtype", -3),
    ("bad_d", -2), ("neg_R", -2), ("long_seq", -4), ("null_out", -1), ("small_ws", -5),
    ("null_ws", -5), ("misaligned_ws", -5), ("misaligned_emb", -2), ("count_gt_total", -2),
])
def test_nn_select_argument_errors(case, status):
    s, c = fake_seq(), fake_cands()
    kw = {}
    k = 8
    if case == "null_seq":
        s = None
    elif case == "null_cands":
        c = None
    elif case == "k0":
        k = 0
    elif case == "k_big":
        k = 1025
    elif case == "bad_dtype":
        s.dtype = 7
    elif case == "bad_d":
        s.d = 60
    elif case == "neg_R":
        s.num_requests = -1
    elif case == "long_seq":
        s.max_len = 40000
    elif case == "null_out":
        kw["idx"] = None
    elif case == "small_ws":
        kw["wsb"] = 16
    elif case == "null_ws":
        kw["ws"] = None
    elif case == "misaligned_ws":
        kw["ws"] = FAKE + 8
    elif case == "misaligned_emb":
        s.emb = FAKE + 2
    elif case == "count_gt_total":
        c.max_count = 11
    assert call_select(s, c, k, **kw) == status


def test_empty_candidate_set_is_a_no_op():
    assert call_select(fake_seq(), fake_cands(total=0, max_count=0), 8, idx=None, score=None,
                       ws=None, wsb=0) == 0


@pytest.mark.parametrize("case,status", [
    ("dtype_mismatch", -3), ("heads", -2), ("dm_unsupported", -4), ("ffn", -4),
    ("max_pos", -2), ("time_mismatch", -2), ("null_layer_ptr", -1), ("T_too_big", -2),
    ("f32_too_big", -4), ("null_out", -1), ("ws", -5), ("d_in", -2),
    ("flags", -2), ("unmasked_two_blocks", -4), ("packed_small", -5), ("packed_misaligned", -5),
    ("d_wide", -4), ("nine_layers", -4),
])
def test_encode_argument_errors(case, status):
    lib = T.load_library()
    w = fake_weights()
    tok = T.Tokens(emb=FAKE, action_type=FAKE, time_bucket=FAKE, valid_len=FAKE, total=10, T=64,
                   d=64, dtype=T.BF16, reserved=0)
    out, ws, wsb = FAKE, FAKE, 1 << 40
    if case == "dtype_mismatch":
        w.dtype = T.F32
    elif case == "heads":
        w.n_heads = 3
    elif case == "dm_unsupported":
        w.d_model, w.n_heads = 128, 2
    elif case == "ffn":
        w.d_ffn = 300
    elif case == "max_pos":
        w.max_pos = 63
    elif case == "time_mismatch":
        tok.time_bucket = None
    elif case == "null_layer_ptr":
        w.layers[1].W_2 = None
    elif case == "T_too_big":
        tok.T = 3000
        w.max_pos = 3000
    elif case == "f32_too_big":
        tok.dtype = T.F32
        w.dtype = T.F32
    elif case == "null_out":
        out = None
    elif case == "ws":       # T > 128 needs the K / V cache workspace
        tok.T = 256
        w.max_pos = 256
        wsb = 10
    elif case == "d_in":
        w.d_in = 32
    elif case == "d_wide":   # bf16 token embeddings wider than 256
        tok.d, w.d_in = 512, 512
    elif case == "nine_layers":
        w = fake_weights(layers=9)
    flags = T.MASK_CAUSAL
    if case == "flags":
        flags = 7
    elif case == "unmasked_two_blocks":   # bf16 unmasked: one block of 128 positions
        flags = T.MASK_NONE
        tok.T = 129
        w.max_pos = 129
    elif case == "packed_small":
        w.packed, w.packed_bytes = FAKE, 1024
    elif case == "packed_misaligned":
        w.packed, w.packed_bytes = FAKE + 16, 1 << 40
    st = lib.tav2_encode(ctypes.byref(tok), FAKE, ctypes.byref(w), flags, out, ws, wsb, None)
    assert st == status


def test_small_encoder_queries():
    """d_model 64 (bf16): the packed form is the kernel's LDS image of the weights
    (per layer: W_qkv, W_o and W_1 in rows of 72 bf16, W_2 in rows of FFN + 8, the
    eight vectors in fp32; then W_in's token half in rows of d + 8); a workspace of
    per-workgroup K / V caches past one 64-position block (layers x 2 x T padded
    to 64 x d_model bf16 per workgroup, one workgroup per candidate up to 256);
    the shapes whose weights outgrow the on-chip memory are unsupported."""
    lib = T.load_library()
    w = fake_weights(d=32, dm=64, heads=1, ffn=32, layers=2, max_pos=2048)
    per_layer = (3 * 64 * 72 + 64 * 72 + 32 * 72 + 64 * 40) * 2 + (9 * 64 + 32) * 4
    image = 2 * per_layer + 64 * 40 * 2
    assert lib.tav2_pack_weights_bytes(ctypes.byref(w)) == -(-image // 256) * 256
    tok = T.Tokens(emb=FAKE, action_type=FAKE, time_bucket=FAKE, valid_len=FAKE, total=10,
                   T=64, d=32, dtype=T.BF16, reserved=0)
    assert lib.tav2_encode_workspace(ctypes.byref(tok), ctypes.byref(w)) == 0
    tok.T = 192
    assert lib.tav2_encode_workspace(ctypes.byref(tok), ctypes.byref(w)) == 10 * 2 * 2 * 192 * 64 * 2
    tok.T, tok.total = 2000, 1000
    assert (lib.tav2_encode_workspace(ctypes.byref(tok), ctypes.byref(w))
            == 256 * 2 * 2 * 2048 * 64 * 2)
    # the unmasked mode: one block of 64 positions (then the missing output is reported)
    tok.T, tok.total = 64, 10
    assert lib.tav2_encode(ctypes.byref(tok), FAKE, ctypes.byref(w), T.MASK_NONE, None, FAKE,
                           1 << 40, None) == -1
    tok.T = 65
    assert lib.tav2_encode(ctypes.byref(tok), FAKE, ctypes.byref(w), T.MASK_NONE, FAKE, FAKE,
                           1 << 40, None) == -4
    for bad in (dict(layers=3), dict(ffn=64), dict(d=128), dict(ffn=48)):
        kw = dict(d=32, dm=64, heads=1, ffn=32, layers=2, max_pos=2048)
        kw.update(bad)
        wb = fake_weights(**kw)
        tok.T, tok.d = 64, kw["d"]
        assert lib.tav2_encode(ctypes.byref(tok), FAKE, ctypes.byref(wb), T.MASK_CAUSAL, FAKE,
                               FAKE, 1 << 40, None) == -4, bad


def test_int8_codes_feed_only_the_small_encoder():
    """int8 sequences (and int8 explicit tokens) go to the d_model-64 encoder with
    bf16 weights; d_model 256 reports unsupported, float32 weights a dtype error."""
    lib = T.load_library()
    s = fake_seq(R=1, d=32, dtype=T.I8, max_len=16384)
    c = fake_cands(total=10, max_count=10)
    small = fake_weights(d=32, dm=64, heads=1, ffn=32, layers=2, max_pos=128)
    assert lib.tav2_select_encode_workspace(ctypes.byref(s), None, ctypes.byref(c), 128,
                                            ctypes.byref(small)) > 0
    big = fake_weights(d=32, dm=256, heads=4, ffn=512, layers=2, max_pos=128)
    assert lib.tav2_select_encode_workspace(ctypes.byref(s), None, ctypes.byref(c), 128,
                                            ctypes.byref(big)) == 0
    call = lambda w: lib.tav2_select_encode(ctypes.byref(s), None, ctypes.byref(c), 128,
                                            ctypes.byref(w), T.MASK_CAUSAL, FAKE, FAKE, FAKE,
                                            FAKE, 1 << 40, None)
    assert call(big) == -4
    f32 = fake_weights(d=32, dm=64, heads=1, ffn=32, layers=2, max_pos=128, dtype=T.F32)
    assert call(f32) == -3
    tok = T.Tokens(emb=FAKE, action_type=FAKE, time_bucket=FAKE, valid_len=FAKE, total=10,
                   T=64, d=32, dtype=T.I8, reserved=0)
    assert lib.tav2_encode_workspace(ctypes.byref(tok), ctypes.byref(small)) == 0   # one block
    tok.T = 65
    assert lib.tav2_encode_workspace(ctypes.byref(tok), ctypes.byref(small)) > 0
    tok.T = 64
    enc = lambda w: lib.tav2_encode(ctypes.byref(tok), FAKE, ctypes.byref(w), T.MASK_CAUSAL,
                                    FAKE, FAKE, 1 << 40, None)
    assert enc(big) == -4
    assert enc(f32) == -3


def test_fp32_encoder_envelope():
    """float32 encoder: T <= 64, d_model <= 128, FFN <= 512, d <= 256, with d_model,
    the head width and the FFN width multiples of 4.  Shapes inside pass every check
    (the call then reports the missing output); shapes outside are unsupported."""
    lib = T.load_library()

    def enc(T_, d, dm, heads, ffn):
        w = fake_weights(d=d, dm=dm, heads=heads, ffn=ffn, layers=2, max_pos=128, dtype=T.F32)
        tok = T.Tokens(emb=FAKE, action_type=FAKE, time_bucket=FAKE, valid_len=FAKE, total=10,
                       T=T_, d=d, dtype=T.F32, reserved=0)
        return lib.tav2_encode(ctypes.byref(tok), FAKE, ctypes.byref(w), T.MASK_CAUSAL, None, FAKE,
                               1 << 40, None)

    assert enc(64, 256, 128, 4, 512) == -1    # the envelope's corner
    assert enc(17, 16, 32, 8, 36) == -1       # heads of 4
    assert enc(40, 48, 96, 3, 200) == -1
    assert enc(65, 256, 128, 4, 512) == -4    # T
    assert enc(64, 256, 132, 4, 512) == -4    # d_model
    assert enc(64, 256, 128, 4, 516) == -4    # FFN
    assert enc(64, 272, 128, 4, 512) == -4    # d
    assert enc(64, 64, 24, 4, 64) == -4       # heads of 6
    assert enc(64, 64, 64, 2, 130) == -4      # FFN not a multiple of 4


def test_unmasked_encoder_accepted_within_one_block():
    """TAV2_MASK_NONE passes the checks at T = 128 (the error then comes from the
    missing output), and for float32 at any supported T."""
    lib = T.load_library()
    w = fake_weights(max_pos=128)
    tok = T.Tokens(emb=FAKE, action_type=FAKE, time_bucket=FAKE, valid_len=FAKE, total=10,
                   T=128, d=64, dtype=T.BF16, reserved=0)
    assert lib.tav2_encode(ctypes.byref(tok), FAKE, ctypes.byref(w), T.MASK_NONE, None, FAKE,
                           1 << 40, None) == -1
    wf = fake_weights(dm=64, heads=2, ffn=128, layers=1, dtype=T.F32)
    tokf = T.Tokens(emb=FAKE, action_type=FAKE, time_bucket=FAKE, valid_len=FAKE, total=10,
                    T=64, d=64, dtype=T.F32, reserved=0)
    assert lib.tav2_encode(ctypes.byref(tokf), FAKE, ctypes.byref(wf), T.MASK_NONE, None, FAKE,
                           1 << 40, None) == -1


def test_packed_weights_queries_and_errors():
    lib = T.load_library()
    w = fake_weights()
    need = lib.tav2_pack_weights_bytes(ctypes.byref(w))
    assert need > 0 and need % 256 == 0
    tok = T.Tokens(emb=FAKE, action_type=FAKE, time_bucket=FAKE, valid_len=FAKE, total=10, T=64,
                   d=64, dtype=T.BF16, reserved=0)
    ws_unpacked = lib.tav2_encode_workspace(ctypes.byref(tok), ctypes.byref(w))
    w.packed, w.packed_bytes = FAKE, need
    # with packed weights the workspace no longer holds a packed copy
    assert lib.tav2_encode_workspace(ctypes.byref(tok), ctypes.byref(w)) == ws_unpacked - need
    assert lib.tav2_pack_weights(ctypes.byref(w), None, need, None) == -5
    assert lib.tav2_pack_weights(ctypes.byref(w), FAKE, need - 256, None) == -5
    assert lib.tav2_pack_weights(None, FAKE, need, None) == -1
    wf = fake_weights(dm=64, heads=2, ffn=128, layers=1, dtype=T.F32)
    assert lib.tav2_pack_weights_bytes(ctypes.byref(wf)) == 0
    assert lib.tav2_pack_weights(ctypes.byref(wf), None, 0, None) == 0   # nothing to pack


def test_select_encode_checks_realtime_and_positions():
    lib = T.load_library()
    s, c = fake_seq(d=64), fake_cands()
    rt = fake_seq(d=64, max_len=100)
    w = fake_weights(max_pos=64 + 99)
    st = lib.tav2_select_encode(ctypes.byref(s), ctypes.byref(rt), ctypes.byref(c), 64,
                                ctypes.byref(w), 0, FAKE, FAKE, FAKE, FAKE, 1 << 40, None)
    assert st == -2          # k + rt->max_len exceeds max_pos
    rt2 = fake_seq(R=3, d=64, max_len=10)
    st = lib.tav2_select_encode(ctypes.byref(s), ctypes.byref(rt2), ctypes.byref(c), 64,
                                ctypes.byref(fake_weights(max_pos=100)), 0, FAKE, FAKE, FAKE,
                                FAKE, 1 << 40, None)
    assert st == -2          # real-time batch with a different request count
    st = lib.tav2_select_encode(ctypes.byref(s), None, ctypes.byref(c), 64,
                                ctypes.byref(fake_weights(time=False)), 0, FAKE, FAKE, FAKE, FAKE,
                                1 << 40, None)
    assert st == -2          # sequence has time buckets, weights have no time table
    st = lib.tav2_select_encode(ctypes.byref(s), None, ctypes.byref(c), 64,
                                ctypes.byref(fake_weights(max_pos=200)), 2, FAKE, FAKE, FAKE,
                                FAKE, 1 << 40, None)
    assert st == -2          # unknown flags


def test_status_strings():
    lib = T.load_library()
    for code in range(-6, 1):
        assert lib.tav2_status_string(code).decode()
    assert lib.tav2_abi_version() >= 1


def test_int8_sequence_is_for_the_nn_search_only():
    """TAV2_I8 passes the NN search's argument checks (the error comes from the
    empty output pointer, i.e. after the dtype was accepted); gather, encode and
    select_encode refuse it as unsupported."""
    lib = T.load_library()
    s, c = fake_seq(dtype=T.I8, d=32), fake_cands()
    assert call_select(s, c, 8, idx=None) == -1
    assert lib.tav2_nn_select_workspace(ctypes.byref(s), ctypes.byref(c), 8) == 10 * 128 * 4
    st = lib.tav2_gather(ctypes.byref(s), None, ctypes.byref(c), FAKE, 8, FAKE, FAKE, FAKE, FAKE,
                         None)
    assert st == -4
    w = fake_weights(d=32)
    tok = T.Tokens(emb=FAKE, action_type=FAKE, time_bucket=FAKE, valid_len=FAKE, total=10, T=64,
                   d=32, dtype=T.I8, reserved=0)
    assert lib.tav2_encode(ctypes.byref(tok), FAKE, ctypes.byref(w), 0, FAKE, FAKE, 1 << 40,
                           None) == -4
    st = lib.tav2_select_encode(ctypes.byref(s), None, ctypes.byref(c), 8, ctypes.byref(w), 0,
                                FAKE, FAKE, FAKE, FAKE, 1 << 40, None)
    assert st == -4


def test_fused_search_workspace_does_not_scale_with_the_sequence():
    """Sequences of more than 4096 rows (bf16 and int8) keep their scores on chip:
    the workspace holds per candidate 1024 sampled 16-bit keys, a threshold, a
    count, a survivor list of 2 k + 1024 (rounded up to 64) 8-byte values and a
    queue slot; shorter ones, and float32, hold the score rows."""
    lib = T.load_library()
    c = fake_cands(total=10, max_count=10)

    def a256(x):
        return (x + 255) // 256 * 256

    for dt in (T.BF16, T.I8):
        for L in (16384, 32768):
            s = fake_seq(R=1, d=64, dtype=dt, max_len=L)
            want = (a256(10 * 1024 * 2) + a256(40) + a256(40) + a256(10 * 1536 * 8) + a256(80)
                    + a256(4))
            assert lib.tav2_nn_select_workspace(ctypes.byref(s), ctypes.byref(c), 256) == want
        s = fake_seq(R=1, d=64, dtype=dt, max_len=4096)
        assert lib.tav2_nn_select_workspace(ctypes.byref(s), ctypes.byref(c), 256) == 10 * 4096 * 4
    s = fake_seq(R=1, d=64, dtype=T.F32, max_len=16384)
    assert lib.tav2_nn_select_workspace(ctypes.byref(s), ctypes.byref(c), 256) == 10 * 16384 * 4


def test_eq2_struct_layout_and_argument_errors(tmp_path):
    src = tmp_path / "eq2.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "tav2.h"\n'
                   'int main(void){printf("%zu %zu %zu\\n", sizeof(tav2_eq2),'
                   'offsetof(tav2_eq2, imp), offsetof(tav2_eq2, k_imp));return 0;}\n')
    exe = tmp_path / "eq2"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o",
                    str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    assert got == [ctypes.sizeof(T.Eq2), T.Eq2.imp.offset, T.Eq2.k_imp.offset]

    lib = T.load_library()
    s, c = fake_seq(d=64), fake_cands()
    rt, imp = fake_seq(d=64, max_len=100), fake_seq(d=64, max_len=80)

    def call(eq2, k=64, w=None):
        w = w or fake_weights(max_pos=1024)
        return lib.tav2_select_encode_eq2(ctypes.byref(s), ctypes.byref(eq2) if eq2 else None,
                                          ctypes.byref(c), k, ctypes.byref(w), 0, FAKE, FAKE, None,
                                          FAKE, 1 << 40, None)

    P = ctypes.pointer
    assert call(None) == -1
    assert call(T.Eq2(rt=None, r=0, k_rt=8, imp=None, k_imp=0)) == -1      # k_rt without S_RT
    assert call(T.Eq2(rt=None, r=4, k_rt=0, imp=None, k_imp=0)) == -1      # r without S_RT
    assert call(T.Eq2(rt=P(rt), r=4, k_rt=0, imp=None, k_imp=8)) == -1     # k_imp without S_imp
    assert call(T.Eq2(rt=P(rt), r=-1, k_rt=0, imp=None, k_imp=0)) == -2
    assert call(T.Eq2(rt=P(rt), r=4, k_rt=2000, imp=None, k_imp=0)) == -2  # k_rt > K_MAX
    assert call(T.Eq2(rt=P(rt), r=100, k_rt=512, imp=P(imp), k_imp=512)) == -2   # T > 1024
    assert call(T.Eq2(rt=P(rt), r=8, k_rt=8, imp=P(imp), k_imp=8),
                w=fake_weights(max_pos=64 + 8 + 8 + 7)) == -2              # T > max_pos
    other = fake_seq(R=3, d=64, max_len=80)
    assert call(T.Eq2(rt=P(rt), r=8, k_rt=8, imp=P(other), k_imp=8)) == -2  # request count
    # valid: the error comes from the missing output
    assert call(T.Eq2(rt=P(rt), r=8, k_rt=8, imp=P(imp), k_imp=8)) == -1
    need = lib.tav2_select_encode_eq2_workspace(
        ctypes.byref(s), ctypes.byref(T.Eq2(rt=P(rt), r=8, k_rt=8, imp=P(imp), k_imp=8)),
        ctypes.byref(c), 64, ctypes.byref(fake_weights(max_pos=1024)))
    plain = lib.tav2_select_encode_workspace(ctypes.byref(s), None, ctypes.byref(c), 64,
                                             ctypes.byref(fake_weights(max_pos=1024)))
    assert need > plain > 0


@pytest.mark.parametrize("case,status", [("null_cfg", -1), ("dtype", -3), ("d", -2),
                                         ("requests", -2), ("cands", -2), ("time", -2)])
def test_batcher_config_errors(case, status):
    """A bad configuration is refused before anything is allocated."""
    lib = T.load_library()
    cfg = T.BatcherConfig(dtype=T.I8, d=32, has_time=1, max_requests=8, max_rows=1000,
                          max_rt_rows=0, max_cands=64)
    if case == "dtype":
        cfg.dtype = 7
    elif case == "d":
        cfg.d = 20
    elif case == "requests":
        cfg.max_requests = 0
    elif case == "cands":
        cfg.max_cands = 0
    elif case == "time":
        cfg.has_time = 2
    h = ctypes.c_void_p()
    st = lib.tav2_batcher_create(None if case == "null_cfg" else ctypes.byref(cfg), ctypes.byref(h))
    assert st == status and not h.value


def test_batcher_null_handles():
    lib = T.load_library()
    assert lib.tav2_batcher_reset(None) == -1
    assert lib.tav2_batcher_add(None, None) == -1
    assert lib.tav2_batcher_upload(None, None) == -1
    assert lib.tav2_batcher_views(None, None, None, None) == -1
    assert lib.tav2_batcher_arena_bytes(None) == 0
    lib.tav2_batcher_destroy(None)
