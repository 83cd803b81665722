// C ABI of the NN-select + encode library: host-side argument validation,
// workspace carving and kernel launches.  No allocation, no synchronisation.
#include <algorithm>
#include <mutex>
#include <string.h>

#include "common.h"
#include "internal.h"

using namespace tav2;

namespace {

constexpr int32_t ABI_VERSION = 2;
constexpr size_t WS_ALIGN = 256;

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

tav2_status hip_status(hipError_t e) { return e == hipSuccess ? TAV2_OK : TAV2_ERR_HIP; }

size_t elem_size(int32_t dtype) { return dtype == TAV2_BF16 ? 2 : 4; }

tav2_status check_dtype(int32_t dt) {
  return (dt == TAV2_F32 || dt == TAV2_BF16) ? TAV2_OK : TAV2_ERR_DTYPE;
}

// A sequence batch.  `for_select` adds the limits of the NN search kernels.
tav2_status check_seq(const tav2_seq* s, bool for_select) {
  if (!s) return TAV2_ERR_NULL;
  tav2_status st = s->dtype == TAV2_I8 ? TAV2_OK : check_dtype(s->dtype);
  if (st) return st;
  if (s->num_requests < 0 || s->max_len < 0) return TAV2_ERR_SHAPE;
  if (s->d < 16 || s->d > 512 || s->d % 16) return TAV2_ERR_SHAPE;
  if (for_select && s->max_len > SEL_MAX_LEN) return TAV2_ERR_UNSUPPORTED;
  if (s->num_requests > 0) {
    if (!s->offset || !s->len || !s->action_type) return TAV2_ERR_NULL;
    if (s->max_len > 0 && !s->emb) return TAV2_ERR_NULL;
    if (s->emb && !aligned(s->emb, 16)) return TAV2_ERR_SHAPE;
  }
  return TAV2_OK;
}

tav2_status check_cands(const tav2_cands* c, const tav2_seq* s) {
  if (!c) return TAV2_ERR_NULL;
  if (c->total < 0 || c->max_count < 0 || c->max_count > c->total) return TAV2_ERR_SHAPE;
  if (c->total > 0 && c->max_count == 0) return TAV2_ERR_SHAPE;
  if (c->total > 0 && s->num_requests == 0) return TAV2_ERR_SHAPE;
  if (c->total > (int64_t(1) << 31) - 1 || c->max_count > 65535) return TAV2_ERR_UNSUPPORTED;
  if (s->num_requests > 65535) return TAV2_ERR_UNSUPPORTED;
  if (s->num_requests > 0 && !c->offset) return TAV2_ERR_NULL;
  if (c->total > 0) {
    if (!c->emb) return TAV2_ERR_NULL;
    if (!aligned(c->emb, 16)) return TAV2_ERR_SHAPE;
  }
  return TAV2_OK;
}

tav2_status check_k(int32_t k) { return (k >= 1 && k <= TAV2_K_MAX) ? TAV2_OK : TAV2_ERR_SHAPE; }

bool vec_ok(const float* p) { return p && aligned(p, 16); }

// Weights for an encoder over T positions of width-d tokens; has_time says
// whether the tokens carry a time bucket.
tav2_status check_weights(const tav2_weights* w, int d, int dtype, int T, bool has_time) {
  if (!w) return TAV2_ERR_NULL;
  if (w->dtype != dtype) return TAV2_ERR_DTYPE;
  if (w->d_in != d) return TAV2_ERR_SHAPE;
  if (w->d_model < 1 || w->n_heads < 1 || w->d_model % w->n_heads || w->d_ffn < 1 ||
      w->n_layers < 1)
    return TAV2_ERR_SHAPE;
  if (T < 1 || T > TAV2_T_MAX || w->max_pos < T) return TAV2_ERR_SHAPE;
  if (!w->W_in || !w->E_act || !w->E_pos || !w->W_pool || !w->layers) return TAV2_ERR_NULL;
  if (!vec_ok(w->b_in) || !vec_ok(w->b_pool)) return w->b_in && w->b_pool ? TAV2_ERR_SHAPE : TAV2_ERR_NULL;
  if ((w->E_time != nullptr) != has_time) return TAV2_ERR_SHAPE;
  for (int i = 0; i < w->n_layers; ++i) {
    const tav2_layer& L = w->layers[i];
    if (!L.W_qkv || !L.W_o || !L.W_1 || !L.W_2) return TAV2_ERR_NULL;
    const float* v[] = {L.b_qkv, L.b_o, L.ln1_g, L.ln1_b, L.b_1, L.b_2, L.ln2_g, L.ln2_b};
    for (const float* p : v) {
      if (!p) return TAV2_ERR_NULL;
      if (!aligned(p, 16)) return TAV2_ERR_SHAPE;
    }
  }
  if (dtype == TAV2_BF16) {
    const bool small = encode_small_supported(d, *w);   // d_model 64
    if (small && !encode_small_aligned(*w)) return TAV2_ERR_SHAPE;
    if (!small && (!encode_fused_supported(d, *w) || w->d_ffn > 4096)) return TAV2_ERR_UNSUPPORTED;
    if (w->packed) {   // packed by tav2_pack_weights
      const size_t need = small ? encode_small_packed_bytes(*w) : encode_fused_packed_bytes(*w);
      if (!aligned(w->packed, WS_ALIGN) || w->packed_bytes < need) return TAV2_ERR_WORKSPACE;
    }
  } else {
    if (!encode_f32_fits(T, *w) || d > 256) return TAV2_ERR_UNSUPPORTED;
  }
  return TAV2_OK;
}

// The encoder's mask flags: TAV2_MASK_CAUSAL, or TAV2_MASK_NONE (the bf16 encoder
// keeps positions in blocks of 128 that see only earlier blocks: unmasked, T must
// fit one block).
tav2_status check_flags(uint32_t flags, const tav2_weights* w, int T) {
  if (flags != TAV2_MASK_CAUSAL && flags != TAV2_MASK_NONE) return TAV2_ERR_SHAPE;
  if (flags == TAV2_MASK_NONE && w->dtype == TAV2_BF16 &&
      T > (encode_small_supported(w->d_in, *w) ? SMALL_UNMASKED_MAX_T : 128))
    return TAV2_ERR_UNSUPPORTED;
  return TAV2_OK;
}

tav2_status check_ws(const void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return TAV2_OK;
  if (!ws || ws_bytes < need) return TAV2_ERR_WORKSPACE;
  if (!aligned(ws, WS_ALIGN)) return TAV2_ERR_WORKSPACE;
  return TAV2_OK;
}

int rt_len_max(const tav2_seq* rt) { return rt ? rt->max_len : 0; }

tav2_status check_rt(const tav2_seq* rt, const tav2_seq* seq) {
  if (!rt) return TAV2_OK;
  tav2_status st = check_seq(rt, false);
  if (st) return st;
  if (rt->num_requests != seq->num_requests || rt->d != seq->d) return TAV2_ERR_SHAPE;
  if (rt->dtype != seq->dtype) return TAV2_ERR_DTYPE;
  if ((rt->time_bucket != nullptr) != (seq->time_bucket != nullptr)) return TAV2_ERR_SHAPE;
  return TAV2_OK;
}

// The NN search's workspace: survivor lists when the scores stay on chip, else
// the materialised score rows.
size_t select_ws_bytes(const tav2_seq* s, const tav2_cands* c, int k) {
  if (select_fused_applies(*s)) return align_up(select_fused_workspace(*c, k), WS_ALIGN);
  return align_up(size_t(c->total) * size_t(score_ld(s->max_len)) * 4, WS_ALIGN);
}

// NN search writing rows of out_ld elements (the k results first).
hipError_t run_select(const tav2_seq& s, const tav2_cands& c, int k, int32_t* out_idx,
                      float* out_score, int out_ld, int32_t* cand_req, void* ws, hipStream_t st) {
  if (select_fused_applies(s))
    return launch_select_fused(s, c, k, out_idx, out_score, out_ld, cand_req, ws, st);
  float* scores = static_cast<float*>(ws);
  const int64_t ld = score_ld(s.max_len);
  hipError_t e = launch_scores(s, c, scores, ld, st);
  if (e == hipSuccess)
    e = launch_topk(s, c, scores, ld, k, out_idx, out_score, out_ld, cand_req, st);
  return e;
}

size_t encode_ws_bytes(int64_t total, int T, const tav2_weights* w) {
  if (w->dtype == TAV2_F32) return 0;
  if (encode_small_supported(w->d_in, *w))
    return align_up(encode_small_workspace(total, T, *w), WS_ALIGN);
  return align_up(encode_fused_workspace(total, T, *w), WS_ALIGN);
}

tav2_status run_encode(const TokenSource& src, const void* cand_emb, int64_t total,
                       const tav2_weights* w, uint32_t flags, float* out, void* ws,
                       hipStream_t st) {
  const bool unmasked = flags == TAV2_MASK_NONE;
  if (w->dtype == TAV2_BF16 && encode_small_supported(w->d_in, *w))
    return hip_status(launch_encode_small(src, cand_emb, total, *w, out, ws, unmasked, st));
  if (w->dtype == TAV2_BF16)
    return hip_status(launch_encode_fused(src, cand_emb, total, *w, out, ws, unmasked, st));
  return hip_status(launch_encode_f32(src, cand_emb, total, *w, out, unmasked, st));
}

// Eq. 2's sources besides the lifelong sequence: the real-time rows kept
// (S_RT[:r]) and searched (NN(S_RT[r:], c), k_rt rows), the impressions
// searched (k_imp rows).
struct Sources {
  const tav2_seq* rt;
  int r, k_rt;
  const tav2_seq* imp;
  int k_imp;
};
Sources keep_all(const tav2_seq* rt) { return Sources{rt, rt ? rt->max_len : 0, 0, nullptr, 0}; }
Sources sources_of(const tav2_eq2& e) { return Sources{e.rt, e.r, e.k_rt, e.imp, e.k_imp}; }

// Encoder positions: the searched rows, the kept real-time rows (at most the
// longest real-time request) and the other searches' rows.
int positions(const Sources& src, int k) {
  const int keep = src.rt ? (src.r < src.rt->max_len ? src.r : src.rt->max_len) : 0;
  return k + keep + src.k_rt + src.k_imp;
}

// A sequence that must look like the lifelong one (requests, width, dtype, time
// feature); `search`: an NN search runs over it.
tav2_status check_source(const tav2_seq* x, const tav2_seq* seq, bool search) {
  tav2_status st;
  if ((st = check_rt(x, seq))) return st;
  if (search && x->max_len > SEL_MAX_LEN) return TAV2_ERR_UNSUPPORTED;
  return TAV2_OK;
}

tav2_status check_select_encode(const tav2_seq* seq, const Sources& src, const tav2_cands* cands,
                                int k, const tav2_weights* w, uint32_t flags, int* T_out) {
  tav2_status st;
  if ((st = check_seq(seq, true)) || (st = check_cands(cands, seq)) || (st = check_k(k))) return st;
  // int8 codes feed the d_model-64 encoder (bf16 weights) only
  const bool codes = seq->dtype == TAV2_I8;
  if (codes && (!w || w->dtype != TAV2_BF16)) return w ? TAV2_ERR_DTYPE : TAV2_ERR_NULL;
  if (codes && !encode_small_supported(seq->d, *w)) return TAV2_ERR_UNSUPPORTED;
  if (src.r < 0 || src.k_rt < 0 || src.k_imp < 0) return TAV2_ERR_SHAPE;
  if (src.k_rt > TAV2_K_MAX || src.k_imp > TAV2_K_MAX) return TAV2_ERR_SHAPE;
  if ((src.k_rt > 0 || src.r > 0) && !src.rt) return TAV2_ERR_NULL;
  if (src.k_imp > 0 && !src.imp) return TAV2_ERR_NULL;
  if (src.rt && (st = check_source(src.rt, seq, src.k_rt > 0))) return st;
  if (src.imp && (st = check_source(src.imp, seq, true))) return st;
  const int64_t T = int64_t(k) + (src.rt ? std::min(src.r, src.rt->max_len) : 0) + src.k_rt +
                    src.k_imp;
  if (T > TAV2_T_MAX) return TAV2_ERR_SHAPE;
  if ((st = check_weights(w, seq->d, codes ? TAV2_BF16 : seq->dtype, int(T),
                          seq->time_bucket != nullptr)))
    return st;
  if ((st = check_flags(flags, w, int(T)))) return st;
  *T_out = int(T);
  return TAV2_OK;
}

// The S_RT[r:] view of the real-time batch (offsets and lengths in the workspace).
tav2_seq rest_view(const tav2_seq& rt, int r, int64_t* off, int32_t* len) {
  tav2_seq v = rt;
  v.offset = off;
  v.len = len;
  v.max_len = rt.max_len > r ? rt.max_len - r : 0;
  return v;
}

// Workspace: one NN-search region reused by the searches in turn, the S_RT[r:]
// view, each candidate's request, the encoder's part.
struct SeLayout {
  size_t sel, view_off, view_len, req, enc, total;
};
SeLayout select_encode_layout(const tav2_seq* seq, const Sources& src, const tav2_cands* cands,
                              int k, const tav2_weights* w, int T) {
  size_t sel = select_ws_bytes(seq, cands, k);
  const size_t R = size_t(seq->num_requests);
  if (src.k_rt > 0) {
    const tav2_seq v = rest_view(*src.rt, src.r, nullptr, nullptr);
    sel = std::max(sel, select_ws_bytes(&v, cands, src.k_rt));
  }
  if (src.k_imp > 0) sel = std::max(sel, select_ws_bytes(src.imp, cands, src.k_imp));
  SeLayout l{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align_up(bytes, WS_ALIGN);
    return at;
  };
  l.sel = take(sel);
  l.view_off = take(src.k_rt > 0 ? R * 8 : 0);
  l.view_len = take(src.k_rt > 0 ? R * 4 : 0);
  l.req = take(size_t(cands->total) * 4);
  l.enc = take(encode_ws_bytes(cands->total, T, w));
  l.total = off;
  return l;
}

tav2_status select_encode(const tav2_seq* seq, const Sources& src, const tav2_cands* cands,
                          int32_t k, const tav2_weights* w, uint32_t flags, int32_t* out_idx,
                          float* out_score, float* out, void* ws, size_t ws_bytes,
                          hipStream_t s) {
  tav2_status st;
  int T = 0;
  if ((st = check_select_encode(seq, src, cands, k, w, flags, &T))) return st;
  if (cands->total == 0) return TAV2_OK;
  if (!out_idx || !out_score || !out) return TAV2_ERR_NULL;
  if (!aligned(out, 16)) return TAV2_ERR_SHAPE;
  const SeLayout lay = select_encode_layout(seq, src, cands, k, w, T);
  if ((st = check_ws(ws, ws_bytes, lay.total))) return st;
  uint8_t* base = static_cast<uint8_t*>(ws);
  int32_t* cand_req = reinterpret_cast<int32_t*>(base + lay.req);
  const int ld = k + src.k_rt + src.k_imp;   // the searches' results side by side
  // the searches, one after the other in the same workspace region
  if (run_select(*seq, *cands, k, out_idx, out_score, ld, cand_req, base + lay.sel, s))
    return TAV2_ERR_HIP;
  if (src.k_rt > 0) {
    int64_t* voff = reinterpret_cast<int64_t*>(base + lay.view_off);
    int32_t* vlen = reinterpret_cast<int32_t*>(base + lay.view_len);
    if (launch_seq_view(*src.rt, src.r, voff, vlen, s)) return TAV2_ERR_HIP;
    const tav2_seq v = rest_view(*src.rt, src.r, voff, vlen);
    if (run_select(v, *cands, src.k_rt, out_idx + k, out_score + k, ld, nullptr, base + lay.sel, s))
      return TAV2_ERR_HIP;
  }
  if (src.k_imp > 0 &&
      run_select(*src.imp, *cands, src.k_imp, out_idx + k + src.k_rt, out_score + k + src.k_rt,
                 ld, nullptr, base + lay.sel, s))
    return TAV2_ERR_HIP;
  TokenSource ts{};
  ts.explicit_tokens = false;
  ts.codes = seq->dtype == TAV2_I8;
  ts.seq_emb = seq->emb;
  ts.seq_act = seq->action_type;
  ts.seq_time = seq->time_bucket;
  ts.seq_off = seq->offset;
  ts.seq_len = seq->len;
  ts.idx = out_idx;
  ts.k = k;
  ts.idx_ld = ld;
  if (src.rt) {
    ts.rt_emb = src.rt->emb;
    ts.rt_act = src.rt->action_type;
    ts.rt_time = src.rt->time_bucket;
    ts.rt_off = src.rt->offset;
    ts.rt_len = src.rt->len;
    ts.rt_keep = src.r;
    ts.idx_rt = out_idx + k;
    ts.k_rt = src.k_rt;
  }
  if (src.k_imp > 0) {
    ts.imp_emb = src.imp->emb;
    ts.imp_act = src.imp->action_type;
    ts.imp_time = src.imp->time_bucket;
    ts.imp_off = src.imp->offset;
    ts.imp_len = src.imp->len;
    ts.idx_imp = out_idx + k + src.k_rt;
    ts.k_imp = src.k_imp;
  }
  ts.cand_req = cand_req;
  ts.T = T;
  ts.d = seq->d;
  return run_encode(ts, cands->emb, cands->total, w, flags, out, base + lay.enc, s);
}

}  // namespace

extern "C" {

const char* tav2_status_string(tav2_status s) {
  switch (s) {
    case TAV2_OK: return "ok";
    case TAV2_ERR_NULL: return "a required pointer is NULL";
    case TAV2_ERR_SHAPE: return "a size is out of range or inconsistent";
    case TAV2_ERR_DTYPE: return "unknown or mismatched dtype";
    case TAV2_ERR_UNSUPPORTED: return "valid request not implemented by this build";
    case TAV2_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case TAV2_ERR_HIP: return "HIP launch failed";
    case TAV2_ERR_TOO_LARGE: return "request needs more scratch than the library's static buffer holds";
    default: return "unknown status";
  }
}

int32_t tav2_abi_version(void) { return ABI_VERSION; }

size_t tav2_nn_select_workspace(const tav2_seq* seq, const tav2_cands* cands, int32_t k) {
  if (check_seq(seq, true) || check_cands(cands, seq) || check_k(k)) return 0;
  return select_ws_bytes(seq, cands, k);
}

tav2_status tav2_nn_select(const tav2_seq* seq, const tav2_cands* cands, int32_t k,
                           int32_t* out_idx, float* out_score, void* ws, size_t ws_bytes,
                           void* stream) {
  tav2_status st;
  if ((st = check_seq(seq, true)) || (st = check_cands(cands, seq)) || (st = check_k(k))) return st;
  if (seq->dtype != TAV2_F32 && seq->dtype != TAV2_BF16 && seq->dtype != TAV2_I8)
    return TAV2_ERR_DTYPE;
  if (cands->total == 0) return TAV2_OK;
  if (!out_idx || !out_score) return TAV2_ERR_NULL;
  if ((st = check_ws(ws, ws_bytes, select_ws_bytes(seq, cands, k)))) return st;
  return hip_status(run_select(*seq, *cands, k, out_idx, out_score, k, nullptr, ws,
                               static_cast<hipStream_t>(stream)));
}

tav2_status tav2_gather(const tav2_seq* seq, const tav2_seq* rt, const tav2_cands* cands,
                        const int32_t* idx, int32_t k, void* tok_emb, uint8_t* tok_act,
                        uint8_t* tok_time, int32_t* valid_len, void* stream) {
  tav2_status st;
  if ((st = check_seq(seq, false)) || (st = check_cands(cands, seq)) || (st = check_k(k))) return st;
  if (seq->dtype == TAV2_I8) return TAV2_ERR_UNSUPPORTED;
  if ((st = check_rt(rt, seq))) return st;
  if (cands->total == 0) return TAV2_OK;
  if (!idx || !tok_emb || !tok_act || !valid_len) return TAV2_ERR_NULL;
  if (!aligned(tok_emb, 16)) return TAV2_ERR_SHAPE;
  const int T = k + rt_len_max(rt);
  if (T > TAV2_T_MAX + TAV2_K_MAX) return TAV2_ERR_SHAPE;
  return hip_status(launch_gather(*seq, rt, *cands, idx, k, T, tok_emb, tok_act, tok_time,
                                  valid_len, static_cast<hipStream_t>(stream)));
}

size_t tav2_encode_workspace(const tav2_tokens* tok, const tav2_weights* w) {
  if (!tok || !w) return 0;
  const int dt = tok->dtype == TAV2_I8 ? TAV2_BF16 : tok->dtype;   // codes: bf16 weights
  if (check_weights(w, tok->d, dt, tok->T, tok->time_bucket != nullptr)) return 0;
  return encode_ws_bytes(tok->total, tok->T, w);
}

size_t tav2_pack_weights_bytes(const tav2_weights* w) {
  if (!w || w->dtype != TAV2_BF16) return 0;
  if (check_weights(w, w->d_in, TAV2_BF16, 1, w->E_time != nullptr)) return 0;
  if (encode_small_supported(w->d_in, *w))
    return align_up(encode_small_packed_bytes(*w), WS_ALIGN);
  return align_up(encode_fused_packed_bytes(*w), WS_ALIGN);
}

tav2_status tav2_pack_weights(const tav2_weights* w, void* packed, size_t bytes, void* stream) {
  if (!w) return TAV2_ERR_NULL;
  tav2_status st;
  if ((st = check_dtype(w->dtype))) return st;
  if (w->d_in < 16 || w->d_in > 512 || w->d_in % 16) return TAV2_ERR_SHAPE;
  if ((st = check_weights(w, w->d_in, w->dtype, 1, w->E_time != nullptr))) return st;
  if (w->dtype == TAV2_F32) return TAV2_OK;
  const bool small = encode_small_supported(w->d_in, *w);
  const size_t need = small ? encode_small_packed_bytes(*w) : encode_fused_packed_bytes(*w);
  if (!packed || !aligned(packed, WS_ALIGN) || bytes < need) return TAV2_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  return hip_status(small ? launch_encode_small_pack(*w, packed, hs)
                          : launch_encode_fused_pack(*w, packed, hs));
}

tav2_status tav2_encode(const tav2_tokens* tok, const void* cand_emb, const tav2_weights* w,
                        uint32_t flags, float* out, void* ws, size_t ws_bytes, void* stream) {
  if (!tok || !w) return TAV2_ERR_NULL;
  tav2_status st;
  // int8 codes feed the d_model-64 encoder (bf16 weights) only
  const bool codes = tok->dtype == TAV2_I8;
  if (codes && w->dtype != TAV2_BF16) return TAV2_ERR_DTYPE;
  if (!codes && (st = check_dtype(tok->dtype))) return st;
  if (tok->total < 0 || tok->d < 16 || tok->d > 512 || tok->d % 16) return TAV2_ERR_SHAPE;
  if (tok->total > (int64_t(1) << 31) - 1) return TAV2_ERR_UNSUPPORTED;
  if (codes && !encode_small_supported(tok->d, *w)) return TAV2_ERR_UNSUPPORTED;
  if ((st = check_weights(w, tok->d, codes ? TAV2_BF16 : tok->dtype, tok->T,
                          tok->time_bucket != nullptr)))
    return st;
  if ((st = check_flags(flags, w, tok->T))) return st;
  if (tok->total == 0) return TAV2_OK;
  if (!tok->emb || !tok->action_type || !tok->valid_len || !cand_emb || !out) return TAV2_ERR_NULL;
  if (!aligned(tok->emb, 16) || !aligned(cand_emb, 16) || !aligned(out, 16)) return TAV2_ERR_SHAPE;
  if ((st = check_ws(ws, ws_bytes, encode_ws_bytes(tok->total, tok->T, w)))) return st;
  TokenSource src{};
  src.explicit_tokens = true;
  src.codes = codes;
  src.tok_emb = tok->emb;
  src.tok_act = tok->action_type;
  src.tok_time = tok->time_bucket;
  src.valid_len = tok->valid_len;
  src.T = tok->T;
  src.d = tok->d;
  return run_encode(src, cand_emb, tok->total, w, flags, out, ws,
                    static_cast<hipStream_t>(stream));
}

size_t tav2_select_encode_workspace(const tav2_seq* seq, const tav2_seq* rt,
                                    const tav2_cands* cands, int32_t k, const tav2_weights* w) {
  const Sources src = keep_all(rt);
  int T = 0;
  if (check_select_encode(seq, src, cands, k, w, TAV2_MASK_CAUSAL, &T)) return 0;
  return select_encode_layout(seq, src, cands, k, w, T).total;
}

tav2_status tav2_select_encode(const tav2_seq* seq, const tav2_seq* rt, const tav2_cands* cands,
                               int32_t k, const tav2_weights* w, uint32_t flags,
                               int32_t* out_idx, float* out_score, float* out, void* ws,
                               size_t ws_bytes, void* stream) {
  return select_encode(seq, keep_all(rt), cands, k, w, flags, out_idx, out_score, out, ws,
                       ws_bytes, static_cast<hipStream_t>(stream));
}

size_t tav2_select_encode_eq2_workspace(const tav2_seq* seq, const tav2_eq2* eq2,
                                        const tav2_cands* cands, int32_t k,
                                        const tav2_weights* w) {
  if (!eq2) return 0;
  const Sources src = sources_of(*eq2);
  int T = 0;
  if (check_select_encode(seq, src, cands, k, w, TAV2_MASK_CAUSAL, &T)) return 0;
  return select_encode_layout(seq, src, cands, k, w, T).total;
}

tav2_status tav2_select_encode_eq2(const tav2_seq* seq, const tav2_eq2* eq2,
                                   const tav2_cands* cands, int32_t k, const tav2_weights* w,
                                   uint32_t flags, int32_t* out_idx, float* out_score, float* out,
                                   void* ws, size_t ws_bytes, void* stream) {
  if (!eq2) return TAV2_ERR_NULL;
  return select_encode(seq, sources_of(*eq2), cands, k, w, flags, out_idx, out_score, out, ws,
                       ws_bytes, static_cast<hipStream_t>(stream));
}

}  // extern "C"

// ---------------------------------------------------------------- no allocation
// The NN search for callers that cannot allocate: its workspace is a file-scope
// device array of TAV2_SCRATCH_BYTES (one per GPU, held until the process
// ends).  Host code never passes the array's name to a kernel: each device's
// address of it is looked up once (hipGetSymbolAddress, with that device
// current) and kept.
namespace {
__device__ __align__(256) uint8_t scratch[TAV2_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch[MAX_DEVICES] = {};

// This device's address of `scratch`, or nullptr with *err set.
void* device_scratch(hipError_t* err) {
  int dev = 0;
  *err = hipGetDevice(&dev);
  if (*err != hipSuccess) return nullptr;
  if (dev < 0 || dev >= MAX_DEVICES) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    *err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (*err != hipSuccess) return nullptr;
    g_scratch[dev] = p;
  }
  return g_scratch[dev];
}
}  // namespace

extern "C" {

size_t tav2_scratch_bytes(void) { return TAV2_SCRATCH_BYTES; }

tav2_status tav2_nn_select_noalloc(const tav2_seq* seq, const tav2_cands* cands, int32_t k,
                                   int32_t* out_idx, float* out_score, void* stream) {
  tav2_status st;
  if ((st = check_seq(seq, true)) || (st = check_cands(cands, seq)) || (st = check_k(k))) return st;
  if (cands->total == 0) return TAV2_OK;
  if (!out_idx || !out_score) return TAV2_ERR_NULL;
  if (select_ws_bytes(seq, cands, k) > TAV2_SCRATCH_BYTES) return TAV2_ERR_TOO_LARGE;
  hipError_t e = hipSuccess;
  void* ws = device_scratch(&e);
  if (!ws) return TAV2_ERR_HIP;
  return hip_status(run_select(*seq, *cands, k, out_idx, out_score, k, nullptr, ws,
                               static_cast<hipStream_t>(stream)));
}

}  // extern "C"
