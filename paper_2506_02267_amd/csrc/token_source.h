// Where encoder position p of candidate n reads its action row from (shared by
// the standalone gather and the encoders' fused gathers).
//
// The token set is Eq. 2's S_all = NN(S_LL, c) + S_RT[:r] + NN(S_RT[r:], c) +
// NN(S_imp, c): each NN part by ascending score (rank t - 1 - q at its q-th
// position, as Eq. 3's ascending argsort returns it, best match last), the kept
// real-time rows oldest first; the valid tokens of all parts are packed from
// position 0 and later positions are padding.
#pragma once

#include "common.h"
#include "internal.h"

namespace tav2 {

// Per-request and per-candidate metadata (lengths, offsets, request ids; written,
// if at all, by an earlier launch, never by the kernel reading it): read through
// the constant address space, so that a wave-uniform index gives a scalar load,
// whose wait does not also wait for the wave's vector memory loads in flight.
template <class T>
__device__ __forceinline__ T ld_meta(const T* p) {
  return *(const __attribute__((address_space(4))) T*)p;
}

struct TokenRef {
  const uint8_t* emb;   // row start (bytes), nullptr for padding
  int act;              // clamped to [0, 8)
  int time;             // clamped to [0, 64)
};

__device__ __forceinline__ int clamp_act(int a) { return a < 8 ? a : 7; }
__device__ __forceinline__ int clamp_time(int t) { return t < 64 ? t : 63; }

__device__ __forceinline__ TokenRef source_row(const void* emb, const uint8_t* act,
                                               const uint8_t* time, int64_t row, int row_bytes) {
  TokenRef t;
  t.emb = static_cast<const uint8_t*>(emb) + row * row_bytes;
  t.act = clamp_act(act[row]);
  t.time = time ? clamp_time(time[row]) : 0;
  return t;
}

// Valid tokens of each part for candidate n of request r.
struct TokenParts {
  int t_ll, keep, t_rt, t_imp;
};
__device__ __forceinline__ TokenParts token_parts(const TokenSource& s, int r) {
  TokenParts q{0, 0, 0, 0};
  const int L = ld_meta(s.seq_len + r);
  q.t_ll = s.k < L ? s.k : L;
  if (s.rt_len) {
    const int lrt = ld_meta(s.rt_len + r);
    q.keep = s.rt_keep < lrt ? s.rt_keep : lrt;
    const int rest = lrt - q.keep;
    q.t_rt = s.k_rt < rest ? s.k_rt : rest;
  }
  if (s.imp_len) {
    const int li = ld_meta(s.imp_len + r);
    q.t_imp = s.k_imp < li ? s.k_imp : li;
  }
  return q;
}

// Position p of candidate n of request r, selection path.
__device__ __forceinline__ TokenRef selected_token(const TokenSource& s, int64_t n, int r, int p,
                                                   int row_bytes) {
  TokenRef t{nullptr, 0, 0};
  const TokenParts q = token_parts(s, r);
  if (p < q.t_ll) {
    const int i = s.idx[n * s.idx_ld + q.t_ll - 1 - p];
    if (i >= 0 && i < ld_meta(s.seq_len + r))
      t = source_row(s.seq_emb, s.seq_act, s.seq_time, ld_meta(s.seq_off + r) + i, row_bytes);
    return t;
  }
  p -= q.t_ll;
  if (p < q.keep)
    return source_row(s.rt_emb, s.rt_act, s.rt_time, ld_meta(s.rt_off + r) + (q.keep - 1 - p),
                      row_bytes);
  p -= q.keep;
  if (p < q.t_rt) {
    const int i = s.idx_rt[n * s.idx_ld + q.t_rt - 1 - p];
    if (i >= 0 && q.keep + i < ld_meta(s.rt_len + r))
      t = source_row(s.rt_emb, s.rt_act, s.rt_time, ld_meta(s.rt_off + r) + q.keep + i, row_bytes);
    return t;
  }
  p -= q.t_rt;
  if (p < q.t_imp) {
    const int i = s.idx_imp[n * s.idx_ld + q.t_imp - 1 - p];
    if (i >= 0 && i < ld_meta(s.imp_len + r))
      t = source_row(s.imp_emb, s.imp_act, s.imp_time, ld_meta(s.imp_off + r) + i, row_bytes);
  }
  return t;
}

// Resolve (candidate n, position p) for either source kind; `row_bytes` = d * sizeof(elem).
__device__ __forceinline__ TokenRef resolve_token(const TokenSource& s, int64_t n, int p,
                                                  int row_bytes) {
  if (!s.explicit_tokens) return selected_token(s, n, ld_meta(s.cand_req + n), p, row_bytes);
  TokenRef t{nullptr, 0, 0};
  if (p < ld_meta(s.valid_len + n)) {
    const int64_t m = n * s.T + p;
    t.emb = static_cast<const uint8_t*>(s.tok_emb) + m * row_bytes;
    t.act = clamp_act(s.tok_act[m]);
    t.time = s.tok_time ? clamp_time(s.tok_time[m]) : 0;
  }
  return t;
}

__device__ __forceinline__ int token_valid_len(const TokenSource& s, int64_t n) {
  int v;
  if (s.explicit_tokens) {
    v = ld_meta(s.valid_len + n);
  } else {
    const TokenParts q = token_parts(s, ld_meta(s.cand_req + n));
    v = q.t_ll + q.keep + q.t_rt + q.t_imp;
  }
  return v < 0 ? 0 : (v > s.T ? s.T : v);
}

}  // namespace tav2
