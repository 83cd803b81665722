// Where encoder position p of candidate n reads its action row from (shared by
// the standalone gather and the encoder's fused gather).
#pragma once

#include "common.h"
#include "internal.h"

namespace tav2 {

// Selected rows in ascending score order (rank t_ll-1-p at position p), then the
// real-time tail oldest first.  Returns a sequence row (>= 0), a real-time row
// encoded as -2 - row, or -1 for padding.
__device__ __forceinline__ int64_t token_row(int p, int t_ll, int lrt, const int32_t* idx_n,
                                             int L, int64_t seq_base, int64_t rt_base) {
  if (p < t_ll) {
    const int i = idx_n[t_ll - 1 - p];
    return (i >= 0 && i < L) ? seq_base + i : -1;
  }
  if (p < t_ll + lrt) return -2 - (rt_base + (lrt - 1 - (p - t_ll)));
  return -1;
}

struct TokenRef {
  const uint8_t* emb;   // row start (bytes), nullptr for padding
  int act;              // clamped to [0, 8)
  int time;             // clamped to [0, 64)
};

__device__ __forceinline__ int clamp_act(int a) { return a < 8 ? a : 7; }
__device__ __forceinline__ int clamp_time(int t) { return t < 64 ? t : 63; }

// Resolve (candidate n, position p) for either source kind; `row_bytes` = d * sizeof(elem).
__device__ __forceinline__ TokenRef resolve_token(const TokenSource& s, int64_t n, int p,
                                                  int row_bytes) {
  TokenRef t{nullptr, 0, 0};
  if (s.explicit_tokens) {
    if (p < s.valid_len[n]) {
      const int64_t m = n * s.T + p;
      t.emb = static_cast<const uint8_t*>(s.tok_emb) + m * row_bytes;
      t.act = clamp_act(s.tok_act[m]);
      t.time = s.tok_time ? clamp_time(s.tok_time[m]) : 0;
    }
    return t;
  }
  const int r = s.cand_req[n];
  const int L = s.seq_len[r];
  const int t_ll = s.k < L ? s.k : L;
  const int lrt = s.rt_len ? s.rt_len[r] : 0;
  const int64_t row = token_row(p, t_ll, lrt, s.idx + n * s.k, L, s.seq_off[r],
                                s.rt_len ? s.rt_off[r] : 0);
  if (row >= 0) {
    t.emb = static_cast<const uint8_t*>(s.seq_emb) + row * row_bytes;
    t.act = clamp_act(s.seq_act[row]);
    t.time = s.seq_time ? clamp_time(s.seq_time[row]) : 0;
  } else if (row <= -2) {
    const int64_t rr = -2 - row;
    t.emb = static_cast<const uint8_t*>(s.rt_emb) + rr * row_bytes;
    t.act = clamp_act(s.rt_act[rr]);
    t.time = s.rt_time ? clamp_time(s.rt_time[rr]) : 0;
  }
  return t;
}

__device__ __forceinline__ int token_valid_len(const TokenSource& s, int64_t n) {
  int v;
  if (s.explicit_tokens) {
    v = s.valid_len[n];
  } else {
    const int r = s.cand_req[n];
    const int L = s.seq_len[r];
    v = (s.k < L ? s.k : L) + (s.rt_len ? s.rt_len[r] : 0);
  }
  return v < 0 ? 0 : (v > s.T ? s.T : v);
}

}  // namespace tav2
