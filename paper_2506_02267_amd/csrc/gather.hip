// Token assembly (Eq. 2 restricted to NN(S_LL, c) followed by the kept
// most-recent real-time actions S_RT[:r]; Eq. 3's ascending argsort order).
//
// One workgroup per candidate copies whole rows in 16-byte pieces; the
// request's rows are read from its single stored copy.
#include "common.h"
#include "internal.h"
#include "token_source.h"

namespace tav2 {

__global__ __launch_bounds__(256) void gather_kernel(
    const uint8_t* __restrict__ seq_emb, const uint8_t* __restrict__ seq_act,
    const uint8_t* __restrict__ seq_time, const int64_t* __restrict__ seq_off,
    const int32_t* __restrict__ seq_len, const uint8_t* __restrict__ rt_emb,
    const uint8_t* __restrict__ rt_act, const uint8_t* __restrict__ rt_time,
    const int64_t* __restrict__ rt_off, const int32_t* __restrict__ rt_len,
    const int64_t* __restrict__ cand_off, const int32_t* __restrict__ idx, int k, int T,
    int row_bytes, uint8_t* __restrict__ tok_emb, uint8_t* __restrict__ tok_act,
    uint8_t* __restrict__ tok_time, int32_t* __restrict__ valid_len) {
  const int r = blockIdx.y;
  const int64_t n = cand_off[r] + blockIdx.x;
  if (n >= cand_off[r + 1]) return;
  const int L = seq_len[r];
  const int t_ll = k < L ? k : L;
  const int lrt = rt_len ? rt_len[r] : 0;
  const int64_t sb = seq_off[r];
  const int64_t rb = rt_len ? rt_off[r] : 0;
  const int32_t* idx_n = idx + n * k;
  const int chunks = row_bytes / 16;
  uint4* dst = reinterpret_cast<uint4*>(tok_emb + n * int64_t(T) * row_bytes);
  for (int e = threadIdx.x; e < T * chunks; e += 256) {
    const int p = e / chunks, c = e % chunks;
    const int64_t row = token_row(p, t_ll, lrt, idx_n, L, sb, rb);
    uint4 v = make_uint4(0, 0, 0, 0);
    if (row >= 0) v = reinterpret_cast<const uint4*>(seq_emb + row * row_bytes)[c];
    else if (row <= -2) v = reinterpret_cast<const uint4*>(rt_emb + (-2 - row) * row_bytes)[c];
    dst[int64_t(p) * chunks + c] = v;
  }
  for (int p = threadIdx.x; p < T; p += 256) {
    const int64_t row = token_row(p, t_ll, lrt, idx_n, L, sb, rb);
    uint8_t a = 0, t = 0;
    if (row >= 0) {
      a = seq_act[row];
      t = seq_time ? seq_time[row] : 0;
    } else if (row <= -2) {
      a = rt_act[-2 - row];
      t = rt_time ? rt_time[-2 - row] : 0;
    }
    tok_act[n * T + p] = a;
    if (tok_time) tok_time[n * T + p] = t;
  }
  if (threadIdx.x == 0) valid_len[n] = t_ll + lrt;
}

hipError_t launch_gather(const tav2_seq& seq, const tav2_seq* rt, const tav2_cands& c,
                         const int32_t* idx, int k, int T, void* tok_emb, uint8_t* tok_act,
                         uint8_t* tok_time, int32_t* valid_len, hipStream_t st) {
  if (seq.num_requests == 0 || c.total == 0) return hipSuccess;
  const int es = seq.dtype == TAV2_BF16 ? 2 : 4;
  dim3 grid(unsigned(c.max_count), unsigned(seq.num_requests));
  ProfScope prof("gather", st);
  gather_kernel<<<grid, 256, 0, st>>>(
      static_cast<const uint8_t*>(seq.emb), seq.action_type, seq.time_bucket, seq.offset, seq.len,
      rt ? static_cast<const uint8_t*>(rt->emb) : nullptr, rt ? rt->action_type : nullptr,
      rt ? rt->time_bucket : nullptr, rt ? rt->offset : nullptr, rt ? rt->len : nullptr,
      c.offset, idx, k, T, seq.d * es, static_cast<uint8_t*>(tok_emb), tok_act, tok_time,
      valid_len);
  return hipGetLastError();
}

}  // namespace tav2
