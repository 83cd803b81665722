// Token assembly of Eq. 2 in encoder order (token_source.h): one workgroup per
// candidate copies whole rows in 16-byte pieces from the request's single stored
// copy of each source; positions past the valid tokens are zero.
#include "common.h"
#include "internal.h"
#include "token_source.h"

namespace tav2 {

__global__ __launch_bounds__(256) void gather_kernel(TokenSource s, const int64_t* __restrict__ cand_off,
                                                     int row_bytes, uint8_t* __restrict__ tok_emb,
                                                     uint8_t* __restrict__ tok_act,
                                                     uint8_t* __restrict__ tok_time,
                                                     int32_t* __restrict__ valid_len) {
  const int r = blockIdx.y;
  const int64_t n = cand_off[r] + blockIdx.x;
  if (n >= cand_off[r + 1]) return;
  const int T = s.T;
  const int chunks = row_bytes / 16;
  uint4* dst = reinterpret_cast<uint4*>(tok_emb + n * int64_t(T) * row_bytes);
  for (int e = threadIdx.x; e < T * chunks; e += 256) {
    const int p = e / chunks, c = e % chunks;
    const TokenRef t = selected_token(s, n, r, p, row_bytes);
    dst[int64_t(p) * chunks + c] = t.emb ? reinterpret_cast<const uint4*>(t.emb)[c]
                                         : make_uint4(0, 0, 0, 0);
  }
  for (int p = threadIdx.x; p < T; p += 256) {
    const TokenRef t = selected_token(s, n, r, p, row_bytes);
    tok_act[n * T + p] = uint8_t(t.emb ? t.act : 0);
    if (tok_time) tok_time[n * T + p] = uint8_t(t.emb ? t.time : 0);
  }
  if (threadIdx.x == 0) {
    const TokenParts q = token_parts(s, r);
    valid_len[n] = q.t_ll + q.keep + q.t_rt + q.t_imp;
  }
}

hipError_t launch_gather(const tav2_seq& seq, const tav2_seq* rt, const tav2_cands& c,
                         const int32_t* idx, int k, int T, void* tok_emb, uint8_t* tok_act,
                         uint8_t* tok_time, int32_t* valid_len, hipStream_t st) {
  if (seq.num_requests == 0 || c.total == 0) return hipSuccess;
  const int es = seq.dtype == TAV2_BF16 ? 2 : 4;
  TokenSource s{};
  s.seq_emb = seq.emb;
  s.seq_act = seq.action_type;
  s.seq_time = seq.time_bucket;
  s.seq_off = seq.offset;
  s.seq_len = seq.len;
  s.idx = idx;
  s.k = k;
  s.idx_ld = k;
  if (rt) {   // every real-time row kept
    s.rt_emb = rt->emb;
    s.rt_act = rt->action_type;
    s.rt_time = rt->time_bucket;
    s.rt_off = rt->offset;
    s.rt_len = rt->len;
    s.rt_keep = rt->max_len;
  }
  s.T = T;
  s.d = seq.d;
  dim3 grid(unsigned(c.max_count), unsigned(seq.num_requests));
  ProfScope prof("gather", st);
  gather_kernel<<<grid, 256, 0, st>>>(s, c.offset, seq.d * es, static_cast<uint8_t*>(tok_emb),
                                      tok_act, tok_time, valid_len);
  return hipGetLastError();
}

// The view S_RT[r:] of a batch: offsets and lengths of the rows from r on.
__global__ void seq_view_kernel(const int64_t* __restrict__ off, const int32_t* __restrict__ len,
                                int R, int r, int64_t* __restrict__ off_out,
                                int32_t* __restrict__ len_out) {
  const int q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= R) return;
  const int l = len[q];
  const int skip = r < l ? r : l;
  off_out[q] = off[q] + skip;
  len_out[q] = l - skip;
}

hipError_t launch_seq_view(const tav2_seq& s, int r, int64_t* off_out, int32_t* len_out,
                           hipStream_t st) {
  if (s.num_requests == 0) return hipSuccess;
  ProfScope prof("seq_view", st);
  seq_view_kernel<<<unsigned(cdiv(s.num_requests, 256)), 256, 0, st>>>(
      s.offset, s.len, s.num_requests, r, off_out, len_out);
  return hipGetLastError();
}

}  // namespace tav2
