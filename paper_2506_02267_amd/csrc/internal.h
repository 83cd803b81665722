// Internal launch interface between the C ABI layer (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/tav2.h"

namespace tav2 {

constexpr int SEL_MAX_LEN = 32768;   // longest request sequence the NN search accepts

// Brackets one kernel launch with HIP events when profiling is enabled
// (tav2_profile_enable); a no-op otherwise.
class ProfScope {
 public:
  ProfScope(const char* name, hipStream_t st);
  ~ProfScope();
  ProfScope(const ProfScope&) = delete;
  ProfScope& operator=(const ProfScope&) = delete;

 private:
  const char* name_;
  hipStream_t st_;
  void* start_;
};

// ---- select.hip
int64_t score_ld(int32_t max_len);
hipError_t launch_scores(const tav2_seq& seq, const tav2_cands& c, float* scores, int64_t ld,
                         hipStream_t st);
// cand_req (nullable): also receives each candidate's request index.
// out_ld: row stride (elements) of out_idx and out_score (>= k).
hipError_t launch_topk(const tav2_seq& seq, const tav2_cands& c, const float* scores, int64_t ld,
                       int k, int32_t* out_idx, float* out_score, int out_ld, int32_t* cand_req,
                       hipStream_t st);

// ---- select_fused.hip: NN search with the scores kept on chip (bf16 and int8
// sequences whose longest request exceeds FUSED_MIN_LEN rows)
constexpr int FUSED_MIN_LEN = 4096;
bool select_fused_applies(const tav2_seq& seq);
size_t select_fused_workspace(const tav2_cands& c, int k);
// cand_req (nullable): also receives each candidate's request index; out_ld: row
// stride of the outputs.
hipError_t launch_select_fused(const tav2_seq& seq, const tav2_cands& c, int k,
                               int32_t* out_idx, float* out_score, int out_ld, int32_t* cand_req,
                               void* ws, hipStream_t st);

// ---- gather.hip
// Where encoder tokens come from: either explicit token tensors, or the
// selections into the request-level sources of Eq. 2: NN(S_LL, c), the kept
// real-time rows S_RT[:r], NN(S_RT[r:], c) and NN(S_imp, c).
struct TokenSource {
  // explicit tokens [total, T, ...]
  const void* tok_emb;
  const uint8_t* tok_act;
  const uint8_t* tok_time;
  const int32_t* valid_len;
  // selection path: the lifelong sequence and its top-k rows
  const void* seq_emb;
  const uint8_t* seq_act;
  const uint8_t* seq_time;
  const int64_t* seq_off;
  const int32_t* seq_len;
  const int32_t* idx;        // [total, idx_ld]: rank order, -1 padded
  int k;
  int idx_ld;
  // real-time sequence (rt_len == nullptr: none): rows [0, rt_keep) kept, and
  // the top-k_rt of the rest (idx_rt counts rows from rt_keep; k_rt = 0: none)
  const void* rt_emb;
  const uint8_t* rt_act;
  const uint8_t* rt_time;
  const int64_t* rt_off;
  const int32_t* rt_len;
  int rt_keep;
  const int32_t* idx_rt;     // [total, idx_ld]
  int k_rt;
  // impression sequence (imp_len == nullptr: none) and its top-k_imp rows
  const void* imp_emb;
  const uint8_t* imp_act;
  const uint8_t* imp_time;
  const int64_t* imp_off;
  const int32_t* imp_len;
  const int32_t* idx_imp;    // [total, idx_ld]
  int k_imp;
  const int32_t* cand_req;   // [total] request of each candidate
  int T;
  int d;
  bool explicit_tokens;
  bool codes;   // rows are int8 codes (d bytes each); the encoder dequantises them
};

// The view S_RT[r:] of a sequence batch: off_out[q] = off[q] + min(r, len[q]),
// len_out[q] = max(len[q] - r, 0) (device arrays of num_requests entries).
hipError_t launch_seq_view(const tav2_seq& s, int r, int64_t* off_out, int32_t* len_out,
                           hipStream_t st);

hipError_t launch_gather(const tav2_seq& seq, const tav2_seq* rt, const tav2_cands& c,
                         const int32_t* idx, int k, int T, void* tok_emb, uint8_t* tok_act,
                         uint8_t* tok_time, int32_t* valid_len, hipStream_t st);

// ---- encoder_fused.hip
bool encode_fused_supported(int d, const tav2_weights& w);
size_t encode_fused_workspace(int64_t total, int T, const tav2_weights& w);
size_t encode_fused_packed_bytes(const tav2_weights& w);
hipError_t launch_encode_fused_pack(const tav2_weights& w, void* dst, hipStream_t st);
hipError_t launch_encode_fused(const TokenSource& src, const void* cand_emb, int64_t total,
                               const tav2_weights& w, float* out, void* ws, bool unmasked,
                               hipStream_t st);

// ---- encoder_small.hip: bf16 encoder for d_model 64 (all layer weights in LDS)
constexpr int SMALL_UNMASKED_MAX_T = 64;   // the unmasked mode: one 64-position block
bool encode_small_supported(int d, const tav2_weights& w);
bool encode_small_aligned(const tav2_weights& w);   // matrices 16-byte, tables 8-byte aligned
size_t encode_small_packed_bytes(const tav2_weights& w);
hipError_t launch_encode_small_pack(const tav2_weights& w, void* packed, hipStream_t st);
size_t encode_small_workspace(int64_t total, int T, const tav2_weights& w);
hipError_t launch_encode_small(const TokenSource& src, const void* cand_emb, int64_t total,
                               const tav2_weights& w, float* out, void* ws, bool unmasked,
                               hipStream_t st);

// ---- encoder_f32.hip
constexpr int F32_MAX_T = 64;
constexpr int F32_MAX_DM = 128;
constexpr int F32_MAX_FFN = 512;
constexpr int F32_MAX_D = 256;
bool encode_f32_fits(int T, const tav2_weights& w);
hipError_t launch_encode_f32(const TokenSource& src, const void* cand_emb, int64_t total,
                             const tav2_weights& w, float* out, bool unmasked, hipStream_t st);

}  // namespace tav2
