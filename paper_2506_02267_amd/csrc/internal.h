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
hipError_t launch_topk(const tav2_seq& seq, const tav2_cands& c, const float* scores, int64_t ld,
                       int k, int32_t* out_idx, float* out_score, int32_t* cand_req,
                       hipStream_t st);

// ---- select_fused.hip: NN search with the scores kept on chip (bf16 and int8
// sequences whose longest request exceeds FUSED_MIN_LEN rows)
constexpr int FUSED_MIN_LEN = 4096;
bool select_fused_applies(const tav2_seq& seq);
size_t select_fused_workspace(const tav2_cands& c, int k);
// cand_req (nullable): also receives each candidate's request index.
hipError_t launch_select_fused(const tav2_seq& seq, const tav2_cands& c, int k,
                               int32_t* out_idx, float* out_score, int32_t* cand_req, void* ws,
                               hipStream_t st);

// ---- gather.hip
// Where encoder tokens come from: either explicit token tensors, or the
// selection (idx) into the request sequence plus an optional real-time tail.
struct TokenSource {
  // explicit tokens [total, T, ...]
  const void* tok_emb;
  const uint8_t* tok_act;
  const uint8_t* tok_time;
  const int32_t* valid_len;
  // selection path
  const void* seq_emb;
  const uint8_t* seq_act;
  const uint8_t* seq_time;
  const int64_t* seq_off;
  const int32_t* seq_len;
  const void* rt_emb;
  const uint8_t* rt_act;
  const uint8_t* rt_time;
  const int64_t* rt_off;
  const int32_t* rt_len;
  const int32_t* idx;        // [total, k]
  const int32_t* cand_req;   // [total] request of each candidate
  int k;
  int T;
  int d;
  bool explicit_tokens;
};

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

// ---- encoder_f32.hip
constexpr int F32_MAX_T = 64;
constexpr int F32_MAX_DM = 128;
constexpr int F32_MAX_FFN = 512;
constexpr int F32_LDS_FLOATS = 36 * 1024;
bool encode_f32_fits(int T, const tav2_weights& w);
hipError_t launch_encode_f32(const TokenSource& src, const void* cand_emb, int64_t total,
                             const tav2_weights& w, float* out, bool unmasked, hipStream_t st);

}  // namespace tav2
