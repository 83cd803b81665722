// Device pieces shared by the NN-search kernels (select.hip, select_fused.hip):
// int8 code conversion, and selection over 48-bit (key, row) values.
#pragma once

#include "common.h"

namespace tav2 {

// The int8 sequence storage (codes q, Sec. 3.2.1) enters the products as bf16
// (exact: |q| <= 127); the lane also accumulates the squares of its 8 codes
// (exact in fp32: a row's sum of squares is an integer below 2^24).
__device__ __forceinline__ bf16x8 codes_to_bf16(uint2 raw, float& sq) {
  bf16x8 v;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t word = j < 4 ? raw.x : raw.y;
    const float x = float(int8_t((word >> (8 * (j & 3))) & 0xFF));
    sq = fmaf(x, x, sq);
    v[j] = static_cast<__bf16>(x);
  }
  return v;
}

// Normalised score of Sec. 3.4.2's fused dequantisation: <q, c> / |q| from the
// exact dot product and the exact sum of squares ss (0 for an all-zero row).  The
// division and the square root are rounded to nearest (the build keeps them
// correctly rounded).
__device__ __forceinline__ float i8_score(float dot, float ss) {
  return ss > 0.f ? dot / sqrtf(ss) : 0.f;
}

// 48-bit selection value of a row: its 32-bit score key above 0xFFFF - row, so
// that the larger value is the row earlier in the order (score desc, row asc).
// Rows are below 65536.
__device__ __forceinline__ uint64_t sel_value(uint32_t key, int row) {
  return (uint64_t(key) << 16) | uint64_t(0xFFFFu - uint32_t(row));
}
__device__ __forceinline__ int sel_row(uint64_t v) { return int(0xFFFFu - uint32_t(v & 0xFFFFu)); }
__device__ __forceinline__ uint32_t sel_key(uint64_t v) { return uint32_t(v >> 16); }

// Orders a wave's LDS writes before its later LDS reads of words other lanes
// wrote (no workgroup barrier: the data is the wave's own).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Wave-wide scans and reductions through DPP row shifts and row broadcasts
// (no LDS round trip): row_shr 1, 2, 4, 8 combine within rows of 16 lanes, then
// row_bcast 15 and 31 carry row totals upwards.  Lanes a shift leaves without a
// source take the identity (the `old` operand).
#define TAV2_DPP_STEPS(OP, ID)                                                          \
  v = v OP uint32_t(__builtin_amdgcn_update_dpp(ID, int(v), 0x111, 0xf, 0xf, false)); \
  v = v OP uint32_t(__builtin_amdgcn_update_dpp(ID, int(v), 0x112, 0xf, 0xf, false)); \
  v = v OP uint32_t(__builtin_amdgcn_update_dpp(ID, int(v), 0x114, 0xf, 0xf, false)); \
  v = v OP uint32_t(__builtin_amdgcn_update_dpp(ID, int(v), 0x118, 0xf, 0xf, false)); \
  v = v OP uint32_t(__builtin_amdgcn_update_dpp(ID, int(v), 0x142, 0xa, 0xf, false)); \
  v = v OP uint32_t(__builtin_amdgcn_update_dpp(ID, int(v), 0x143, 0xc, 0xf, false));
// Inclusive prefix sum over the lanes.
__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t v) {
  TAV2_DPP_STEPS(+, 0)
  return v;
}
// OR / AND over the lanes, returned to every lane (lane 63 holds the result).
__device__ __forceinline__ uint64_t wave_or64(uint64_t x) {
  uint32_t v = uint32_t(x);
  TAV2_DPP_STEPS(|, 0)
  const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(v), 63));
  v = uint32_t(x >> 32);
  TAV2_DPP_STEPS(|, 0)
  return (uint64_t(uint32_t(__builtin_amdgcn_readlane(int(v), 63))) << 32) | lo;
}
__device__ __forceinline__ uint64_t wave_and64(uint64_t x) {
  uint32_t v = uint32_t(x);
  TAV2_DPP_STEPS(&, -1)
  const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(v), 63));
  v = uint32_t(x >> 32);
  TAV2_DPP_STEPS(&, -1)
  return (uint64_t(uint32_t(__builtin_amdgcn_readlane(int(v), 63))) << 32) | lo;
}
#undef TAV2_DPP_STEPS

// One digit step of a descending radix select, done by a whole wave on a
// 256-bin histogram h in LDS: the digit whose bin holds the need-th largest
// value (1 <= need <= the histogram's total) and the rank of that value among
// the bin's values (rest).  Lane l takes bins 255 - 4l .. 252 - 4l; every lane
// returns the result.
__device__ __forceinline__ void radix_digit(const uint32_t* h, uint32_t need, uint32_t& digit,
                                            uint32_t& rest) {
  const int lane = threadIdx.x % WAVE;
  const uint4 q = *reinterpret_cast<const uint4*>(h + 252 - 4 * lane);
  const uint32_t hb[4] = {q.w, q.z, q.y, q.x};   // bins 255 - 4l - i
  const uint32_t sum = hb[0] + hb[1] + hb[2] + hb[3];
  const uint32_t incl = wave_incl_sum(sum);
  const uint32_t before = incl - sum;
  uint32_t dg = 0, rs = 0, cum = before;
  bool hit = false;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (!hit && cum + hb[i] >= need) {
      hit = true;
      dg = uint32_t(255 - 4 * lane - i);
      rs = need - cum;
    }
    cum += hb[i];
  }
  // exactly one lane holds the crossing
  const uint64_t who = __builtin_amdgcn_ballot_w64(before < need && need <= incl);
  const int src = int(__builtin_ctzll(who));
  digit = uint32_t(__builtin_amdgcn_readlane(int(dg), src));
  rest = uint32_t(__builtin_amdgcn_readlane(int(rs), src));
}

// The need-th largest (1-based) of the cnt distinct 48-bit values v[] in LDS,
// by an 8-bit radix select, most significant byte first, with NT threads.  The
// bytes above the highest bit in which the values differ are common to all of
// them and are skipped (their passes would put every value in one bin).  Every
// wave reads each histogram and finds the digit itself, and the histograms
// rotate over three buffers (a buffer is cleared in the pass after its own, two
// passes before its next use), so that a pass costs one barrier.  hist (3 x 256
// words, 16-byte aligned) and red (2 x NT / 64 values) are LDS scratch.  Starts
// and ends with a barrier; every thread returns the value.
template <int NT>
__device__ __forceinline__ uint64_t radix_select48(const uint64_t* v, int cnt, int need,
                                                   uint32_t* hist, uint64_t* red) {
  static_assert(NT >= 256, "one histogram bin per thread");
  constexpr int NW = NT / WAVE;
  const int tid = threadIdx.x, lane = tid % WAVE, wid = tid / WAVE;
  __syncthreads();   // v[] is complete
  uint64_t any = 0, all = ~uint64_t(0);
  for (int i = tid; i < cnt; i += NT) {
    any |= v[i];
    all &= v[i];
  }
  any = wave_or64(any);
  all = wave_and64(all);
  if (lane == 0) {
    red[wid] = any;
    red[NW + wid] = all;
  }
  if (tid < 256) hist[tid] = hist[256 + tid] = 0u;
  __syncthreads();
  any = 0;
  all = ~uint64_t(0);
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    any |= red[w];
    all &= red[NW + w];
  }
  const uint64_t diff = (any ^ all) & ((uint64_t(1) << 48) - 1);
  // first pass: the byte holding the highest differing bit (0 when cnt == 1)
  const int top = diff ? 63 - __builtin_clzll(diff) : 0;
  const int sh0 = top / 8 * 8;
  uint64_t pre = sh0 + 8 >= 48 ? 0 : all >> (sh0 + 8);
  uint32_t nd = uint32_t(need);
  int buf = 0;
  for (int sh = sh0; sh >= 0; sh -= 8) {
    uint32_t* h = hist + 256 * buf;
    for (int i = tid; i < cnt; i += NT) {
      const uint64_t x = v[i];
      if ((x >> (sh + 8)) == pre) atomicAdd(&h[(x >> sh) & 255u], 1u);
    }
    __syncthreads();
    const int clr = buf == 0 ? 2 : buf - 1;   // the previous pass's buffer: read by now
    if (tid < 256) hist[256 * clr + tid] = 0u;
    uint32_t digit, rest;
    radix_digit(h, nd, digit, rest);
    pre = (pre << 8) | uint64_t(digit);
    nd = rest;
    buf = buf == 2 ? 0 : buf + 1;
  }
  __syncthreads();
  return pre;
}

// The kk distinct selection values sel[] (LDS, any order, 16-byte aligned) to
// their ranks in the order: out_idx[rank] = row, out_score[rank] = score.  The
// rank of a value is the number of larger values (each thread reads the list
// two values per 16-byte LDS read, the same address across the wave: broadcasts).
template <int NT>
__device__ __forceinline__ void place_by_rank(const uint64_t* sel, int kk, int32_t* oi, float* os) {
  const uint4* s2 = reinterpret_cast<const uint4*>(sel);
  for (int s = threadIdx.x; s < kk; s += NT) {
    const uint64_t me = sel[s];
    int rank = 0;
    int t = 0;
    for (; t + 8 <= kk; t += 8) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint4 v = s2[t / 2 + u];
        rank += (uint64_t(v.y) << 32 | v.x) > me ? 1 : 0;
        rank += (uint64_t(v.w) << 32 | v.z) > me ? 1 : 0;
      }
    }
    for (; t < kk; ++t) rank += sel[t] > me ? 1 : 0;
    oi[rank] = sel_row(me);
    os[rank] = key_score(sel_key(me));
  }
}

}  // namespace tav2
