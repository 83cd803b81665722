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

// The need-th largest (1-based) of the cnt distinct 48-bit values v[] in LDS,
// by an 8-bit radix select, most significant byte first, with NT threads.  The
// bytes above the highest bit in which the values differ are common to all of
// them and are skipped (their passes would put every value in one bin).  hist
// (256 words), misc (2 words) and common (2 words) are LDS scratch.  Ends with
// a barrier; every thread returns the value.
template <int NT>
__device__ __forceinline__ uint64_t radix_select48(const uint64_t* v, int cnt, int need,
                                                   uint32_t* hist, int* misc,
                                                   unsigned long long* common) {
  static_assert(NT >= 256, "one histogram bin per thread");
  const int tid = threadIdx.x, lane = tid % WAVE, wid = tid / WAVE;
  uint64_t any = 0, all = ~uint64_t(0);
  for (int i = tid; i < cnt; i += NT) {
    any |= v[i];
    all &= v[i];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    any |= __shfl_xor(any, o, WAVE);
    all &= __shfl_xor(all, o, WAVE);
  }
  if (tid == 0) {
    common[0] = 0ull;
    common[1] = ~0ull;
  }
  __syncthreads();
  if (lane == 0) {
    atomicOr(&common[0], (unsigned long long)any);
    atomicAnd(&common[1], (unsigned long long)all);
  }
  __syncthreads();
  const uint64_t diff = (uint64_t(common[0]) ^ uint64_t(common[1])) & ((uint64_t(1) << 48) - 1);
  // first pass: the byte holding the highest differing bit (0 when cnt == 1)
  const int top = diff ? 63 - __builtin_clzll(diff) : 0;
  const int sh0 = top / 8 * 8;
  uint64_t pre = sh0 + 8 >= 48 ? 0 : uint64_t(common[1]) >> (sh0 + 8);
  for (int sh = sh0; sh >= 0; sh -= 8) {
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    for (int i = tid; i < cnt; i += NT) {
      const uint64_t x = v[i];
      if ((x >> (sh + 8)) == pre) atomicAdd(&hist[(x >> sh) & 255u], 1u);
    }
    __syncthreads();
    if (wid == 0) {   // bins in descending order: lane l holds bins 255 - 4l - q
      uint32_t h[4], sum = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        h[q] = hist[255 - 4 * lane - q];
        sum += h[q];
      }
      uint32_t incl = sum;
#pragma unroll
      for (int o = 1; o < WAVE; o <<= 1) {
        const uint32_t t = __shfl_up(incl, o, WAVE);
        if (lane >= o) incl += t;
      }
      const uint32_t before = incl - sum;
      if (before < uint32_t(need) && uint32_t(need) <= incl) {
        uint32_t cum = before;
        int digit = 0, rest = 0;
        bool hit = false;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (!hit && cum + h[q] >= uint32_t(need)) {
            hit = true;
            digit = 255 - 4 * lane - q;
            rest = need - int(cum);
          }
          cum += h[q];
        }
        misc[0] = digit;
        misc[1] = rest;
      }
    }
    __syncthreads();
    pre = (pre << 8) | uint64_t(misc[0]);
    need = misc[1];
    __syncthreads();   // misc and hist are rewritten by the next pass
  }
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
