// NN search of Eq. 3 (Sec. 3.2.2): candidate x action dot-product scores over the
// de-duplicated request-level sequence, then the per-candidate top-k under the
// total order (score desc, row asc).
//
// Scores: bf16 operands on the 32x32x16 MFMA with fp32 accumulation (float32
// inputs use fp32 FMA; int8 sequence codes are dequantised and L2-normalised in
// the score kernel).  Each request's rows are read by every candidate tile of
// that request straight from the one stored copy (no per-candidate broadcast).
//
// Top-k, one workgroup per candidate, scores as order-preserving 32-bit keys.
// Rows of up to 4096 keys: the row is held in registers, the k-th largest key
// found by a 32-step bitwise search (each step one block-wide count), every key
// above it kept plus the lowest-indexed rows equal to it (an ordered compaction
// by block-wide prefix sum).  Longer rows are streamed once against a threshold
// taken from a sample, the keys above it compacted into LDS and the k-th largest
// found there by a radix select (an exact streaming search when the sample
// gives no usable threshold).  Either way the k survivors are placed by counting,
// for each, how many survivors precede it in the total order.
#include <atomic>

#include "common.h"
#include "internal.h"
#include "select_common.h"

namespace tav2 {

// ---------------------------------------------------------------- scores, bf16
// Block: 4 waves, 128 candidates x 256 rows; wave w covers rows [64w, 64w + 64)
// of all 128 candidates.  Candidates are the MFMA rows (A) and come from LDS (the
// block's 128 x d tile, loaded once), sequence rows the MFMA columns (B) and come
// straight from global memory (each wave its own rows), so each D register holds
// one candidate and 32 consecutive lanes 32 consecutive rows.  The tile sizes keep
// the re-reads of both operands small next to the score rows written.
constexpr int SC_CANDS = 128;
constexpr int SC_ROWS = 256;
constexpr int SC_PAD = 8;   // LDS row padding (bf16) of the candidate tile

__global__ __launch_bounds__(256) void score_bf16_kernel(
    const bf16_t* __restrict__ emb, const int64_t* __restrict__ seq_off,
    const int32_t* __restrict__ seq_len, const bf16_t* __restrict__ cand,
    const int64_t* __restrict__ cand_off, int d, int max_len, float* __restrict__ scores,
    int64_t ld) {
  extern __shared__ __attribute__((aligned(16))) bf16_t ctile[];   // [SC_CANDS][d + SC_PAD]
  const int r = blockIdx.z;
  const int64_t c_begin = cand_off[r], c_end = cand_off[r + 1];
  const int64_t n0 = c_begin + int64_t(blockIdx.y) * SC_CANDS;
  if (n0 >= c_end) return;
  const int L = min(seq_len[r], max_len);
  if (int(blockIdx.x) * SC_ROWS >= L) return;
  const int cld = d + SC_PAD;
  // candidate tile into LDS (rows past the request's candidates: its last one)
  for (int e = threadIdx.x; e < SC_CANDS * (d / 8); e += 256) {
    const int row = e / (d / 8), c = e % (d / 8);
    int64_t n = n0 + row;
    n = n < c_end ? n : c_end - 1;
    *reinterpret_cast<uint4*>(ctile + row * cld + c * 8) =
        *reinterpret_cast<const uint4*>(cand + n * d + c * 8);
  }
  __syncthreads();
  const int row0 = blockIdx.x * SC_ROWS + (threadIdx.x / WAVE) * 64;
  if (row0 >= L) return;
  const int lane = threadIdx.x % WAVE;
  const int h = lane / 32, l32 = lane % 32;
  const bf16_t* seq = emb + seq_off[r] * int64_t(d);
  const bf16_t* brow[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    int i = row0 + t * 32 + l32;
    i = i < L ? i : L - 1;   // clamped; not stored
    brow[t] = seq + int64_t(i) * d + 8 * h;
  }
  const bf16_t* arow = ctile + l32 * cld + 8 * h;
  f32x16 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};
  bf16x8 bv[2], bn[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) bv[t] = as_bf16x8(*reinterpret_cast<const uint4*>(brow[t]));
  for (int k0 = 0; k0 < d; k0 += 16) {
    const int kn = k0 + 16 < d ? k0 + 16 : k0;   // next k-block (the last one reloads itself)
#pragma unroll
    for (int t = 0; t < 2; ++t) bn[t] = as_bf16x8(*reinterpret_cast<const uint4*>(brow[t] + kn));
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const bf16x8 av = as_bf16x8(*reinterpret_cast<const uint4*>(arow + a * 32 * cld + k0));
#pragma unroll
      for (int b = 0; b < 2; ++b) acc[a][b] = mfma32(av, bv[b], acc[a][b]);
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) bv[t] = bn[t];
  }

#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int i = row0 + b * 32 + l32;
    if (i >= L) continue;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
#pragma unroll
      for (int reg = 0; reg < 16; ++reg) {
        const int64_t n = n0 + a * 32 + 8 * (reg / 4) + 4 * h + (reg % 4);
        if (n < c_end) scores[n * ld + i] = acc[a][b][reg];
      }
    }
  }
}

// ---------------------------------------------------------------- scores, int8
// The int8 sequence storage (codes q, Sec. 3.2.1) with dequantisation and L2
// normalisation fused into the score kernel (Sec. 3.4.2): s = <q_i, c> / |q_i|
// (the dequantisation scale cancels in the normalisation); codes_to_bf16 and
// i8_score (select_common.h) give the products' operands and the epilogue.
// Block: 4 waves, 32 candidates x 256 rows (a narrow candidate tile: the codes are
// short, so the block count, not operand reuse, sets the speed).  The normalised
// scores are staged in LDS and leave as one 1 KB non-temporal store per candidate
// row.
constexpr int SI_CANDS = 32;
constexpr int SI_ROWS = 256;
constexpr int SI_SLD = SI_ROWS + 8;   // staged score row stride (floats)

__global__ __launch_bounds__(256) void score_i8_kernel(
    const int8_t* __restrict__ emb, const int64_t* __restrict__ seq_off,
    const int32_t* __restrict__ seq_len, const bf16_t* __restrict__ cand,
    const int64_t* __restrict__ cand_off, int d, int max_len, float* __restrict__ scores,
    int64_t ld) {
  extern __shared__ __attribute__((aligned(16))) uint8_t si_smem[];
  float* stile = reinterpret_cast<float*>(si_smem);                           // [32][SI_SLD]
  bf16_t* ctile = reinterpret_cast<bf16_t*>(si_smem + SI_CANDS * SI_SLD * 4);  // [32][d + pad]
  const int r = blockIdx.z;
  const int64_t c_begin = cand_off[r], c_end = cand_off[r + 1];
  const int64_t n0 = c_begin + int64_t(blockIdx.y) * SI_CANDS;
  if (n0 >= c_end) return;
  const int L = min(seq_len[r], max_len);
  const int ib = blockIdx.x * SI_ROWS;
  if (ib >= L) return;
  const int cld = d + SC_PAD;
  for (int e = threadIdx.x; e < SI_CANDS * (d / 8); e += 256) {
    const int row = e / (d / 8), c = e % (d / 8);
    int64_t n = n0 + row;
    n = n < c_end ? n : c_end - 1;
    *reinterpret_cast<uint4*>(ctile + row * cld + c * 8) =
        *reinterpret_cast<const uint4*>(cand + n * d + c * 8);
  }
  __syncthreads();
  const int w = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  const int h = lane / 32, l32 = lane % 32;
  const int8_t* seq = emb + seq_off[r] * int64_t(d);
  const int8_t* brow[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    int i = ib + 64 * w + t * 32 + l32;
    i = i < L ? i : L - 1;   // clamped; never stored
    brow[t] = seq + int64_t(i) * d + 8 * h;
  }
  const bf16_t* arow = ctile + l32 * cld + 8 * h;
  f32x16 acc[2] = {f32x16{}, f32x16{}};
  float sq[2] = {0.f, 0.f};
  uint2 raw[2], nxt[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) raw[t] = *reinterpret_cast<const uint2*>(brow[t]);
  for (int k0 = 0; k0 < d; k0 += 16) {
    const int kn = k0 + 16 < d ? k0 + 16 : k0;   // next k-block (the last one reloads itself)
#pragma unroll
    for (int t = 0; t < 2; ++t) nxt[t] = *reinterpret_cast<const uint2*>(brow[t] + kn);
    const bf16x8 av = as_bf16x8(*reinterpret_cast<const uint4*>(arow + k0));
#pragma unroll
    for (int t = 0; t < 2; ++t) acc[t] = mfma32(av, codes_to_bf16(raw[t], sq[t]), acc[t]);
#pragma unroll
    for (int t = 0; t < 2; ++t) raw[t] = nxt[t];
  }
  // D register 4j + i of tile t: candidate 8j + 4h + i, row 64w + 32t + l32
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const float ss = sq[t] + __shfl_xor(sq[t], 32, WAVE);   // the row's other half
#pragma unroll
    for (int reg = 0; reg < 16; ++reg)
      stile[(8 * (reg / 4) + 4 * h + (reg % 4)) * SI_SLD + 64 * w + 32 * t + l32] =
          i8_score(acc[t][reg], ss);
  }
  __syncthreads();
  const int nv = min(SI_ROWS, L - ib);   // valid rows of this block
  const int ii = 4 * lane;
#pragma unroll
  for (int q = 0; q < SI_CANDS / 4; ++q) {
    const int c = (SI_CANDS / 4) * w + q;
    const int64_t n = n0 + c;
    if (n >= c_end || ii >= nv) continue;
    const float4 v = *reinterpret_cast<const float4*>(stile + c * SI_SLD + ii);
    float* dst = scores + n * ld + ib + ii;
    if (ii + 4 <= nv) {
      // streaming store: the scores are read once, by the top-k
      __builtin_nontemporal_store(f32x4{v.x, v.y, v.z, v.w}, reinterpret_cast<f32x4*>(dst));
    } else {
      dst[0] = v.x;
      if (ii + 1 < nv) dst[1] = v.y;
      if (ii + 2 < nv) dst[2] = v.z;
    }
  }
}

// ---------------------------------------------------------------- scores, fp32
__global__ __launch_bounds__(256) void score_f32_kernel(
    const float* __restrict__ emb, const int64_t* __restrict__ seq_off,
    const int32_t* __restrict__ seq_len, const float* __restrict__ cand,
    const int64_t* __restrict__ cand_off, int d, int max_len, float* __restrict__ scores,
    int64_t ld) {
  __shared__ float cv[512];
  const int r = blockIdx.z;
  const int64_t n = cand_off[r] + blockIdx.y;
  if (n >= cand_off[r + 1]) return;
  const int L = min(seq_len[r], max_len);
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (blockIdx.x * 256 >= L) return;
  for (int j = threadIdx.x; j < d; j += 256) cv[j] = cand[n * d + j];
  __syncthreads();
  if (i >= L) return;
  const float4* row = reinterpret_cast<const float4*>(emb + (seq_off[r] + i) * int64_t(d));
  float s = 0.f;
  for (int j = 0; j < d / 4; ++j) {
    float4 v = row[j];
    s = fmaf(v.x, cv[4 * j], s);
    s = fmaf(v.y, cv[4 * j + 1], s);
    s = fmaf(v.z, cv[4 * j + 2], s);
    s = fmaf(v.w, cv[4 * j + 3], s);
  }
  scores[n * ld + i] = s;
}

// ---------------------------------------------------------------- top-k
constexpr int TK_THREADS = 512;

// Exclusive prefix (in thread order) and block total of NV 64-bit values per
// thread; sw holds NV per wave.  sw is read after the one barrier inside: the
// caller synchronizes again before sw is written by a later scan.
template <int NV>
__device__ __forceinline__ void block_excl_scan(const uint64_t (&v)[NV], uint64_t (&excl)[NV],
                                                uint64_t (&total)[NV], uint64_t* sw, int lane,
                                                int wid) {
  uint64_t incl[NV];
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    uint64_t x = v[q];
#pragma unroll
    for (int o = 1; o < WAVE; o <<= 1) {
      const uint64_t t = __shfl_up(x, o, WAVE);
      if (lane >= o) x += t;
    }
    incl[q] = x;
    if (lane == WAVE - 1) sw[wid * NV + q] = x;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    uint64_t pre = 0, all = 0;
#pragma unroll
    for (int w = 0; w < TK_THREADS / WAVE; ++w) {
      const uint64_t t = sw[w * NV + q];
      pre += w < wid ? t : 0;
      all += t;
    }
    excl[q] = pre + incl[q] - v[q];
    total[q] = all;
  }
}

template <int PT>
__global__ __launch_bounds__(TK_THREADS) void topk_kernel(
    const float* __restrict__ scores, int64_t ld, const int64_t* __restrict__ cand_off,
    const int32_t* __restrict__ seq_len, int max_len, int k, int32_t* __restrict__ out_idx,
    float* __restrict__ out_score, int out_ld, int32_t* __restrict__ cand_req) {
  __shared__ int red[2][TK_THREADS / WAVE];
  __shared__ uint64_t scan_w[(TK_THREADS / WAVE) * 5];
  __shared__ __attribute__((aligned(16))) uint64_t sel[TAV2_K_MAX];

  const int r = blockIdx.y;
  const int64_t n = cand_off[r] + blockIdx.x;
  if (n >= cand_off[r + 1]) return;
  if (cand_req && threadIdx.x == 0) cand_req[n] = r;   // the candidate's request, for the encoder
  const int L = min(seq_len[r], max_len);
  const int tid = threadIdx.x, lane = tid % WAVE, wid = tid / WAVE;
  const int kk = k < L ? k : L;
  int32_t* oi = out_idx + n * out_ld;
  float* os = out_score + n * out_ld;
  for (int p = kk + tid; p < k; p += TK_THREADS) {
    oi[p] = -1;
    os[p] = -__builtin_inff();
  }
  if (kk == 0) return;

  // this thread's rows: chunk c (0 .. PT / 4 - 1) holds rows CH c + 4 tid + u, so
  // that every load instruction reads 1 KB of consecutive scores per wave; rows
  // past L get key 0 (below every score)
  constexpr int NC = PT / 4;
  constexpr int CH = TK_THREADS * 4;
  const float* srow = scores + n * ld;
  uint32_t key[PT];   // key[4 c + u]: row CH c + 4 tid + u
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int r0 = c * CH + tid * 4;
    if (r0 + 4 <= L) {
      const float4 v = *reinterpret_cast<const float4*>(srow + r0);
      key[4 * c] = score_key(v.x);
      key[4 * c + 1] = score_key(v.y);
      key[4 * c + 2] = score_key(v.z);
      key[4 * c + 3] = score_key(v.w);
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u) key[4 * c + u] = (r0 + u < L) ? score_key(srow[r0 + u]) : 0u;
    }
  }

  {
  // exhaustive: largest threshold t with count(key >= t) >= kk, one bit at a time
  uint32_t thr = 0;
  for (int b = 31; b >= 0; --b) {
    const uint32_t probe = thr | (1u << b);
    // wave-level count: one compare per key, the lane mask counted on the scalar unit
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < PT; ++j) cnt += __popcll(__builtin_amdgcn_ballot_w64(key[j] >= probe));
    if (lane == 0) red[b & 1][wid] = cnt;
    __syncthreads();
    int tot = 0;
#pragma unroll
    for (int w = 0; w < TK_THREADS / WAVE; ++w) tot += red[b & 1][w];
    if (tot >= kk) thr = probe;
  }

  // compaction: keys above thr anywhere in sel[0, count_gt) (the rank sort orders
  // them), then the need_eq lowest rows whose key equals thr.  Rows are ordered by
  // (chunk, thread, u), so the equal keys are counted per chunk: 16-bit fields,
  // four chunks per 64-bit word, summed in one block scan with the above count.
  constexpr int NW = (NC + 3) / 4;
  uint64_t word[NW + 1];   // word[0]: keys above thr; word[1 + c / 4]: equal keys of chunk c
#pragma unroll
  for (int q = 0; q <= NW; ++q) word[q] = 0;
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      word[0] += key[4 * c + u] > thr ? 1u : 0u;
      word[1 + c / 4] += key[4 * c + u] == thr ? (uint64_t(1) << (16 * (c % 4))) : 0u;
    }
  uint64_t excl[NW + 1], total[NW + 1];
  block_excl_scan<NW + 1>(word, excl, total, scan_w, lane, wid);
  const int count_gt = int(total[0]);
  const int need_eq = kk - count_gt;
  int gpos = int(excl[0]);
  int eq_before = 0;   // equal keys in chunks before c, over all threads
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int sh = 16 * (c % 4);
    int e = eq_before + int((excl[1 + c / 4] >> sh) & 0xFFFFu);
    eq_before += int((total[1 + c / 4] >> sh) & 0xFFFFu);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t kv = key[4 * c + u];
      const uint32_t row = uint32_t(c * CH + tid * 4 + u);
      const uint64_t packed = (uint64_t(kv) << 32) | uint64_t(0xFFFFFFFFu - row);
      if (kv > thr) {
        sel[gpos++] = packed;
      } else if (kv == thr) {
        if (e < need_eq) sel[count_gt + e] = packed;
        ++e;
      }
    }
  }
  __syncthreads();
  }

  // survivors are distinct under (key, -row): rank = number of survivors before it
  for (int s = tid; s < kk; s += TK_THREADS) {
    const uint64_t me = sel[s];
    int rank = 0;
    // 8 independent LDS reads per iteration (the survivor count is not a
    // multiple of 8 in general: the tail is handled one by one)
    int t = 0;
    for (; t + 8 <= kk; t += 8) {
#pragma unroll
      for (int u = 0; u < 8; ++u) rank += sel[t + u] > me ? 1 : 0;
    }
    for (; t < kk; ++t) rank += sel[t] > me ? 1 : 0;
    oi[rank] = int32_t(0xFFFFFFFFu - uint32_t(me));
    os[rank] = key_score(uint32_t(me >> 32));
  }
}

// ---------------------------------------------------------------- top-k, long rows
// Rows of more than 4096 keys: instead of holding the row in registers (which
// limits a compute unit to two rows at a time), the row is streamed once.
//  1. Threshold t from a sample: blocks of 64 consecutive rows at a fixed spacing
//     (at most 2048 sampled rows, one load per thread); t is the r-th largest
//     sampled key cut to its top 16 bits, r a few standard deviations above the
//     expected number of sampled keys among the kk largest.
//  2. Stream the row once, appending every key >= t to LDS as the unique 48-bit
//     value (key, 0xFFFF - row) (positions from one LDS counter per wave and
//     chunk: the order does not matter, the final rank sort sets it).
//  3. Radix select of the kk-th largest appended value (8 bits per pass); the kk
//     values at or above it are the result (ties between equal scores go to the
//     lower row through the 48-bit value).
// When the sample gives no usable t (fewer than kk or more than TK_CAP keys
// >= t), a streaming exhaustive search takes over: the largest t with at least
// kk keys >= t, one bit per pass over the row, then every key above t and the
// lowest rows equal to it (an ordered compaction, chunk by chunk).
constexpr int TS_THREADS = 512;
constexpr int TS_NW = TS_THREADS / WAVE;
constexpr int TK_CAP = 2048;            // appended keys at most (else the exhaustive search)
constexpr int TS_CH = TS_THREADS * 4;   // rows per streamed chunk (4 per thread)
constexpr int TS_SBLK = 64;             // sampled rows come in blocks of 64

// Keys of rows r0 .. r0 + 3 (r0 a multiple of 4); rows past L get key 0, which
// lies below every score.  One buffer load over the row (its stride, a multiple
// of 64 that is >= L, in bytes as the range: reads past it return zeros).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const float* srow, int64_t ld) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(srow), (short)0, int(ld * 4),
                                           0x00020000);
}
__device__ __forceinline__ void load_keys4(__amdgpu_buffer_rsrc_t rs, int r0, int L,
                                           uint32_t (&kv)[4]) {
  const float4 v = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, r0 * 4, 0, 0));
  kv[0] = r0 < L ? score_key(v.x) : 0u;
  kv[1] = r0 + 1 < L ? score_key(v.y) : 0u;
  kv[2] = r0 + 2 < L ? score_key(v.z) : 0u;
  kv[3] = r0 + 3 < L ? score_key(v.w) : 0u;
}
// Block-wide sum of a wave-uniform count (one value per wave); red[parity] must
// not be in use by the previous call (alternate the parity).
__device__ __forceinline__ int block_sum_waves(int cnt, int* red, int lane, int wid) {
  if (lane == 0) red[wid] = cnt;
  __syncthreads();
  int tot = 0;
#pragma unroll
  for (int w = 0; w < TS_NW; ++w) tot += red[w];
  return tot;
}
__device__ __forceinline__ int lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi(uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0));
}

__global__ __launch_bounds__(TS_THREADS) void topk_stream_kernel(
    const float* __restrict__ scores, int64_t ld, const int64_t* __restrict__ cand_off,
    const int32_t* __restrict__ seq_len, int max_len, int k, int32_t* __restrict__ out_idx,
    float* __restrict__ out_score, int out_ld, int32_t* __restrict__ cand_req) {
  __shared__ int red[2][TS_NW];
  __shared__ uint64_t scan_w[TS_NW];
  __shared__ __attribute__((aligned(16))) uint64_t sel[TAV2_K_MAX];
  __shared__ uint64_t cand[TK_CAP];
  __shared__ uint32_t hist[256];
  __shared__ int misc[4];   // radix digit, rest, selected count, appended count

  const int r = blockIdx.y;
  const int64_t n = cand_off[r] + blockIdx.x;
  if (n >= cand_off[r + 1]) return;
  if (cand_req && threadIdx.x == 0) cand_req[n] = r;   // the candidate's request, for the encoder
  const int L = min(seq_len[r], max_len);
  const int tid = threadIdx.x, lane = tid % WAVE, wid = tid / WAVE;
  const int kk = k < L ? k : L;
  int32_t* oi = out_idx + n * out_ld;
  float* os = out_score + n * out_ld;
  for (int p = kk + tid; p < k; p += TS_THREADS) {
    oi[p] = -1;
    os[p] = -__builtin_inff();
  }
  if (kk == 0) return;
  const __amdgpu_buffer_rsrc_t rs = row_rsrc(scores + n * ld, ld);
  const int nch = (L + TS_CH - 1) / TS_CH;
  int par = 0;   // parity of the next block_sum_waves buffer

  // 1. threshold from the sample (rows of a short row all survive: key >= 1)
  bool ok = true;
  uint32_t thr = 1;
  if (L > TK_CAP) {
    const int sp = TS_SBLK * ((L + TK_CAP - 1) / TK_CAP);   // block spacing: <= 32 blocks
    const int j0 = 4 * tid;                                 // sample slots j0 .. j0 + 3
    uint32_t smp[4];
    load_keys4(rs, sp * (j0 / TS_SBLK) + j0 % TS_SBLK, L, smp);
    const int nb = (L + sp - 1) / sp;
    const int ns = (nb - 1) * TS_SBLK + min(TS_SBLK, L - (nb - 1) * sp);   // sampled rows < L
    const float expct = float(kk) * float(ns) / float(L);
    const int rr = int(expct + 4.f * sqrtf(expct) + 8.f);
    if (rr > ns) {
      ok = false;
    } else {
      thr = 0;
      for (int b = 31; b >= 16; --b) {
        const uint32_t probe = thr | (1u << b);
        int cnt = 0;
#pragma unroll
        for (int u = 0; u < 4; ++u) cnt += __popcll(__builtin_amdgcn_ballot_w64(smp[u] >= probe));
        if (block_sum_waves(cnt, red[par], lane, wid) >= rr) thr = probe;
        par ^= 1;
      }
      if (thr == 0) thr = 1;
    }
  }

  // 2. stream the row, appending the keys >= thr
  if (ok) {
    if (tid == 0) misc[3] = 0;
    __syncthreads();
    for (int c = 0; c < nch; ++c) {
      const int r0 = c * TS_CH + 4 * tid;
      uint32_t kv[4];
      load_keys4(rs, r0, L, kv);
      uint64_t bm[4];
      int tot = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        bm[u] = __builtin_amdgcn_ballot_w64(kv[u] >= thr);
        tot += __popcll(bm[u]);
      }
      if (tot == 0) continue;   // wave-uniform
      int base = 0;             // one counter update per wave and chunk
      if (lane == 0) base = atomicAdd(&misc[3], tot);
      base = __shfl(base, 0, WAVE);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int pos = base + lanes_below(bm[u]);
        if (kv[u] >= thr && pos < TK_CAP)
          cand[pos] = (uint64_t(kv[u]) << 16) | uint64_t(0xFFFFu - uint32_t(r0 + u));
        base += __popcll(bm[u]);
      }
    }
    __syncthreads();
    const int clo = misc[3];
    if (clo < kk || clo > TK_CAP) ok = false;
    if (ok) {
      // 3. radix select of the kk-th largest 48-bit value, most significant byte first
      uint64_t pre = 0;
      int need = kk;
      for (int sh = 40; sh >= 0; sh -= 8) {
        if (tid < 256) hist[tid] = 0;
        __syncthreads();
        for (int i = tid; i < clo; i += TS_THREADS) {
          const uint64_t v = cand[i];
          if ((v >> (sh + 8)) == pre) atomicAdd(&hist[(v >> sh) & 255u], 1u);
        }
        __syncthreads();
        if (wid == 0) {   // bins in descending order: lane l holds 255 - 4l - q
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
      // exactly kk values are >= pre
      if (tid == 0) misc[2] = 0;
      __syncthreads();
      for (int i = tid; i < clo; i += TS_THREADS) {
        const uint64_t v = cand[i];
        if (v >= pre) {
          const uint32_t kv = uint32_t(v >> 16), row = 0xFFFFu - uint32_t(v & 0xFFFFu);
          sel[atomicAdd(&misc[2], 1)] = (uint64_t(kv) << 32) | uint64_t(0xFFFFFFFFu - row);
        }
      }
      __syncthreads();
    }
  }

  if (!ok) {
    // exhaustive: largest t with count(key >= t) >= kk, one bit (one pass) at a time
    uint32_t t = 0;
    for (int b = 31; b >= 0; --b) {
      const uint32_t probe = t | (1u << b);
      int cnt = 0;
      for (int c = 0; c < nch; ++c) {
        uint32_t kv[4];
        load_keys4(rs, c * TS_CH + 4 * tid, L, kv);
#pragma unroll
        for (int u = 0; u < 4; ++u) cnt += __popcll(__builtin_amdgcn_ballot_w64(kv[u] >= probe));
      }
      if (block_sum_waves(cnt, red[par], lane, wid) >= kk) t = probe;
      par ^= 1;
    }
    // every key above t (any order), then the need_eq lowest rows equal to t
    int gt = 0;
    for (int c = 0; c < nch; ++c) {
      uint32_t kv[4];
      load_keys4(rs, c * TS_CH + 4 * tid, L, kv);
#pragma unroll
      for (int u = 0; u < 4; ++u) gt += __popcll(__builtin_amdgcn_ballot_w64(kv[u] > t));
    }
    const int count_gt = block_sum_waves(gt, red[par], lane, wid);
    par ^= 1;
    const int need_eq = kk - count_gt;
    if (tid == 0) misc[2] = 0;
    __syncthreads();
    int eq_before = 0;   // equal keys in earlier chunks (block-uniform)
    for (int c = 0; c < nch; ++c) {
      const int r0 = c * TS_CH + 4 * tid;
      uint32_t kv[4];
      load_keys4(rs, r0, L, kv);
      uint64_t bm[4];
      int tot = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        bm[u] = __builtin_amdgcn_ballot_w64(kv[u] > t);
        tot += __popcll(bm[u]);
      }
      if (tot > 0) {   // wave-uniform
        int base = 0;
        if (lane == 0) base = atomicAdd(&misc[2], tot);
        base = __shfl(base, 0, WAVE);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (kv[u] > t)
            sel[base + lanes_below(bm[u])] =
                (uint64_t(kv[u]) << 32) | uint64_t(0xFFFFFFFFu - uint32_t(r0 + u));
          base += __popcll(bm[u]);
        }
      }
      // equal keys in row order: rows of the chunk are ordered by (thread, u)
      uint64_t e[1] = {0}, excl[1], total[1];
#pragma unroll
      for (int u = 0; u < 4; ++u) e[0] += kv[u] == t ? 1u : 0u;
      block_excl_scan<1>(e, excl, total, scan_w, lane, wid);
      int pos = eq_before + int(excl[0]);
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (kv[u] == t) {
          if (pos < need_eq)
            sel[count_gt + pos] = (uint64_t(kv[u]) << 32) | uint64_t(0xFFFFFFFFu - uint32_t(r0 + u));
          ++pos;
        }
      eq_before += int(total[0]);
      __syncthreads();   // scan_w is rewritten by the next chunk's scan
    }
  }

  // survivors are distinct under (key, -row): rank = number of survivors before it
  for (int s = tid; s < kk; s += TS_THREADS) {
    const uint64_t me = sel[s];
    int rank = 0;
    int t = 0;
    for (; t + 8 <= kk; t += 8) {
#pragma unroll
      for (int u = 0; u < 8; ++u) rank += sel[t + u] > me ? 1 : 0;
    }
    for (; t < kk; ++t) rank += sel[t] > me ? 1 : 0;
    oi[rank] = int32_t(0xFFFFFFFFu - uint32_t(me));
    os[rank] = key_score(uint32_t(me >> 32));
  }
}

// ---------------------------------------------------------------- launchers
// Allow a kernel its largest dynamic LDS (`lds`: the size at the largest d) on the
// current device, once per device (done[dev]).  Every caller sets the same value,
// so calls from several host threads at most repeat the attribute call.
static hipError_t allow_dynamic_lds(const void* kernel, size_t lds, std::atomic<bool>* done) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const bool cached = dev >= 0 && dev < 64;
  if (cached && done[dev].load(std::memory_order_acquire)) return hipSuccess;
  e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  if (cached) done[dev].store(true, std::memory_order_release);
  return hipSuccess;
}

hipError_t launch_scores(const tav2_seq& seq, const tav2_cands& c, float* scores, int64_t ld,
                         hipStream_t st) {
  if (seq.num_requests == 0 || c.total == 0 || seq.max_len == 0) return hipSuccess;
  if (seq.dtype == TAV2_BF16) {
    dim3 grid(unsigned(cdiv(seq.max_len, SC_ROWS)), unsigned(cdiv(c.max_count, SC_CANDS)),
              unsigned(seq.num_requests));
    ProfScope prof("score_bf16", st);
    const size_t lds = size_t(SC_CANDS) * size_t(seq.d + SC_PAD) * 2;   // d <= 512: <= 133 KB
    static std::atomic<bool> lds_done[64] = {};
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(score_bf16_kernel),
                                           size_t(SC_CANDS) * (512 + SC_PAD) * 2, lds_done);
    if (e != hipSuccess) return e;
    score_bf16_kernel<<<grid, 256, lds, st>>>(
        static_cast<const bf16_t*>(seq.emb), seq.offset, seq.len,
        static_cast<const bf16_t*>(c.emb), c.offset, seq.d, seq.max_len, scores, ld);
  } else if (seq.dtype == TAV2_I8) {
    dim3 grid(unsigned(cdiv(seq.max_len, SI_ROWS)), unsigned(cdiv(c.max_count, SI_CANDS)),
              unsigned(seq.num_requests));
    ProfScope prof("score_i8", st);
    const size_t lds = size_t(SI_CANDS) * SI_SLD * 4 + size_t(SI_CANDS) * size_t(seq.d + SC_PAD) * 2;
    static std::atomic<bool> lds_done[64] = {};
    const hipError_t e = allow_dynamic_lds(
        reinterpret_cast<const void*>(score_i8_kernel),
        size_t(SI_CANDS) * SI_SLD * 4 + size_t(SI_CANDS) * (512 + SC_PAD) * 2, lds_done);
    if (e != hipSuccess) return e;
    score_i8_kernel<<<grid, 256, lds, st>>>(
        static_cast<const int8_t*>(seq.emb), seq.offset, seq.len,
        static_cast<const bf16_t*>(c.emb), c.offset, seq.d, seq.max_len, scores, ld);
  } else {
    dim3 grid(unsigned(cdiv(seq.max_len, 256)), unsigned(c.max_count), unsigned(seq.num_requests));
    ProfScope prof("score_f32", st);
    score_f32_kernel<<<grid, 256, 0, st>>>(
        static_cast<const float*>(seq.emb), seq.offset, seq.len,
        static_cast<const float*>(c.emb), c.offset, seq.d, seq.max_len, scores, ld);
  }
  return hipGetLastError();
}

hipError_t launch_topk(const tav2_seq& seq, const tav2_cands& c, const float* scores, int64_t ld,
                       int k, int32_t* out_idx, float* out_score, int out_ld, int32_t* cand_req,
                       hipStream_t st) {
  if (seq.num_requests == 0 || c.total == 0) return hipSuccess;
  dim3 grid(unsigned(c.max_count), unsigned(seq.num_requests));
  const int per = int(cdiv(seq.max_len > 0 ? seq.max_len : 1, TK_THREADS));
  ProfScope prof("topk", st);
#define TAV2_TOPK(PT) \
  topk_kernel<PT><<<grid, TK_THREADS, 0, st>>>(scores, ld, c.offset, seq.len, seq.max_len, k, \
                                               out_idx, out_score, out_ld, cand_req)
  if (per <= 4) TAV2_TOPK(4);
  else if (per <= 8) TAV2_TOPK(8);
  else
    topk_stream_kernel<<<grid, TS_THREADS, 0, st>>>(scores, ld, c.offset, seq.len, seq.max_len, k,
                                                     out_idx, out_score, out_ld, cand_req);
#undef TAV2_TOPK
  return hipGetLastError();
}

int64_t score_ld(int32_t max_len) { return int64_t(align_up(size_t(max_len > 0 ? max_len : 1), 64)); }

}  // namespace tav2
