// NN search of Eq. 3 for long request sequences with the score products kept on
// chip: only each candidate's few hundred best rows ever reach memory.
//
// Per candidate the search needs its k largest scores under the order (score
// desc, row asc).  A row can only be among them if its score is at least the
// k-th largest, so a lower bound t on that value lets the score GEMM drop every
// row below t as soon as its product is formed.  The launches:
//  1. sample: scores of a fixed sample of the request's rows (up to 32 blocks of
//     32 consecutive rows, evenly spaced), kept as the top 16 bits of their keys;
//  2. threshold: per candidate, t = the r-th largest sampled key cut to 16 bits,
//     with r a few standard deviations above the expected number of sampled rows
//     among the k best (the whole row sampled: r = k exactly);
//  3. filter: the full score GEMM; each product's key is compared with its
//     candidate's t in the epilogue and the survivors, as 48-bit (key, row)
//     values, are appended to the candidate's list (staged per workgroup in LDS,
//     one global counter update per candidate and workgroup);
//  4. select: per candidate, when the list holds at least k values and did not
//     overflow, every one of the k best rows is in it (at least k keys are >= t,
//     so the k-th largest key is >= t); a radix select over the list finds them
//     and they are placed by rank.  Otherwise the candidate is queued;
//  5. fallback: each queued candidate's scores are recomputed into LDS with the
//     same products (bit-identical keys) and searched exhaustively.
// The result is exact in every case; the threshold only decides how much work
// the exact part does.
#include <atomic>

#include "common.h"
#include "internal.h"
#include "select_common.h"

namespace tav2 {

constexpr int FS_BLK = 32;                  // rows per sampled block
constexpr int FS_MAXBLK = 32;               // sampled blocks per request at most
constexpr int FS_NS = FS_BLK * FS_MAXBLK;   // sampled rows at most
constexpr int FS_PAD = 8;                   // LDS row padding (bf16) of candidate tiles
constexpr int FB_CANDS = 128;               // bf16: candidates per tile
constexpr int FB_ROWS = 256;                // bf16 filter: rows per workgroup (4 waves x 64)
constexpr int FB_SROWS = 64;                // bf16 sample: slots per workgroup (wave w: tile w)
constexpr int FI_CANDS = 32;                // int8: candidates per tile
constexpr int FI_ROWS = 256;                // int8: rows (or slots) per workgroup
constexpr int FF_THREADS = 512;             // fallback kernel
constexpr int FF_GRID = 64;                 // fallback workgroups (each loops over the queue)
constexpr int FS_FILTER_D = 8;              // bf16 filter: sequence k-blocks in flight

int64_t fused_cap(int k) { return int64_t(align_up(size_t(2 * k + 1024), 64)); }
constexpr int FS_CAP_MAX = 2 * TAV2_K_MAX + 1024;

// Sample geometry of a request of L rows: the row's 32-row blocks are sampled
// every q-th block (q = 1: all of them), nsb blocks, ns rows.
struct SampleGeom {
  int q, nsb, ns;
};
__host__ __device__ __forceinline__ SampleGeom sample_geom(int L) {
  if (L <= 0) return SampleGeom{1, 0, 0};
  const int nblk = (L + FS_BLK - 1) / FS_BLK;
  const int q = (nblk + FS_MAXBLK - 1) / FS_MAXBLK;
  const int nsb = (nblk + q - 1) / q;
  const int last = (nsb - 1) * q;   // index of the last sampled block
  const int tail = L - last * FS_BLK < FS_BLK ? L - last * FS_BLK : FS_BLK;
  return SampleGeom{q, nsb, (nsb - 1) * FS_BLK + tail};
}
// Sequence row of sample slot s (>= L for the slots past the row's end).
__device__ __forceinline__ int sample_row(int s, int q) {
  return (s / FS_BLK) * q * FS_BLK + s % FS_BLK;
}

struct FusedArgs {
  const void* emb;             // sequence rows (bf16 or int8 codes)
  const int64_t* seq_off;
  const int32_t* seq_len;
  const bf16_t* cand;          // [total, d]
  const int64_t* cand_off;     // [R + 1]
  int d, max_len, k, cap;
  int out_ld;                  // row stride of the outputs (>= k)
  uint16_t* samp;              // [total][FS_NS] top 16 bits of the sampled keys
  uint32_t* thr;               // [total] threshold key
  uint32_t* cnt;               // [total] survivors appended (may exceed cap)
  uint64_t* surv;              // [total][cap] survivor values
  int32_t* fb;                 // [total][2] queued (candidate, request) pairs
  uint32_t* nfb;               // queued candidates
};

// Candidate tile [nc rows][d + FS_PAD] of bf16 in LDS (rows past the request's
// candidates repeat its last one).  Each thread issues up to CT_BATCH 16-byte
// loads before it stores any of them, so their memory latencies overlap.
constexpr int CT_BATCH = 16;
__device__ __forceinline__ void load_cand_tile(bf16_t* ctile, const bf16_t* cand, int64_t n0,
                                               int64_t c_end, int nc, int d) {
  const int cld = d + FS_PAD, per_row = d / 8, total = nc * per_row;
  for (int base = 0; base < total; base += 256 * CT_BATCH) {
    uint4 v[CT_BATCH];
#pragma unroll
    for (int u = 0; u < CT_BATCH; ++u) {
      const int e = base + 256 * u + int(threadIdx.x);
      const int row = e / per_row, c = e - row * per_row;
      int64_t n = n0 + row;
      n = n < c_end ? n : c_end - 1;
      v[u] = e < total ? *reinterpret_cast<const uint4*>(cand + n * d + c * 8) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < CT_BATCH; ++u) {
      const int e = base + 256 * u + int(threadIdx.x);
      const int row = e / per_row, c = e - row * per_row;
      if (e < total) *reinterpret_cast<uint4*>(ctile + row * cld + c * 8) = v[u];
    }
  }
}

// ---------------------------------------------------------------- products
// bf16: acc[a][b] = S_b C_a^T for the two 32-row sequence tiles b (A operand:
// brow[b] at the lane's row and k-half) and candidate tiles a (B operand: 32
// candidates from LDS, arow pointing at the lane's candidate and k-half of tile
// 0), over the nkb k-blocks in ascending order.  D register 4j + i of lane l
// holds row 8j + 4(l / 32) + i of its row tile and candidate l % 32 of its
// tile, so a lane keeps one candidate's scores of 16 rows per tile pair.  (Each
// product depends only on its own row, candidate and k-block order: the
// fallback recomputes the same bits with a one-candidate B operand.)
// The sequence fragments stream from memory D k-blocks ahead of their use (slot
// u of the ring holds k-blocks u, u + D, ...); the caller issues the first D
// (bf16_prefetch) before it stages the candidate tile, so their latency overlaps
// that.
template <int D>
__device__ __forceinline__ void bf16_prefetch(bf16x8 (&bq)[D][2], const bf16_t* brow0,
                                              const bf16_t* brow1, int nkb) {
#pragma unroll
  for (int u = 0; u < D; ++u)
    if (u < nkb) {
      bq[u][0] = as_bf16x8(*reinterpret_cast<const uint4*>(brow0 + 16 * u));
      bq[u][1] = as_bf16x8(*reinterpret_cast<const uint4*>(brow1 + 16 * u));
    }
}
template <int NA, int D>
__device__ __forceinline__ void bf16_products(const bf16_t* arow, int cld, const bf16_t* brow0,
                                              const bf16_t* brow1, int nkb, bf16x8 (&bq)[D][2],
                                              f32x16 (&acc)[NA][2]) {
#pragma unroll
  for (int a = 0; a < NA; ++a) acc[a][0] = acc[a][1] = f32x16{};
  bf16x8 av[NA];
#pragma unroll
  for (int a = 0; a < NA; ++a) av[a] = as_bf16x8(*reinterpret_cast<const uint4*>(arow + a * 32 * cld));
  for (int kb0 = 0; kb0 < nkb; kb0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int kb = kb0 + u;
      if (kb < nkb) {   // wave-uniform
        bf16x8 an[NA];
        const int ka = kb + 1 < nkb ? kb + 1 : kb;   // next k-block's candidate fragments
#pragma unroll
        for (int a = 0; a < NA; ++a)
          an[a] = as_bf16x8(*reinterpret_cast<const uint4*>(arow + a * 32 * cld + 16 * ka));
#pragma unroll
        for (int a = 0; a < NA; ++a) {
          acc[a][0] = mfma32(bq[u][0], av[a], acc[a][0]);
          acc[a][1] = mfma32(bq[u][1], av[a], acc[a][1]);
        }
        const int kn = kb + D;
        if (kn < nkb) {
          bq[u][0] = as_bf16x8(*reinterpret_cast<const uint4*>(brow0 + 16 * kn));
          bq[u][1] = as_bf16x8(*reinterpret_cast<const uint4*>(brow1 + 16 * kn));
        }
#pragma unroll
        for (int a = 0; a < NA; ++a) av[a] = an[a];
      }
    }
  }
}

// int8 codes: acc[b] = C S_b^T (one 32-candidate tile) with the lane's partial
// sums of squares sq[b]; the full sum of a row's squares is sq + the partner
// lane's (l ^ 32).
__device__ __forceinline__ void i8_products(const bf16_t* arow, const int8_t* brow0,
                                            const int8_t* brow1, int d, f32x16 (&acc)[2],
                                            float (&sq)[2]) {
  acc[0] = acc[1] = f32x16{};
  sq[0] = sq[1] = 0.f;
  uint2 raw[2], nxt[2];
  raw[0] = *reinterpret_cast<const uint2*>(brow0);
  raw[1] = *reinterpret_cast<const uint2*>(brow1);
  for (int k0 = 0; k0 < d; k0 += 16) {
    const int kn = k0 + 16 < d ? k0 + 16 : k0;
    nxt[0] = *reinterpret_cast<const uint2*>(brow0 + kn);
    nxt[1] = *reinterpret_cast<const uint2*>(brow1 + kn);
    const bf16x8 av = as_bf16x8(*reinterpret_cast<const uint4*>(arow + k0));
    acc[0] = mfma32(av, codes_to_bf16(raw[0], sq[0]), acc[0]);
    acc[1] = mfma32(av, codes_to_bf16(raw[1], sq[1]), acc[1]);
    raw[0] = nxt[0];
    raw[1] = nxt[1];
  }
}

// ---------------------------------------------------------------- 1. sample
// bf16: wave w = candidate tile w (32 candidates) x 64 sample slots, the
// workgroup's 4 waves over the same slots (their row loads after the first hit
// L1).  The operands come straight from memory, D k-blocks ahead of their use:
// each wave is the only reader of its candidates.  The products are the
// filter's (same operands, same k-block order).  samp[n][s0 .. s0 + 63] gets
// the top 16 bits of the keys of those slots in some order within each 32-slot
// tile (0 for slots past the row's end, below every score's key); the
// threshold takes a candidate's keys as a multiset.
constexpr int FS_SAMPLE_D = 16;   // k-blocks in flight (all of them at d <= 256)
__global__ __launch_bounds__(256) void fsel_sample_bf16(FusedArgs A) {
  const int r = blockIdx.z;
  const int w = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  const int hf = lane / 32, l32 = lane % 32;
  const int64_t c_end = A.cand_off[r + 1];
  const int64_t nt = A.cand_off[r] + int64_t(blockIdx.y) * FB_CANDS + 32 * w;
  if (nt >= c_end) return;   // wave-uniform
  const int L = min(A.seq_len[r], A.max_len);
  const SampleGeom g = sample_geom(L);
  const int s0 = blockIdx.x * FB_SROWS;
  if (s0 >= g.nsb * FS_BLK) return;
  const int d = A.d, nkb = d / 16;
  const bf16_t* seq = static_cast<const bf16_t*>(A.emb) + A.seq_off[r] * int64_t(d);
  const bf16_t* brow[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int sl = s0 + 32 * b + l32;
    const int row = sample_row(sl, g.q);
    const bool ok = sl < g.nsb * FS_BLK && row < L;
    brow[b] = seq + int64_t(ok ? row : L - 1) * d + 8 * hf;
  }
  const int64_t n = nt + l32;
  const bf16_t* crow = A.cand + (n < c_end ? n : c_end - 1) * d + 8 * hf;
  constexpr int D = FS_SAMPLE_D;
  bf16x8 q0[D], q1[D], qc[D];
#pragma unroll
  for (int u = 0; u < D; ++u)
    if (u < nkb) {
      q0[u] = as_bf16x8(*reinterpret_cast<const uint4*>(brow[0] + 16 * u));
      q1[u] = as_bf16x8(*reinterpret_cast<const uint4*>(brow[1] + 16 * u));
      qc[u] = as_bf16x8(*reinterpret_cast<const uint4*>(crow + 16 * u));
    }
  f32x16 acc[2] = {f32x16{}, f32x16{}};
  for (int kb0 = 0; kb0 < nkb; kb0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int kb = kb0 + u;
      if (kb < nkb) {   // wave-uniform
        acc[0] = mfma32(q0[u], qc[u], acc[0]);
        acc[1] = mfma32(q1[u], qc[u], acc[1]);
        const int kn = kb + D;
        if (kn < nkb) {
          q0[u] = as_bf16x8(*reinterpret_cast<const uint4*>(brow[0] + 16 * kn));
          q1[u] = as_bf16x8(*reinterpret_cast<const uint4*>(brow[1] + 16 * kn));
          qc[u] = as_bf16x8(*reinterpret_cast<const uint4*>(crow + 16 * kn));
        }
      }
    }
  }
  if (n >= c_end) return;
  // register 4 j + i of tile b: slot s0 + 32 b + 8 j + 4 hf + i; stored at
  // position 16 hf + 4 j + i of the tile, two 16-byte stores per tile
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    uint32_t wd[8];
#pragma unroll
    for (int reg = 0; reg < 16; reg += 2) {
      uint32_t k2[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int sl = s0 + 32 * b + 8 * ((reg + e) / 4) + 4 * hf + (reg + e) % 4;
        const bool valid = sl < g.nsb * FS_BLK && sample_row(sl, g.q) < L;
        k2[e] = valid ? score_key(acc[b][reg + e]) >> 16 : 0u;
      }
      wd[reg / 2] = k2[0] | (k2[1] << 16);
    }
    uint4* dst = reinterpret_cast<uint4*>(A.samp + n * FS_NS + s0 + 32 * b + 16 * hf);
    dst[0] = make_uint4(wd[0], wd[1], wd[2], wd[3]);
    dst[1] = make_uint4(wd[4], wd[5], wd[6], wd[7]);
  }
}

// int8: workgroup = 32 candidates x 256 sample slots (wave w: slots 64 w ..).
__global__ __launch_bounds__(256) void fsel_sample_i8(FusedArgs A) {
  extern __shared__ __attribute__((aligned(16))) uint8_t fs_smem[];
  bf16_t* ctile = reinterpret_cast<bf16_t*>(fs_smem);
  const int r = blockIdx.z;
  const int64_t c_begin = A.cand_off[r], c_end = A.cand_off[r + 1];
  const int64_t n0 = c_begin + int64_t(blockIdx.y) * FI_CANDS;
  if (n0 >= c_end) return;
  const int L = min(A.seq_len[r], A.max_len);
  const SampleGeom g = sample_geom(L);
  const int sb = blockIdx.x * FI_ROWS;
  if (sb >= g.nsb * FS_BLK) return;
  const int d = A.d, cld = d + FS_PAD;
  load_cand_tile(ctile, A.cand, n0, c_end, FI_CANDS, d);
  __syncthreads();
  const int w = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  const int hf = lane / 32, l32 = lane % 32;
  const int8_t* seq = static_cast<const int8_t*>(A.emb) + A.seq_off[r] * int64_t(d);
  const int s0 = sb + 64 * w;
  int row[2];
  bool ok[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int s = s0 + 32 * b + l32;
    row[b] = sample_row(s, g.q);
    ok[b] = s < g.nsb * FS_BLK && row[b] < L;
  }
  f32x16 acc[2];
  float sq[2];
  i8_products(ctile + l32 * cld + 8 * hf, seq + int64_t(ok[0] ? row[0] : L - 1) * d + 8 * hf,
              seq + int64_t(ok[1] ? row[1] : L - 1) * d + 8 * hf, d, acc, sq);
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int s = s0 + 32 * b + l32;
    const float ss = sq[b] + __shfl_xor(sq[b], 32, WAVE);   // the row's other half
#pragma unroll
    for (int reg = 0; reg < 16; ++reg) {
      const int64_t n = n0 + 8 * (reg / 4) + 4 * hf + (reg % 4);
      if (n < c_end && s < FS_NS)
        A.samp[n * FS_NS + s] = ok[b] ? uint16_t(score_key(i8_score(acc[b][reg], ss)) >> 16) : 0;
    }
  }
}

// ---------------------------------------------------------------- 2. threshold
// One wave per candidate: t = the rr-th largest sampled 16-bit key (two radix
// digits through a histogram of the wave's own in LDS), as a 32-bit key
// threshold.  kk = 0: nothing survives; rr beyond the sample: everything does.
// Also clears the candidate's survivor count and (first wave) the queue count.
__global__ __launch_bounds__(256) void fsel_threshold(FusedArgs A) {
  __shared__ __attribute__((aligned(16))) uint32_t th_hist[4][256];
  const int r = blockIdx.y;
  const int w = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  if (blockIdx.x == 0 && r == 0 && threadIdx.x == 0) *A.nfb = 0u;
  const int64_t n = A.cand_off[r] + int64_t(blockIdx.x) * 4 + w;
  if (n >= A.cand_off[r + 1]) return;   // wave-uniform
  const int L = min(A.seq_len[r], A.max_len);
  const int kk = A.k < L ? A.k : L;
  uint32_t t;
  if (kk == 0) {
    t = 0xFFFFFFFFu;
  } else {
    const SampleGeom g = sample_geom(L);
    int rr = kk;
    if (g.q > 1) {
      const float e = float(kk) * float(g.ns) / float(L);
      rr = int(e + 4.f * sqrtf(e) + 8.f);
    }
    if (rr > g.ns) {
      t = 0u;
    } else {
      // the lane's 16 slots: 8 lane + 512 j + 0..7 (slots past the sample: key 0,
      // below every sampled key that can count)
      const int nslots = g.nsb * FS_BLK;   // a multiple of 8
      uint32_t kw[8];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int s = 8 * lane + 512 * j;
        const uint4 q = s < nslots ? *reinterpret_cast<const uint4*>(A.samp + n * FS_NS + s)
                                   : make_uint4(0u, 0u, 0u, 0u);
        kw[4 * j] = q.x;
        kw[4 * j + 1] = q.y;
        kw[4 * j + 2] = q.z;
        kw[4 * j + 3] = q.w;
      }
      uint32_t* h = th_hist[w];
      *reinterpret_cast<uint4*>(h + 4 * lane) = make_uint4(0u, 0u, 0u, 0u);
      wave_lds_sync();
#pragma unroll
      for (int i = 0; i < 16; ++i) atomicAdd(&h[(kw[i / 2] >> (16 * (i % 2) + 8)) & 255u], 1u);
      wave_lds_sync();
      uint32_t hi, rest;
      radix_digit(h, uint32_t(rr), hi, rest);
      wave_lds_sync();
      *reinterpret_cast<uint4*>(h + 4 * lane) = make_uint4(0u, 0u, 0u, 0u);
      wave_lds_sync();
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const uint32_t key = (kw[i / 2] >> (16 * (i % 2))) & 0xFFFFu;
        if ((key >> 8) == hi) atomicAdd(&h[key & 255u], 1u);
      }
      wave_lds_sync();
      uint32_t lo, rest2;
      radix_digit(h, rest, lo, rest2);
      t = ((hi << 8) | lo) << 16;
    }
  }
  if (lane == 0) {
    A.thr[n] = t;
    A.cnt[n] = 0u;
  }
}

// ---------------------------------------------------------------- 3. filter
// bf16: workgroup = 32 NA candidates (NA = 4, or 2 when that gives too few
// workgroups to fill the GPU) x 256 rows, wave w rows 64 w .. +63.  A lane
// holds candidates l % 32 + 32 a (a < NA) for 32 of the wave's rows (half
// l / 32 of every 8-row group), so its survivors go to its own LDS segments, one
// per (candidate, wave, half), each with a lane-private counter.  The hot loop is
// branch-free: every score is written, to the segment's next slot when it
// survives and to the segment's last slot (never read) when it does not, and the
// counter advances by the compare's result.  A segment keeps FS_LSEG - 1
// survivors (the expected count is about one); a lane with more goes through
// its scores again and sends the rest straight to the candidate's list in
// memory.  Scores are compared as floats with the threshold's value (keys and
// floats are ordered alike), and staged as raw bits with their row.
constexpr int FS_LSEG = 8;
template <int NA>
constexpr int filter_nseg() { return 32 * NA * 4 * 2; }   // (candidate, wave, half)
template <int NA>
__host__ __device__ __forceinline__ int filter_bf16_lds(int d) {
  constexpr int NC = 32 * NA, NSEG = filter_nseg<NA>();
  const int tile = NC * (d + FS_PAD) * 2, stage = NSEG * FS_LSEG * 8;
  return (tile > stage ? tile : stage) + NC * 4 + 2 * NSEG * 4;
}
// Float value a 32-bit threshold key stands for: key 0 lets every score through
// (-inf), key 0xFFFFFFFF none (NaN compares false).
__device__ __forceinline__ float threshold_value(uint32_t t) {
  if (t == 0u) return -__builtin_inff();
  if (t == 0xFFFFFFFFu) return __builtin_nanf("");
  return key_score(t);
}

template <int NA>
__global__ __launch_bounds__(256, 2) void fsel_filter_bf16(FusedArgs A) {
  constexpr int NC = 32 * NA, NSEG = filter_nseg<NA>();
  extern __shared__ __attribute__((aligned(16))) uint8_t fs_smem[];
  const int d = A.d, cld = d + FS_PAD;
  const int tile_b = NC * cld * 2, stage_b = NSEG * FS_LSEG * 8;
  const int region = tile_b > stage_b ? tile_b : stage_b;
  bf16_t* ctile = reinterpret_cast<bf16_t*>(fs_smem);
  uint2* stage = reinterpret_cast<uint2*>(fs_smem);                 // {row, score bits}
  float* thr_f = reinterpret_cast<float*>(fs_smem + region);          // [NC]
  uint32_t* scnt = reinterpret_cast<uint32_t*>(thr_f + NC);           // [NSEG]
  uint32_t* soff = scnt + NSEG;                                       // [NSEG]
  const int r = blockIdx.z;
  const int64_t c_begin = A.cand_off[r], c_end = A.cand_off[r + 1];
  const int64_t n0 = c_begin + int64_t(blockIdx.y) * NC;
  if (n0 >= c_end) return;
  const int L = min(A.seq_len[r], A.max_len);
  const int ib = blockIdx.x * FB_ROWS;
  if (ib >= L) return;
  const int tid = threadIdx.x;
  if (tid < NC) {   // tile columns past the request's candidates keep nothing
    const int64_t n = n0 + tid;
    thr_f[tid] = threshold_value(n < c_end ? A.thr[n] : 0xFFFFFFFFu);
  }
  const int w = tid / WAVE, lane = tid % WAVE;
  const int hf = lane / 32, l32 = lane % 32;
  const int row0 = ib + 64 * w;
  const bool active = row0 < L;
  const bf16_t* seq = static_cast<const bf16_t*>(A.emb) + A.seq_off[r] * int64_t(d);
  const int i0 = min(row0 + l32, L - 1), i1 = min(row0 + 32 + l32, L - 1);   // clamped; not kept
  const bf16_t* brow0 = seq + int64_t(i0) * d + 8 * hf;
  const bf16_t* brow1 = seq + int64_t(i1) * d + 8 * hf;
  bf16x8 bq[FS_FILTER_D][2];
  if (active) bf16_prefetch<FS_FILTER_D>(bq, brow0, brow1, d / 16);
  load_cand_tile(ctile, A.cand, n0, c_end, NC, d);
  __syncthreads();
  f32x16 acc[NA][2];
  if (active)
    bf16_products<NA, FS_FILTER_D>(ctile + l32 * cld + 8 * hf, cld, brow0, brow1, d / 16, bq, acc);
  __syncthreads();   // the candidate tile's region now stages survivors
  // segment of (candidate 32 a + l32, wave w, half hf): lane-consecutive, and the
  // stage slot-major, so that a wave's 64 slot writes are one contiguous 512 bytes
  constexpr uint32_t KEEP = FS_LSEG - 1;   // survivors a segment keeps
  auto seg_of = [](int a, int wv, int l, int h) { return ((a * 4 + wv) * 32 + l) * 2 + h; };
  uint32_t cnt[NA] = {};
  if (active) {
    // register 4 j + i of row tile b holds row row0 + 32 b + 8 j + 4 hf + i
    uint32_t rowok[2] = {0u, 0u};
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int reg = 0; reg < 16; ++reg)
        rowok[b] |= uint32_t(row0 + 32 * b + 8 * (reg / 4) + 4 * hf + (reg % 4) < L) << reg;
#pragma unroll
    for (int a = 0; a < NA; ++a) {
      const int c = 32 * a + l32;
      const float t = thr_f[c];
      uint2* seg = stage + seg_of(a, w, l32, hf);
      uint32_t m = 0;
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int reg = 0; reg < 16; ++reg) {
          const float sc = acc[a][b][reg];
          const bool keep = sc >= t && ((rowok[b] >> reg) & 1u);
          const int row = row0 + 32 * b + 8 * (reg / 4) + 4 * hf + (reg % 4);
          seg[(keep ? min(m, KEEP) : KEEP) * NSEG] = make_uint2(uint32_t(row), __float_as_uint(sc));
          m += keep ? 1u : 0u;
        }
      cnt[a] = m;
      if (m > KEEP) {   // rare: the survivors past the segment's slots go to memory
        uint32_t q = 0;
        const int64_t n = n0 + c;
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) {
            const float sc = acc[a][b][reg];
            if (sc >= t && ((rowok[b] >> reg) & 1u)) {
              if (q >= KEEP) {
                const int row = row0 + 32 * b + 8 * (reg / 4) + 4 * hf + (reg % 4);
                const uint32_t gp = atomicAdd(&A.cnt[n], 1u);
                if (gp < uint32_t(A.cap)) A.surv[n * A.cap + gp] = sel_value(score_key(sc), row);
              }
              ++q;
            }
          }
      }
    }
  }
#pragma unroll
  for (int a = 0; a < NA; ++a) scnt[seg_of(a, w, l32, hf)] = min(cnt[a], KEEP);
  __syncthreads();
  if (tid < NC) {   // one counter update per candidate; its segments' offsets
    const int a = tid / 32, l = tid % 32;
    uint32_t m = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int sg = seg_of(a, q / 2, l, q % 2);
      soff[sg] = m;
      m += scnt[sg];
    }
    const uint32_t base = m ? atomicAdd(&A.cnt[n0 + tid], m) : 0u;
#pragma unroll
    for (int q = 0; q < 8; ++q) soff[seg_of(a, q / 2, l, q % 2)] += base;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < NSEG / 256; ++q) {   // segment sg = tid + 256 q
    const int sg = tid + 256 * q;
    const uint32_t m = scnt[sg], base = soff[sg];
    const int64_t n = n0 + 32 * (sg / 256) + (sg / 2) % 32;
    for (uint32_t i = 0; i < m; ++i) {
      const uint2 e = stage[i * NSEG + sg];
      if (base + i < uint32_t(A.cap))
        A.surv[n * A.cap + base + i] = sel_value(score_key(__uint_as_float(e.y)), int(e.x));
    }
  }
}

// int8: workgroup = 32 candidates x 256 rows, wave w rows 64 w .. +63.  D
// register 4 j + i of row tile b of a lane holds candidate 8 j + 4 hf + i and
// the lane's row 32 b + l32, so for one register and lane half every lane has
// the same candidate: the lanes whose score may survive are compacted with a
// ballot into that (candidate, wave, row tile) segment of LDS, no atomics.  The
// estimate (the hardware reciprocal square root) keeps every score within 64
// units in the last place of the threshold (estimate and score have the same sign
// and differ by a few units in the last place, relative error below 2^-21, and
// keys of same-signed scores are ordered like their ulp counts); the staged ones
// then get the exact score (a correctly rounded square root and division) and
// those below the threshold are dropped before the counts are published.
constexpr int FI_SLOTS = 8;                           // staged entries per segment
constexpr int FI_NSEG = FI_CANDS * 4 * 2;             // (candidate, wave, row tile)
__host__ __device__ __forceinline__ int filter_i8_lds(int d) {
  const int tile = FI_CANDS * (d + FS_PAD) * 2, stage = FI_NSEG * FI_SLOTS * 8;
  return (tile > stage ? tile : stage) + 2 * FI_CANDS * 4 + 2 * FI_NSEG * 4 + FI_ROWS * 4 +
         FI_CANDS * 4;
}
__global__ __launch_bounds__(256) void fsel_filter_i8(FusedArgs A) {
  extern __shared__ __attribute__((aligned(16))) uint8_t fs_smem[];
  const int d = A.d, cld = d + FS_PAD;
  const int tile_b = FI_CANDS * cld * 2, stage_b = FI_NSEG * FI_SLOTS * 8;
  const int region = tile_b > stage_b ? tile_b : stage_b;
  bf16_t* ctile = reinterpret_cast<bf16_t*>(fs_smem);
  uint2* stage = reinterpret_cast<uint2*>(fs_smem);                   // {row, dot bits | key}
  uint32_t* thr_s = reinterpret_cast<uint32_t*>(fs_smem + region);    // [FI_CANDS] keys
  float* thr_e = reinterpret_cast<float*>(thr_s + FI_CANDS);          // [FI_CANDS]
  uint32_t* scnt = reinterpret_cast<uint32_t*>(thr_e + FI_CANDS);     // [FI_NSEG]
  uint32_t* soff = scnt + FI_NSEG;                                    // [FI_NSEG]
  float* ssr = reinterpret_cast<float*>(soff + FI_NSEG);              // [FI_ROWS] row sums of squares
  uint32_t* cbase = reinterpret_cast<uint32_t*>(ssr + FI_ROWS);       // [FI_CANDS]
  const int r = blockIdx.z;
  const int64_t c_begin = A.cand_off[r], c_end = A.cand_off[r + 1];
  const int64_t n0 = c_begin + int64_t(blockIdx.y) * FI_CANDS;
  if (n0 >= c_end) return;
  const int L = min(A.seq_len[r], A.max_len);
  const int ib = blockIdx.x * FI_ROWS;
  if (ib >= L) return;
  const int tid = threadIdx.x;
  if (tid < FI_CANDS) {
    // the key threshold t, and the float an estimate must reach to come within
    // 64 units in the last place of it (keys and floats are ordered alike)
    const int64_t n = n0 + tid;
    const uint32_t t = n < c_end ? A.thr[n] : 0xFFFFFFFFu;
    thr_s[tid] = t;
    thr_e[tid] = threshold_value(t < 64u ? 0u : t - 64u);
  }
  load_cand_tile(ctile, A.cand, n0, c_end, FI_CANDS, d);
  __syncthreads();
  const int w = tid / WAVE, lane = tid % WAVE;
  const int hf = lane / 32, l32 = lane % 32;
  const int row0 = ib + 64 * w;
  const bool active = row0 < L;
  const int8_t* seq = static_cast<const int8_t*>(A.emb) + A.seq_off[r] * int64_t(d);
  f32x16 acc[2];
  float sq[2] = {0.f, 0.f};
  if (active) {
    const int i0 = min(row0 + l32, L - 1), i1 = min(row0 + 32 + l32, L - 1);
    i8_products(ctile + l32 * cld + 8 * hf, seq + int64_t(i0) * d + 8 * hf,
                seq + int64_t(i1) * d + 8 * hf, d, acc, sq);
  }
  __syncthreads();   // the candidate tile's region now stages survivors
  uint32_t cnt_reg[2][4][4];   // per (row tile, j, i): this lane half's staged count
  if (active) {
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const float ss = sq[b] + __shfl_xor(sq[b], 32, WAVE);
      if (hf == 0) ssr[64 * w + 32 * b + l32] = ss;
      const float rs = ss > 0.f ? __builtin_amdgcn_rsqf(ss) : 0.f;
      const int row = row0 + 32 * b + l32;
      const bool row_ok = row < L;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 e4 = *reinterpret_cast<const float4*>(thr_e + 8 * j + 4 * hf);
        const float ev[4] = {e4.x, e4.y, e4.z, e4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int c = 8 * j + 4 * hf + i;
          const float dot = acc[b][4 * j + i];
          const bool maybe = row_ok && dot * rs >= ev[i];
          const uint64_t bm = __builtin_amdgcn_ballot_w64(maybe);
          const uint32_t lo = uint32_t(bm), hi = uint32_t(bm >> 32);
          const uint32_t pos = hf ? __builtin_amdgcn_mbcnt_hi(hi, 0u)
                                  : __builtin_amdgcn_mbcnt_lo(lo, 0u);
          const int sg = (c * 4 + w) * 2 + b;
          if (maybe && pos < uint32_t(FI_SLOTS))
            stage[sg * FI_SLOTS + pos] = make_uint2(uint32_t(row), __float_as_uint(dot));
          cnt_reg[b][j][i] = uint32_t(__popc(hf ? hi : lo));
          if (maybe && pos >= uint32_t(FI_SLOTS)) {   // rare: past the segment, to memory
            const uint32_t key = score_key(i8_score(dot, ss));
            if (key >= thr_s[c]) {
              const int64_t n = n0 + c;
              const uint32_t gp = atomicAdd(&A.cnt[n], 1u);
              if (gp < uint32_t(A.cap)) A.surv[n * A.cap + gp] = sel_value(key, row);
            }
          }
        }
      }
    }
  }
  if (l32 == 0) {   // lanes 0 and 32 publish their half's segment counts
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int sg = ((8 * j + 4 * hf + i) * 4 + w) * 2 + b;
          scnt[sg] = active ? min(cnt_reg[b][j][i], uint32_t(FI_SLOTS)) : 0u;
        }
  }
  __syncthreads();
  {   // the exact score of each staged entry (thread = segment); survivors compacted
    const int sg = tid;
    const int c = sg / 8;   // segment (c, wave, row tile)
    const uint32_t t = thr_s[c];
    const uint32_t m = scnt[sg];
    uint32_t kept = 0;
    for (uint32_t q = 0; q < m; ++q) {
      const uint2 e = stage[sg * FI_SLOTS + q];
      const float ss = ssr[int(e.x) - ib];
      const uint32_t key = score_key(i8_score(__uint_as_float(e.y), ss));
      if (key >= t) stage[sg * FI_SLOTS + (kept++)] = make_uint2(e.x, key);
    }
    scnt[sg] = kept;
  }
  __syncthreads();
  if (tid < FI_CANDS) {   // one counter update per candidate
    uint32_t m = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      soff[tid * 8 + q] = m;
      m += scnt[tid * 8 + q];
    }
    cbase[tid] = m ? atomicAdd(&A.cnt[n0 + tid], m) : 0u;
  }
  __syncthreads();
  {
    const int sg = tid, c = sg / 8;
    const uint32_t m = scnt[sg], base = cbase[c] + soff[sg];
    const int64_t n = n0 + c;
    for (uint32_t q = 0; q < m; ++q) {
      const uint2 e = stage[sg * FI_SLOTS + q];
      if (base + q < uint32_t(A.cap)) A.surv[n * A.cap + base + q] = sel_value(e.y, int(e.x));
    }
  }
}

// ---------------------------------------------------------------- 4. select
// One workgroup per candidate: the k best of its survivors (a radix select of
// the k-th largest, the values at or above it, placed by rank), or the queue.
constexpr int FT_THREADS = 256;
__global__ __launch_bounds__(FT_THREADS) void fsel_select(FusedArgs A, int32_t* __restrict__ out_idx,
                                                          float* __restrict__ out_score,
                                                          int32_t* __restrict__ cand_req) {
  __shared__ uint64_t vals[FS_CAP_MAX];
  __shared__ __attribute__((aligned(16))) uint64_t sel[TAV2_K_MAX];
  __shared__ __attribute__((aligned(16))) uint32_t hist[3 * 256];
  __shared__ uint64_t red[2 * FT_THREADS / WAVE];
  __shared__ int nsel;
  const int r = blockIdx.y;
  const int64_t n = A.cand_off[r] + blockIdx.x;
  if (n >= A.cand_off[r + 1]) return;
  const int tid = threadIdx.x, lane = tid % WAVE;
  if (cand_req && tid == 0) cand_req[n] = r;   // the candidate's request, for the encoder
  const int L = min(A.seq_len[r], A.max_len);
  const int k = A.k;
  const int kk = k < L ? k : L;
  int32_t* oi = out_idx + n * A.out_ld;
  float* os = out_score + n * A.out_ld;
  for (int p = kk + tid; p < k; p += FT_THREADS) {
    oi[p] = -1;
    os[p] = -__builtin_inff();
  }
  if (kk == 0) return;
  const uint32_t cnt = A.cnt[n];
  if (cnt < uint32_t(kk) || cnt > uint32_t(A.cap)) {
    if (tid == 0) {
      const uint32_t q = atomicAdd(A.nfb, 1u);
      A.fb[2 * q] = int32_t(n);
      A.fb[2 * q + 1] = r;
    }
    return;
  }
  const int m = int(cnt);
  {   // every load of the list in flight before the first store
    constexpr int PER = FS_CAP_MAX / FT_THREADS;
    uint64_t v[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = tid + FT_THREADS * u;
      if (i < m) v[u] = A.surv[n * A.cap + i];
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = tid + FT_THREADS * u;
      if (i < m) vals[i] = v[u];
    }
  }
  if (tid == 0) nsel = 0;
  const uint64_t pre = radix_select48<FT_THREADS>(vals, m, kk, hist, red);
  // the values at or above the kk-th largest: exactly kk of them (one counter
  // update per wave and round)
  for (int i0 = 0; i0 < m; i0 += FT_THREADS) {
    const int i = i0 + tid;
    const bool take = i < m && vals[i] >= pre;
    const uint64_t bm = __builtin_amdgcn_ballot_w64(take);
    if (bm) {   // wave-uniform
      int base = 0;
      if (lane == 0) base = atomicAdd(&nsel, __popcll(bm));
      base = __shfl(base, 0, WAVE);
      const int pos = base + int(__builtin_amdgcn_mbcnt_hi(uint32_t(bm >> 32),
                                                           __builtin_amdgcn_mbcnt_lo(uint32_t(bm), 0)));
      if (take) sel[pos] = vals[i];
    }
  }
  __syncthreads();
  place_by_rank<FT_THREADS>(sel, kk, oi, os);
}

// ---------------------------------------------------------------- 5. fallback
// Queued candidates, one per workgroup at a time: every row's key recomputed
// into LDS with the filter's products (the candidate in every row of the A
// operand: each output element depends only on its own row and column, so the
// keys are the filter's bit for bit), then the exhaustive search: the largest t
// with at least kk keys >= t (one bit at a time), every key above t and the
// lowest rows equal to it (in row order), placed by rank.
__device__ __forceinline__ int ff_block_sum(int v, int* red) {
  const int lane = threadIdx.x % WAVE, wid = threadIdx.x / WAVE;
  v = wave_sum_i(v);
  __syncthreads();   // red may still be read by the previous call
  if (lane == 0) red[wid] = v;
  __syncthreads();
  int tot = 0;
#pragma unroll
  for (int w = 0; w < FF_THREADS / WAVE; ++w) tot += red[w];
  return tot;
}

template <bool I8>
__global__ __launch_bounds__(FF_THREADS) void fsel_fallback(FusedArgs A, int32_t* __restrict__ out_idx,
                                                            float* __restrict__ out_score,
                                                            int keys_ld) {
  extern __shared__ __attribute__((aligned(16))) uint8_t ff_smem[];
  uint32_t* keys = reinterpret_cast<uint32_t*>(ff_smem);                       // [keys_ld]
  uint64_t* sel = reinterpret_cast<uint64_t*>(ff_smem + size_t(keys_ld) * 4);  // [K_MAX]
  __shared__ int red[FF_THREADS / WAVE];
  __shared__ int wtot[FF_THREADS / WAVE];
  __shared__ int misc[2];
  const int tid = threadIdx.x, w = tid / WAVE, lane = tid % WAVE;
  const int hf = lane / 32, l32 = lane % 32;
  const uint32_t nq = *A.nfb;
  const int d = A.d;
  for (uint32_t q = blockIdx.x; q < nq; q += gridDim.x) {
    const int64_t n = A.fb[2 * q];
    const int r = A.fb[2 * q + 1];
    const int L = min(A.seq_len[r], A.max_len);
    const int kk = A.k < L ? A.k : L;   // >= 1: only such candidates are queued
    // 1. keys of every row
    const bf16_t* crow = A.cand + n * d + 8 * hf;
    for (int t0 = 32 * w; t0 < L; t0 += 32 * (FF_THREADS / WAVE)) {
      int row = t0 + l32;
      const int rc = row < L ? row : L - 1;
      float s;
      if constexpr (!I8) {
        // the filter's orientation: rows in the A operand, the candidate in every
        // column of B; register 4 j + i of either half holds row 8 j + 4 hf + i,
        // and lane l32 < 16 reports register l32
        const bf16_t* brow = static_cast<const bf16_t*>(A.emb) + (A.seq_off[r] + rc) * int64_t(d) + 8 * hf;
        f32x16 acc = f32x16{};
        for (int k0 = 0; k0 < d; k0 += 16)
          acc = mfma32(as_bf16x8(*reinterpret_cast<const uint4*>(brow + k0)),
                       as_bf16x8(*reinterpret_cast<const uint4*>(crow + k0)), acc);
        s = acc[0];
#pragma unroll
        for (int q = 1; q < 16; ++q) s = l32 == q ? acc[q] : s;
        row = t0 + 8 * ((l32 & 15) / 4) + 4 * hf + (l32 & 3);
        if (l32 >= 16) row = L;   // nothing to report
      } else {
        const int8_t* brow = static_cast<const int8_t*>(A.emb) + (A.seq_off[r] + rc) * int64_t(d) + 8 * hf;
        f32x16 acc = f32x16{};
        float sq = 0.f;
        for (int k0 = 0; k0 < d; k0 += 16)
          acc = mfma32(as_bf16x8(*reinterpret_cast<const uint4*>(crow + k0)),
                       codes_to_bf16(*reinterpret_cast<const uint2*>(brow + k0), sq), acc);
        s = i8_score(acc[0], sq + __shfl_xor(sq, 32, WAVE));
        if (hf) row = L;   // both halves hold the row's score: half 0 reports it
      }
      if (row < L) keys[row] = score_key(s);
    }
    __syncthreads();
    // 2. the kk-th largest key
    uint32_t t = 0;
    for (int b = 31; b >= 0; --b) {
      const uint32_t probe = t | (1u << b);
      int c = 0;
      for (int i = tid; i < L; i += FF_THREADS) c += keys[i] >= probe ? 1 : 0;
      if (ff_block_sum(c, red) >= kk) t = probe;
    }
    int gt = 0;
    for (int i = tid; i < L; i += FF_THREADS) gt += keys[i] > t ? 1 : 0;
    const int count_gt = ff_block_sum(gt, red);
    const int need_eq = kk - count_gt;
    // 3. keys above t in any order, then the need_eq lowest rows equal to t
    if (tid == 0) misc[0] = 0;
    __syncthreads();
    for (int i = tid; i < L; i += FF_THREADS)
      if (keys[i] > t) sel[atomicAdd(&misc[0], 1)] = sel_value(keys[i], i);
    int eq_before = 0;
    for (int c0 = 0; c0 < L && eq_before < need_eq; c0 += FF_THREADS) {
      const int i = c0 + tid;
      const bool eq = i < L && keys[i] == t;
      const uint64_t bm = __builtin_amdgcn_ballot_w64(eq);
      __syncthreads();   // wtot may still be read by the previous chunk
      if (lane == 0) wtot[w] = __popcll(bm);
      __syncthreads();
      int before = eq_before, all = 0;
#pragma unroll
      for (int v = 0; v < FF_THREADS / WAVE; ++v) {
        before += v < w ? wtot[v] : 0;
        all += wtot[v];
      }
      const int pos = before + __builtin_amdgcn_mbcnt_hi(uint32_t(bm >> 32),
                                                         __builtin_amdgcn_mbcnt_lo(uint32_t(bm), 0));
      if (eq && pos < need_eq) sel[count_gt + pos] = sel_value(t, i);
      eq_before += all;
    }
    __syncthreads();
    place_by_rank<FF_THREADS>(sel, kk, out_idx + n * A.out_ld, out_score + n * A.out_ld);
    __syncthreads();   // keys and sel are rewritten by the next queued candidate
  }
}

// ---------------------------------------------------------------- host side
bool select_fused_applies(const tav2_seq& s) {
  return (s.dtype == TAV2_BF16 || s.dtype == TAV2_I8) && s.max_len > FUSED_MIN_LEN;
}

namespace {
struct FusedLayout {
  size_t samp, thr, cnt, surv, fb, nfb, total;
};
FusedLayout fused_layout(int64_t total, int k) {
  FusedLayout l{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align_up(bytes, 256);
    return at;
  };
  const size_t t = size_t(total);
  l.samp = take(t * FS_NS * 2);
  l.thr = take(t * 4);
  l.cnt = take(t * 4);
  l.surv = take(t * size_t(fused_cap(k)) * 8);
  l.fb = take(t * 8);
  l.nfb = take(4);
  l.total = off;
  return l;
}

// Allow a kernel `lds` bytes of dynamic LDS on the current device (once per
// device and kernel; every caller sets the same maximum).
hipError_t allow_lds(const void* kernel, size_t lds, std::atomic<bool>* done) {
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
}  // namespace

size_t select_fused_workspace(const tav2_cands& c, int k) {
  return fused_layout(c.total, k).total;
}

hipError_t launch_select_fused(const tav2_seq& seq, const tav2_cands& c, int k,
                               int32_t* out_idx, float* out_score, int out_ld, int32_t* cand_req,
                               void* ws, hipStream_t st) {
  if (seq.num_requests == 0 || c.total == 0) return hipSuccess;
  const FusedLayout lay = fused_layout(c.total, k);
  uint8_t* base = static_cast<uint8_t*>(ws);
  FusedArgs A{};
  A.emb = seq.emb;
  A.seq_off = seq.offset;
  A.seq_len = seq.len;
  A.cand = static_cast<const bf16_t*>(c.emb);
  A.cand_off = c.offset;
  A.d = seq.d;
  A.max_len = seq.max_len;
  A.k = k;
  A.cap = int(fused_cap(k));
  A.out_ld = out_ld;
  A.samp = reinterpret_cast<uint16_t*>(base + lay.samp);
  A.thr = reinterpret_cast<uint32_t*>(base + lay.thr);
  A.cnt = reinterpret_cast<uint32_t*>(base + lay.cnt);
  A.surv = reinterpret_cast<uint64_t*>(base + lay.surv);
  A.fb = reinterpret_cast<int32_t*>(base + lay.fb);
  A.nfb = reinterpret_cast<uint32_t*>(base + lay.nfb);
  const unsigned R = unsigned(seq.num_requests);
  const bool i8 = seq.dtype == TAV2_I8;
  const int d = seq.d;
  const int nct = i8 ? FI_CANDS : FB_CANDS;
  const unsigned ctiles = unsigned(cdiv(c.max_count, nct));
  // bf16 filter: 128-candidate tiles, unless that leaves fewer workgroups than two
  // per CU (few candidates): then 64
  const unsigned rblocks = unsigned(cdiv(seq.max_len, FB_ROWS));
  const bool narrow = !i8 && int64_t(R) * int64_t(ctiles) * rblocks < 512;
  const unsigned ftiles = narrow ? unsigned(cdiv(c.max_count, FB_CANDS / 2)) : ctiles;
  hipError_t e;
  {
    ProfScope prof("nn_sample", st);
    if (i8) {
      const size_t lds = size_t(nct) * (d + FS_PAD) * 2;
      const size_t lds_max = size_t(nct) * (512 + FS_PAD) * 2;
      static std::atomic<bool> done[64] = {};
      if ((e = allow_lds(reinterpret_cast<const void*>(fsel_sample_i8), lds_max, done))) return e;
      fsel_sample_i8<<<dim3(FS_NS / FI_ROWS, ctiles, R), 256, lds, st>>>(A);
    } else {
      fsel_sample_bf16<<<dim3(FS_NS / FB_SROWS, ctiles, R), 256, 0, st>>>(A);
    }
    if ((e = hipGetLastError())) return e;
  }
  {
    ProfScope prof("nn_threshold", st);
    fsel_threshold<<<dim3(unsigned(cdiv(c.max_count, 4)), R), 256, 0, st>>>(A);
    if ((e = hipGetLastError())) return e;
  }
  {
    ProfScope prof("nn_filter", st);
    if (i8) {
      const size_t lds = size_t(filter_i8_lds(d));
      const size_t lds_max = size_t(filter_i8_lds(512));
      static std::atomic<bool> done[64] = {};
      if ((e = allow_lds(reinterpret_cast<const void*>(fsel_filter_i8), lds_max, done))) return e;
      fsel_filter_i8<<<dim3(rblocks, ctiles, R), 256, lds, st>>>(A);
    } else if (narrow) {
      static std::atomic<bool> done[64] = {};
      if ((e = allow_lds(reinterpret_cast<const void*>(fsel_filter_bf16<2>),
                         size_t(filter_bf16_lds<2>(512)), done)))
        return e;
      fsel_filter_bf16<2><<<dim3(rblocks, ftiles, R), 256, size_t(filter_bf16_lds<2>(d)), st>>>(A);
    } else {
      static std::atomic<bool> done[64] = {};
      if ((e = allow_lds(reinterpret_cast<const void*>(fsel_filter_bf16<4>),
                         size_t(filter_bf16_lds<4>(512)), done)))
        return e;
      fsel_filter_bf16<4><<<dim3(rblocks, ftiles, R), 256, size_t(filter_bf16_lds<4>(d)), st>>>(A);
    }
    if ((e = hipGetLastError())) return e;
  }
  {
    ProfScope prof("nn_select", st);
    fsel_select<<<dim3(unsigned(c.max_count), R), FT_THREADS, 0, st>>>(A, out_idx, out_score,
                                                                        cand_req);
    if ((e = hipGetLastError())) return e;
  }
  {
    ProfScope prof("nn_fallback", st);
    const int keys_ld = int(align_up(size_t(seq.max_len), 4));
    const size_t lds = size_t(keys_ld) * 4 + size_t(TAV2_K_MAX) * 8;
    const size_t lds_max = size_t(SEL_MAX_LEN) * 4 + size_t(TAV2_K_MAX) * 8;
    const unsigned grid = unsigned(c.total < FF_GRID ? c.total : FF_GRID);
    if (i8) {
      static std::atomic<bool> done[64] = {};
      if ((e = allow_lds(reinterpret_cast<const void*>(fsel_fallback<true>), lds_max, done))) return e;
      fsel_fallback<true><<<grid, FF_THREADS, lds, st>>>(A, out_idx, out_score, keys_ld);
    } else {
      static std::atomic<bool> done[64] = {};
      if ((e = allow_lds(reinterpret_cast<const void*>(fsel_fallback<false>), lds_max, done))) return e;
      fsel_fallback<false><<<grid, FF_THREADS, lds, st>>>(A, out_idx, out_score, keys_ld);
    }
    if ((e = hipGetLastError())) return e;
  }
  return hipSuccess;
}

}  // namespace tav2
