// Fused bf16 encoder: one workgroup runs one candidate through feature encoding
// (Eq. 4, early fusion), every causal post-LN layer and the linear + max-pool head
// (Sec. 3.2.2) without writing activations to HBM.
//
// Layout of the work:
//  * The candidate's positions are processed in blocks of 128 tokens.  Under the
//    causal mask a block depends on earlier blocks only through their keys and
//    values, so each block runs through all layers in turn and leaves its K/V in a
//    per-candidate cache (workspace) for the blocks after it.
//  * 4 waves, one per SIMD, each with the full 512-register budget.  The fp32
//    residual stream of the block lives in registers as the transposed product
//    X^T [feature x token] (MFMA accumulator layout: one token per lane, 4
//    consecutive features per register group); wave w owns features 64 w .. +63
//    of all 128 tokens, so each weight fragment of these products is loaded by
//    one wave only.  LayerNorm over features is an in-lane sum, one cross-half
//    exchange and a 4-way exchange through LDS.
//  * Weights stream from L2 straight into registers: each call first packs every
//    matrix (and the side tables, transposed) into MFMA-fragment order (one
//    32 x 16 fragment = 1 KB contiguous, lane-major), so every fragment load is one
//    buffer load of 16 bytes per lane with the fragment offset in a scalar
//    register, and no weight tile passes through LDS or a barrier.  Each phase
//    keeps a fixed look-ahead of 16 fragments in flight and, in its last
//    iterations, starts the next phase's.
//  * LDS holds only activations: the bf16 copy of the block (MFMA operand), the
//    head group's Q / K / V^T, the attention output, the FFN hidden chunk, and
//    cached keys/values of earlier blocks during attention.  Every activation
//    write is 4 consecutive bf16 of one row: products whose consumer needs
//    [token][feature] are computed transposed (weights as MFMA A operand); V is
//    computed untransposed to give V^T [dim][token].
//  * Attention: 16x16x32 MFMAs; wave w owns query tiles w and 7 - w (16 queries
//    each, equal causal work for every wave).  S^T = K Q^T puts one query per lane
//    column, so softmax reductions are in-lane plus two lane-half exchanges, and
//    P^T feeds O^T = V^T P^T straight from the score registers with the matching
//    key order.  Keys are taken 128 at a time (one softmax max and rescale per
//    segment); the block's own keys come first, then earlier blocks' from the cache.
//  * Global loads complete in issue order, so loads whose data is needed soon are
//    issued before the weight look-ahead of the next phase (biases, LayerNorm
//    parameters, table rows), and stores of the K/V cache after it.
#pragma once

#include <type_traits>

#include "common.h"
#include "internal.h"
#include "token_source.h"

namespace tav2 {
namespace fz {

constexpr int DM = 256;          // d_model
constexpr int BT = 128;          // tokens per block
constexpr int NT = 256;          // threads (4 waves)
constexpr int XLD = DM + 8;      // Xs row stride (bf16 elements)
constexpr int QLD = 64 + 8;      // Qs / Ks / Os row stride (one 64-dim head group)
constexpr int VLD = BT + 8;      // Vts row stride
constexpr int FC = 256;          // FFN hidden units per chunk
constexpr int HLD = FC + 8;      // Hs row stride
constexpr int MAX_LAYERS = 8;
constexpr int KIN = 256;         // packed width of the token half of W_in (d zero-padded)
constexpr int N_ACT = 8;         // action-type table rows (types are clamped to 0..7)
constexpr int N_TIME = 64;       // time-bucket table rows (buckets are clamped to 0..63)
constexpr int AT_COLS = 80;      // packed [E_act^T | 0 | E_time^T] columns: 0..7, 16..79
constexpr int NKB_W = DM / 16 + 1;   // k-blocks per packed row of W_qkv, W_o, W_1: 16 + bias

constexpr int XS_BYTES = BT * XLD * 2;                 // 67584
constexpr int QS_BYTES = BT * QLD * 2;                 // 18432
constexpr int VS_BYTES = 64 * VLD * 2;                 // 17408
constexpr int SC_BYTES = 2 * QS_BYTES + VS_BYTES;      // 54272
constexpr int CS_BYTES = QS_BYTES + VS_BYTES;          // 35840: cached K / V^T chunk
constexpr int LDS_BYTES = XS_BYTES + SC_BYTES + CS_BYTES;
static_assert(LDS_BYTES <= 163840, "fused encoder exceeds the 160 KiB of LDS");
// During the FFN the hidden chunk fills the scratch region and runs on into the
// (then free) cache staging area, followed by the second LayerNorm's parameters.
static_assert(BT * HLD * 2 + 2 * DM * 4 <= SC_BYTES + CS_BYTES, "FFN chunk buffers do not fit");
static_assert(2 * BT * 4 * 4 <= QS_BYTES && 2 * DM * 4 <= CS_BYTES, "LayerNorm 1 buffers do not fit");
static_assert(BT * 8 + BT * 8 <= SC_BYTES, "encoding buffers do not fit");

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// The thread index through an empty asm: index and address arithmetic derived
// from it is recomputed inside each phase instead of being hoisted out of the
// block and layer loops (which would keep it live across the whole kernel).
__device__ __forceinline__ int otid() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

#define FZ_LANE_VARS                                                      \
  const int tid_ = otid();                                                \
  const int lane = tid_ % WAVE;                                           \
  const int w = __builtin_amdgcn_readfirstlane(tid_ / WAVE);              \
  const int hf = lane / 32, l32 = lane % 32;                              \
  const int fh = w & 1, th = w >> 1;                                      \
  (void)hf; (void)l32; (void)fh; (void)th;

__device__ __forceinline__ bf16x8 lfrag(const bf16_t* p) {   // 16 bytes from LDS
  return as_bf16x8(*reinterpret_cast<const uint4*>(p));
}
// Fragment `frag` (1 KB, 64 lanes x 16 bytes) of the packed weights: a buffer load
// with the fragment offset in a scalar register and the lane offset as the only
// per-lane address (loads past the packed region would return zeros).
__device__ __forceinline__ bf16x8 wfrag(int frag, int lane);
__device__ __forceinline__ void st4(bf16_t* p, float a, float b, float c, float d) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack2(a, b), pack2(c, d));
}
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }
// MFMA operand with bf16 1.0 at k-rows 0 and 1 of every row / column (lanes 0..31
// hold k-rows 0..7): multiplies a bias k-block fragment [b_hi, b_lo, 0 ...].
__device__ __forceinline__ bf16x8 bias_ones() {
  const unsigned v = (otid() % WAVE) < 32 ? 0x3F803F80u : 0u;
  return __builtin_bit_cast(bf16x8, u32x4{v, 0u, 0u, 0u});
}

struct LayerPk {        // first fragment of each packed matrix (last k-block: bias)
  int qkv;              // [768 rows][16 + 1 kb]
  int o;                // [256][16 + 1]
  int w1;               // [ffn][16 + 1]
  int w2;               // [256][ffn / 16 + 1]
};

struct Args {
  TokenSource s;
  const bf16_t* cand;       // [total, d]
  const bf16_t* W_in;       // [DM, 2d] (candidate half read directly)
  const float* b_in;
  const bf16_t* E_act;
  const bf16_t* E_time;     // may be null
  const bf16_t* E_pos;
  const float* b_pool;
  const float* cvec;        // [chunk, DM]: c W_in[:, d:]^T + b_in per candidate
  const bf16_t* pkw;        // packed weights (fragment order)
  unsigned pk_bytes;
  int pk_in;                // packed token half of W_in, [256][KIN / 16]
  int pk_pool;              // packed W_pool
  int pk_at;                // packed [E_act^T | E_time^T], [256][AT_COLS / 16]
  int pk_pos;               // packed E_pos^T, [256][pos_nkb]
  int pos_nkb;
  tav2_layer layers[MAX_LAYERS];   // LayerNorm vectors (biases are packed)
  LayerPk pk[MAX_LAYERS];
  int n_layers;
  int d;
  int dh;                   // head width, 32 or 64
  int ffn;
  int tpad;                 // cache stride in positions (T rounded up to BT)
  int64_t c0;               // first candidate of this launch
  bf16_t* kcache;           // [chunk][layers][tpad][DM], or null when T <= BT
  bf16_t* vcache;           // [chunk][layers][DM][tpad]
  float* out;               // [total, 2 DM]
};

__device__ __forceinline__ bf16x8 wfrag(int frag, int lane) {
  const Args* AK = (const Args*)(__builtin_amdgcn_kernarg_segment_ptr());
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(AK->pkw), (short)0, int(AK->pk_bytes), 0x00020000);
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, lane * 16, frag * 1024, 0));
}

// ---------------------------------------------------------------- weight stream
// Every GEMM phase streams its weight fragments from L2 into registers ahead of
// use, and its last iterations already load the head of the NEXT phase's stream
// into `pre`, so the stream keeps running across phase boundaries (attention,
// LayerNorm and block boundaries included).  The look-ahead is a fixed number of
// fragments (NSLOT), i.e. NSLOT / NR k-blocks for a phase with NR row tiles,
// which gives every phase about the same look-ahead in MFMA time.
constexpr int NSLOT = 16;
typedef bf16x8 Pre[NSLOT];

// Shape of a GEMM phase: NR weight fragments (row tiles) per k-block, NKB
// k-blocks.  Its look-ahead covers its first D k-blocks (by default as many as
// NSLOT fragments hold): slot i holds k-block i / NR, row tile i % NR, for i < U.
// NR = 0 stands for "no next phase".
constexpr int default_depth(int nr, int nkb) {
  return nr == 0 ? 0 : (NSLOT / nr < nkb ? NSLOT / nr : nkb);
}
template <int NR_, int NKB_, int D_ = default_depth(NR_, NKB_), bool BIAS_ = false>
struct Shape {
  static constexpr int NR = NR_, NKB = NKB_, D = D_;
  static constexpr bool BIAS = BIAS_;      // the last k-block is a bias k-block
  static constexpr int NX = NKB - BIAS;    // k-blocks of activations
  static constexpr int U = D * NR;
  static_assert(U <= NSLOT && D <= NKB, "look-ahead");
};
using NoPhase = Shape<0, 0>;
using ShEmb = Shape<2, KIN / 16>;       // token half of W_in
using ShTab = Shape<2, AT_COLS / 16>;   // [E_act | E_time]
using ShPos = Shape<2, BT / 16>;        // E_pos rows of the block's positions
// Phases whose last k-block is the bias k-block of their matrix: weight fragment
// = [b_hi, b_lo, 0 ...] per row (the two bf16 halves of the fp32 bias), times
// the constant operand bias_ones() (1.0 at k-rows 0 and 1), so the MFMA adds the
// bias to every token's accumulator.
using ShQkv = Shape<3, NKB_W, default_depth(3, NKB_W), true>;   // Q / K / V of one head group
using ShWo = Shape<2, 64 / 16>;                                 // W_o columns of one head group
using ShWoL = Shape<2, 64 / 16 + 1, default_depth(2, 5), true>;  // ... of the last one
using ShF1 = Shape<2, NKB_W, default_depth(2, NKB_W), true>;    // W_1 rows of one hidden chunk
// W_2 columns of one hidden chunk: half of it ahead, so that the L2 traffic of
// the two FFN phases is the same (each loads half of its own weights and half of
// the other's)
using ShF2 = Shape<2, FC / 16, FC / 32>;
using ShF2L = Shape<2, FC / 16 + 1, FC / 32, true>;   // ... of the last hidden chunk
static_assert(ShF1::D == DM / 32, "FFN look-ahead balance");
using ShPool = Shape<2, DM / 16>;       // W_pool

struct WSeg {                            // a phase's weight fragments (all wave-uniform)
  int P;                                 // first fragment of the packed matrix
  int nkb;                               // k-blocks per row of P
  int kb0;                               // first k-block of the phase
  int r0, r1, r2, r3;                    // packed row tiles (the phase uses NR of them)
};

__device__ __forceinline__ int seg_rt(const WSeg& s, int f) {
  return f == 0 ? s.r0 : f == 1 ? s.r1 : f == 2 ? s.r2 : s.r3;
}
template <class Sh>
__device__ __forceinline__ void seg_slot(Pre& pre, int i, const WSeg& s, int lane) {
  if constexpr (Sh::NR > 0)
    if (i < Sh::U) pre[i] = wfrag(s.P + seg_rt(s, i % Sh::NR) * s.nkb + s.kb0 + i / Sh::NR, lane);
}
template <class Sh>
__device__ __forceinline__ void seg_prime(Pre& pre, const WSeg& s, int lane) {
#pragma unroll
  for (int i = 0; i < NSLOT; ++i) seg_slot<Sh>(pre, i, s, lane);
}
// residual-shaped phase of wave w: row tiles 2w, 2w + 1 (features 64 w .. +63)
__device__ __forceinline__ WSeg seg_resid(int P, int nkb, int kb0, int w) {
  return WSeg{P, nkb, kb0, 2 * w, 2 * w + 1, 0, 0};
}
// FFN first layer, chunk c: hidden row tiles (FC / 32) c + 2w + 0..1
__device__ __forceinline__ WSeg seg_ffn1(int P, int c, int w) {
  static_assert(FC == 4 * 64, "one pair of hidden tiles per wave");
  const int r = c * (FC / 32) + 2 * w;
  return WSeg{P, NKB_W, 0, r, r + 1, 0, 0};
}
// Q / K / V of head group g for wave w: q_d, k_d, v_d (d = w >> 1) are the packed
// row tiles 8 part + 2g + d of [W_q | W_k | W_v] (part 0, 1, 2)
__device__ __forceinline__ WSeg seg_qkv(int P, int g, int w) {
  const int d = w >> 1;
  return WSeg{P, NKB_W, 0, 2 * g + d, 8 + 2 * g + d, 16 + 2 * g + d, 0};
}

// Iteration of phase Cur after whose MFMAs slot i of the next phase's look-ahead
// is loaded: spread evenly over Cur's last D iterations, but never before Cur has
// read the fragment the slot still holds.
template <class Cur, class Nxt>
constexpr int refill_at(int i) {
  int q = 0;
  while (Nxt::U * (q + 1) / Cur::D <= i) ++q;   // i in [U q / D, U (q + 1) / D)
  int j = Cur::NKB - Cur::D + q;
  if (i < Cur::U && i / Cur::NR > j) j = i / Cur::NR;
  return j;
}
// Weight fragment (k-block j, row tile f) of the running phase, by value (an
// array copy out of the look-ahead would merge into one wide copy that keeps the
// look-ahead in scratch memory).
template <class Cur>
__device__ __forceinline__ bf16x8 stream_frag(const bf16x8 (&wq)[Cur::NKB][Cur::NR],
                                              const Pre& pre, int j, int f) {
  constexpr int D = Cur::D, NR = Cur::NR;
  return j < D ? pre[(j < D ? j : 0) * NR + f] : wq[j][f];
}
// Loads issued at k-block j: k-block j + D of this phase, or (in the last D
// iterations) this iteration's share of the next phase's look-ahead.
template <class Cur, class Nxt>
__device__ __forceinline__ void stream_fetch(bf16x8 (&wq)[Cur::NKB][Cur::NR], Pre& pre,
                                             const WSeg& cur, const WSeg& nxt, int j, int lane) {
  constexpr int D = Cur::D, NKB = Cur::NKB;
  if (j + D < NKB) {
#pragma unroll
    for (int f = 0; f < Cur::NR; ++f)
      wq[j + D][f] = wfrag(cur.P + seg_rt(cur, f) * cur.nkb + cur.kb0 + j + D, lane);
  } else {
#pragma unroll
    for (int i = 0; i < NSLOT; ++i)   // constant bounds: unrolled before j is known
      if (i < Nxt::U && refill_at<Cur, Nxt>(i) == j) seg_slot<Nxt>(pre, i, nxt, lane);
  }
}

// Work a residual phase carries along: step(j) after the MFMAs of k-block j,
// finish() after the last k-block.
struct NoSide {
  __device__ __forceinline__ void step(int) {}
  __device__ __forceinline__ void finish() {}
};

// acc[ft][tt] += C^T: features 64 w + 32 ft (packed rows of cur), tokens 32 tt
// (rows of ACT in LDS, columns 16 j), over Cur::NKB k-blocks.
template <class Cur, class Nxt, class Side = NoSide>
__device__ __forceinline__ void resid_phase(f32x16 (&acc)[2][4], Pre& pre, const WSeg& cur,
                                            const WSeg& nxt, const bf16_t* ACT, int ald,
                                            Side&& side = Side{}) {
  static_assert(Cur::NR == 2, "residual phases have two row tiles per wave");
  FZ_LANE_VARS
  constexpr int NKB = Cur::NKB;
  bf16x8 wq[NKB][2];
  bf16x8 xq[NKB][4];
  const bf16_t* arow = ACT + l32 * ald + 8 * hf;
#pragma unroll
  for (int tt = 0; tt < 4; ++tt) xq[0][tt] = lfrag(arow + 32 * tt * ald);
#pragma unroll
  for (int j = 0; j < NKB; ++j) {
    if (j + 1 < Cur::NX) {
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) xq[j + 1][tt] = lfrag(arow + 32 * tt * ald + (j + 1) * 16);
    } else if (j + 1 < NKB) {   // the bias k-block
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) xq[j + 1][tt] = bias_ones();
    }
    // token tile by token tile: each tile's operand is last read two products into
    // the k-block rather than six, which leaves the register allocator more room
    {
      const bf16x8 a0 = stream_frag<Cur>(wq, pre, j, 0), a1 = stream_frag<Cur>(wq, pre, j, 1);
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        acc[0][tt] = mfma32(a0, xq[j][tt], acc[0][tt]);
        acc[1][tt] = mfma32(a1, xq[j][tt], acc[1][tt]);
      }
    }
    side.step(j);
    stream_fetch<Cur, Nxt>(wq, pre, cur, nxt, j, lane);
    sched_fence();
  }
  side.finish();
}

// ---------------------------------------------------------------- table rows
// The side tables enter the encoding as products with one-hot matrices built in
// registers: acc^T += E^T onehot, with E^T streamed like the weights.  For the
// 32x32x16 B operand a lane holds column l % 32 (a token) and k-rows
// 8 (l / 32) .. +7, so each fragment has at most one 1.0.
__device__ __forceinline__ bf16x8 onehot8(int idx) {   // 1.0 at element idx (none if outside 0..7)
  const unsigned one = 0x3F80u;                          // bf16 1.0
  u32x4 v;
  v.x = idx == 0 ? one : idx == 1 ? (one << 16) : 0u;
  v.y = idx == 2 ? one : idx == 3 ? (one << 16) : 0u;
  v.z = idx == 4 ? one : idx == 5 ? (one << 16) : 0u;
  v.w = idx == 6 ? one : idx == 7 ? (one << 16) : 0u;
  return __builtin_bit_cast(bf16x8, v);
}

// acc += E_act[act_t] + E_time[time_t] for the block's tokens: k-block 0 holds the
// 8 action types, k-blocks 1..4 the 64 time buckets (at columns 16 + bucket).
template <class Nxt>
__device__ __forceinline__ void table_phase(f32x16 (&acc)[2][4], Pre& pre, const WSeg& cur,
                                            const WSeg& nxt, const int* tinfo) {
  FZ_LANE_VARS
  constexpr int NKB = ShTab::NKB;
  bf16x8 wq[NKB][2];
  int ka[4], kt[4];   // the token's one-hot column, relative to this lane's k-rows
#pragma unroll
  for (int tt = 0; tt < 4; ++tt) {
    const int info = tinfo[tt * 32 + l32];
    ka[tt] = (info & 0xFF) - 8 * hf;
    kt[tt] = 16 + ((info >> 8) & 0xFF) - 8 * hf;
  }
#pragma unroll
  for (int j = 0; j < NKB; ++j) {
    bf16x8 b[4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) b[tt] = onehot8(j == 0 ? ka[tt] : kt[tt] - 16 * j);
#pragma unroll
    for (int ft = 0; ft < 2; ++ft) {
      const bf16x8 a = stream_frag<ShTab>(wq, pre, j, ft);
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) acc[ft][tt] = mfma32(a, b[tt], acc[ft][tt]);
    }
    stream_fetch<ShTab, Nxt>(wq, pre, cur, nxt, j, lane);
    sched_fence();
  }
}

// acc += E_pos[p0 + r] for the block's tokens r: the block's 128 positions are
// the 8 k-blocks of E_pos^T from position p0; k-block j only meets token tile j / 2.
template <class Nxt>
__device__ __forceinline__ void pos_phase(f32x16 (&acc)[2][4], Pre& pre, const WSeg& cur,
                                          const WSeg& nxt) {
  FZ_LANE_VARS
  constexpr int NKB = ShPos::NKB;
  bf16x8 wq[NKB][2];
#pragma unroll
  for (int j = 0; j < NKB; ++j) {
    const int tt = j >> 1;
    const bf16x8 b = onehot8(l32 - 16 * (j & 1) - 8 * hf);
#pragma unroll
    for (int ft = 0; ft < 2; ++ft)
      acc[ft][tt] = mfma32(stream_frag<ShPos>(wq, pre, j, ft), b, acc[ft][tt]);
    stream_fetch<ShPos, Nxt>(wq, pre, cur, nxt, j, lane);
    sched_fence();
  }
}

// ---------------------------------------------------------------- LayerNorm
// The sublayer's gain and offset (2 x DM floats) reach LDS through registers:
// each thread loads its two values before the sublayer's last GEMM phase and
// stores them after it, so the loads are older than that phase's look-ahead
// loads of the next weights and waiting for them never waits for the weight
// stream (vector memory loads complete in issue order).  (The sublayer's output
// bias is already in the accumulators: every packed matrix ends with a bias
// k-block.)
struct LnParams {
  float gain, off;
};
static_assert(NT == DM, "one LayerNorm parameter pair per thread");
__device__ __forceinline__ LnParams ln_params_load(const float* g, const float* b) {
  const int t = otid();
  return LnParams{g[t], b[t]};
}
__device__ __forceinline__ void ln_params_store(const LnParams& q, float* P) {
  const int t = otid();
  P[t] = q.gain;
  P[DM + t] = q.off;
}

// x <- LN(acc) with gain g and offset b over the 256 features of every token,
// with P = [g | b] in LDS; Xs <- bf16(x).  Each wave holds 64
// features of every token: per-token partial sums meet in LDS (red: [BT][4] sums,
// then [BT][4] sums of squares).  Ends with a barrier.
__device__ __forceinline__ void layer_norm(f32x16 (&acc)[2][4], const float* P, float* red,
                                           bf16_t* Xs) {
  FZ_LANE_VARS
  float s[4] = {0.f, 0.f, 0.f, 0.f}, ss[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ft = 0; ft < 2; ++ft)
#pragma unroll
    for (int r = 0; r < 16; ++r)
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        const float v = acc[ft][tt][r];
        s[tt] += v;
        ss[tt] = fmaf(v, v, ss[tt]);
      }
#pragma unroll
  for (int tt = 0; tt < 4; ++tt) {   // both lane halves end with the full sums
    s[tt] = xsum32(s[tt]);
    ss[tt] = xsum32(ss[tt]);
  }
#pragma unroll
  for (int tt = 0; tt < 4; ++tt)     // half 0 stores the sums, half 1 the squares
    red[hf * BT * 4 + (tt * 32 + l32) * 4 + w] = hf ? ss[tt] : s[tt];
  __syncthreads();
  float rstd[4], shift[4];   // x_hat = x rstd + shift
#pragma unroll
  for (int tt = 0; tt < 4; ++tt) {
    const int tok = tt * 32 + l32;
    const float4 a = *reinterpret_cast<const float4*>(red + tok * 4);
    const float4 b = *reinterpret_cast<const float4*>(red + BT * 4 + tok * 4);
    const float mean = ((a.x + a.y) + (a.z + a.w)) * (1.f / DM);
    const float var = fmaxf(((b.x + b.y) + (b.z + b.w)) * (1.f / DM) - mean * mean, 0.f);
    rstd[tt] = rsqrtf(var + 1e-5f);
    shift[tt] = -mean * rstd[tt];
  }
#pragma unroll
  for (int ft = 0; ft < 2; ++ft)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int f = 64 * w + ft * 32 + 8 * j + 4 * hf;
      const float4 gg = *reinterpret_cast<const float4*>(P + f);
      const float4 bb = *reinterpret_cast<const float4*>(P + DM + f);
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        const float v0 = fmaf(fmaf(acc[ft][tt][4 * j], rstd[tt], shift[tt]), gg.x, bb.x);
        const float v1 = fmaf(fmaf(acc[ft][tt][4 * j + 1], rstd[tt], shift[tt]), gg.y, bb.y);
        const float v2 = fmaf(fmaf(acc[ft][tt][4 * j + 2], rstd[tt], shift[tt]), gg.z, bb.z);
        const float v3 = fmaf(fmaf(acc[ft][tt][4 * j + 3], rstd[tt], shift[tt]), gg.w, bb.w);
        acc[ft][tt][4 * j] = v0;
        acc[ft][tt][4 * j + 1] = v1;
        acc[ft][tt][4 * j + 2] = v2;
        acc[ft][tt][4 * j + 3] = v3;
        st4(Xs + (tt * 32 + l32) * XLD + f, v0, v1, v2, v3);
      }
    }
  __syncthreads();
}

// ---------------------------------------------------------------- pooling
// Max over the block's valid tokens (token < nvalid) of Y^T = acc, folded into
// the lane's running maximum pm (b_pool is added to the final max: rounding is
// monotonic, so max(y + b) = max(y) + b exactly).  A lane's 32 values (its
// features' maxima over its 4 tokens) are max-reduced across the 32 lanes of its
// half with a transposing butterfly (each step halves the values a lane keeps),
// which leaves feature pool_feature() of the wave's 64 in each lane.
#define FZ_TMAX(HALF, MASK)                                                   \
  _Pragma("unroll") for (int k = 0; k < (HALF); ++k) {                        \
    const bool up = (l32 & (MASK)) != 0;                                      \
    const float keep = up ? v[k + (HALF)] : v[k];                             \
    const float send = up ? v[k] : v[k + (HALF)];                             \
    v[k] = vmax(keep, __shfl_xor(send, (MASK), WAVE));                       \
  }

__device__ __forceinline__ int pool_feature() {
  FZ_LANE_VARS
  // value index kept by the butterfly: bit i of l32 selected the upper half at
  // the step that halved 32 values to 16 >> i
  const int k = ((l32 & 1) << 4) | ((l32 & 2) << 2) | (l32 & 4) | ((l32 & 8) >> 2) |
                ((l32 & 16) >> 4);
  return 64 * w + (k >> 4) * 32 + 8 * ((k & 15) >> 2) + 4 * hf + (k & 3);
}
__device__ __forceinline__ float pool_block(f32x16 (&acc)[2][4], float pm, int nvalid) {
  FZ_LANE_VARS
  float v[32];
#pragma unroll
  for (int ft = 0; ft < 2; ++ft)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float m = -__builtin_inff();
#pragma unroll
      for (int tt = 0; tt < 4; ++tt)
        if (tt * 32 + l32 < nvalid) m = vmax(m, acc[ft][tt][r]);
      v[ft * 16 + r] = m;
    }
  FZ_TMAX(16, 1)
  FZ_TMAX(8, 2)
  FZ_TMAX(4, 4)
  FZ_TMAX(2, 8)
  FZ_TMAX(1, 16)
  return vmax(pm, v[0]);
}

// ---------------------------------------------------------------- attention
// Causal attention of the block's 128 queries in 8 tiles of 16; wave w owns tiles
// w and 7 - w, which together need the same number of causal key steps for every
// wave.  16x16x32 MFMAs: S^T tile = 16 keys x 16 queries, one query per lane
// column, keys 4 (lane / 16) + i in the tile's 4 registers.
typedef float f32x4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f32x4v mfma16(const bf16x8& a, const bf16x8& b, const f32x4v& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

template <int DH>
struct AttnState {
  bf16x8 qf[DH / 32];   // Q^T fragments (32 dims x 16 queries each)
  f32x4v o[DH / 16];    // O^T accumulators (16 dims x 16 queries each)
  float m, l;           // running max (log2 units) and this lane's partial sum
};

template <int DH>
__device__ __forceinline__ void attn_init(AttnState<DH>& st, const bf16_t* Qs, int col0, int qt) {
  const int lane = otid() % WAVE;
  const int gq = lane / 16, c16 = lane % 16;
#pragma unroll
  for (int kb = 0; kb < DH / 32; ++kb)
    st.qf[kb] = lfrag(Qs + (16 * qt + c16) * QLD + col0 + 32 * kb + 8 * gq);
#pragma unroll
  for (int t = 0; t < DH / 16; ++t) st.o[t] = f32x4v{0.f, 0.f, 0.f, 0.f};
  st.m = -__builtin_inff();
  st.l = 0.f;
}

// One segment of up to 128 keys of K (LDS [key][kld], head dims at col0) and V^T
// (LDS [dim][vld]) for each of the wave's two query tiles qa and qb, which see NPA
// and NPB pairs of 32 keys: S^T for the whole segment first, one row max and one
// rescale of l and O per segment, then P and O^T += V^T P^T per pair.  The pair
// counts are template parameters, so a tile's work is one branch-free block.
// S^T tile 2 kp + t holds keys 32 kp + 16 t + 4 gq + i; the P^T
// fragment of pair kp takes them in that order (keys 4gq.., then 16 + 4gq..), and
// V^T rows store each pair's keys in the same order (vpos), so a lane's V^T
// fragment is one 16-byte read.  exp2 is the hardware instruction (results below 2^-126
// flush to zero, far under the bf16 resolution of P).
//
// Causal mask (DQ = the query tile, or -1 for a segment of earlier keys): only
// the tile's last pair reaches past its first query.  Of its two 16-key halves,
// the half holding keys 16 DQ .. +15 is a triangle (key 4 gq + i of it is
// visible to the lane's query c16 iff 4 gq + i <= c16, the same four lane masks
// for every tile); the other half is entirely visible (odd DQ) or entirely
// masked (even DQ: no products, P = 0).  DQ = -2: no causal mask (the unmasked
// mode, one block only); keys at or past kvl (padding) are masked instead.
template <int DQ, int NP>
constexpr bool dead_half(int kp, int t) {   // all keys of S^T tile 2 kp + t masked
  return DQ >= 0 && (DQ & 1) == 0 && kp == NP - 1 && t == 1;
}
template <int DH, int DQ, int NP>
__device__ __forceinline__ void seg_scores(f32x4v (&s)[8], const AttnState<DH>& st,
                                           const bf16_t* Kl, int kld, int col0, int lane,
                                           int kvl) {
  const int gq = lane / 16, c16 = lane % 16;
#pragma unroll
  for (int kp = 0; kp < NP; ++kp)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if (dead_half<DQ, NP>(kp, t)) continue;
      f32x4v acc = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < DH / 32; ++kb)
        acc = mfma16(lfrag(Kl + (32 * kp + 16 * t + c16) * kld + col0 + 32 * kb + 8 * gq),
                     st.qf[kb], acc);
      s[2 * kp + t] = acc;
    }
  if constexpr (DQ >= 0) {
    constexpr int tri = 2 * (NP - 1) + (DQ & 1);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (4 * gq + i > c16) s[tri][i] = -__builtin_inff();
  }
  if constexpr (DQ == -2) {
#pragma unroll
    for (int q = 0; q < 2 * NP; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (16 * q + 4 * gq + i >= kvl) s[q][i] = -__builtin_inff();
  }
}
// FIRST: the tile's first segment (l and O still zero: no rescale).
template <int DH, int DQ, int NP, bool FIRST>
__device__ __forceinline__ float seg_rescale(AttnState<DH>& st, const f32x4v (&s)[8]) {
  constexpr float sc = (DH == 64 ? 0.125f : 0.17677669529663688f) * 1.4426950408889634f;
  float mx = -__builtin_inff();
#pragma unroll
  for (int q = 0; q < 2 * NP; ++q)
    if (!dead_half<DQ, NP>(q / 2, q % 2))
      mx = vmax(mx, vmax(vmax(s[q][0], s[q][1]), vmax(s[q][2], s[q][3])));
  mx = xmax32(xmax16(mx));
  if constexpr (FIRST) {
    st.m = mx * sc;                 // finite: every segment has a visible key
  } else {
    const float mnew = vmax(st.m, mx * sc);
    const float alpha = __builtin_amdgcn_exp2f(st.m - mnew);
    st.m = mnew;
    st.l *= alpha;
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) st.o[dt] *= alpha;
  }
  return st.m;
}
// V^T fragment (16 dims x the 32 keys of pair kp) for head dims col0 + 16 dt: one
// 16-byte read, since V^T rows keep each pair's keys in P^T fragment order.
template <int DH>
__device__ __forceinline__ void v_frags(bf16x8 (&vf)[DH / 16], const bf16_t* Vl, int vld, int col0,
                                        int kp, int lane) {
  const int gq = lane / 16, c16 = lane % 16;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt)
    vf[dt] = lfrag(Vl + (col0 + 16 * dt + c16) * vld + 32 * kp + 8 * gq);
}
// P^T fragment of pair kp (bf16 probabilities of S^T tiles 2 kp, 2 kp + 1) and its
// contribution to the tile's row sum.
template <int DH, int DQ, int NP>
__device__ __forceinline__ bf16x8 seg_probs(const f32x4v (&s)[8], int kp, float mnew,
                                            float& psum) {
  constexpr float sc = (DH == 64 ? 0.125f : 0.17677669529663688f) * 1.4426950408889634f;
  bf16x8 pb;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    if (dead_half<DQ, NP>(kp, t)) {
#pragma unroll
      for (int i = 0; i < 4; ++i) pb[4 * t + i] = static_cast<__bf16>(0.f);
      continue;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float pv = __builtin_amdgcn_exp2f(fmaf(s[2 * kp + t][i], sc, -mnew));
      psum += pv;
      pb[4 * t + i] = static_cast<__bf16>(pv);
    }
  }
  return pb;
}
// One query tile's segment: S^T, one rescale, then per pair P^T and O^T += V^T P^T,
// the next pair's V^T fragments read while this pair's probabilities are computed
// (vf is first read after the S products: read before them, its registers make the
// compiler serialize the K reads).
template <int DH, int DQ, int NP, bool FIRST>
__device__ __forceinline__ void attn_segment1(AttnState<DH>& st, const bf16_t* Kl, int kld,
                                              const bf16_t* Vl, int vld, int col0, int lane,
                                              int kvl = 0) {
  f32x4v sc[8];
  bf16x8 vf[DH / 16];
  seg_scores<DH, DQ, NP>(sc, st, Kl, kld, col0, lane, kvl);
  v_frags<DH>(vf, Vl, vld, col0, 0, lane);
  const float m = seg_rescale<DH, DQ, NP, FIRST>(st, sc);
  float ps = 0.f;
#pragma unroll
  for (int kp = 0; kp < NP; ++kp) {
    bf16x8 vn[DH / 16];
    if (kp + 1 < NP) v_frags<DH>(vn, Vl, vld, col0, kp + 1, lane);
    const bf16x8 pb = seg_probs<DH, DQ, NP>(sc, kp, m, ps);
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) st.o[dt] = mfma16(vf[dt], pb, st.o[dt]);
    if (kp + 1 < NP) {
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) vf[dt] = vn[dt];
    }
  }
  st.l += ps;
}
// The wave's two query tiles one after the other (both at once keeps twice the
// score and output registers live, which pushes the residual stream into
// accumulator registers and back around every segment; in turn each tile reads
// the segment's V^T fragments itself).
template <int DH, int DQA, int DQB, int NPA, int NPB, bool FIRST>
__device__ __forceinline__ void attn_segment2(AttnState<DH>& sa, AttnState<DH>& sb,
                                              const bf16_t* Kl, int kld, const bf16_t* Vl,
                                              int vld, int col0, int lane, int kvl = 0) {
  attn_segment1<DH, DQA, NPA, FIRST>(sa, Kl, kld, Vl, vld, col0, lane, kvl);
  attn_segment1<DH, DQB, NPB, FIRST>(sb, Kl, kld, Vl, vld, col0, lane, kvl);
}
// The block's own keys for wave W: tiles W and 7 - W see W / 2 + 1 and
// (7 - W) / 2 + 1 pairs.
template <int DH, int W>
__device__ __forceinline__ void attn_own(AttnState<DH>& sa, AttnState<DH>& sb, const bf16_t* Ks,
                                         const bf16_t* Vts, int col0, int lane) {
  attn_segment2<DH, W, 7 - W, W / 2 + 1, (7 - W) / 2 + 1, true>(sa, sb, Ks, QLD, Vts, VLD, col0,
                                                                lane);
}

// O = O^T / l into the tile's rows of Qs (the tile's Q is already in registers).
template <int DH>
__device__ __forceinline__ void attn_finish(AttnState<DH>& st, bf16_t* Qs, int col0, int qt) {
  const int lane = otid() % WAVE;
  const int gq = lane / 16, c16 = lane % 16;
  const float l = xsum32(xsum16(st.l));
  const float inv = 1.f / l;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt)
    st4(Qs + (16 * qt + c16) * QLD + col0 + 16 * dt + 4 * gq, st.o[dt][0] * inv, st.o[dt][1] * inv,
        st.o[dt][2] * inv, st.o[dt][3] * inv);
}

// Cached keys [c0, c0 + 128) of head group g (K rows and V^T columns): the loads
// into registers, and (after the work they overlap) the copy into LDS.
struct CacheChunk {
  u32x4 k[4], v[4];
};
__device__ __forceinline__ void cache_load(CacheChunk& ch, const bf16_t* kc, const bf16_t* vc,
                                           int tpad, int g, int c0) {
  const int tid = otid();
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = tid + q * NT;                      // K: 128 keys x 8 pieces
    const int r = e >> 3, c = (e & 7) * 8;
    ch.k[q] = *reinterpret_cast<const u32x4*>(kc + int64_t(c0 + r) * DM + g * 64 + c);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = tid + q * NT;                      // V^T: 64 dims x 16 pieces
    const int r = e >> 4, c = (e & 15) * 8;
    ch.v[q] = *reinterpret_cast<const u32x4*>(vc + int64_t(g * 64 + r) * tpad + c0 + c);
  }
}
// Ends with a barrier.
__device__ __forceinline__ void cache_put(const CacheChunk& ch, bf16_t* Kc, bf16_t* Vc) {
  const int tid = otid();
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = tid + q * NT;
    *reinterpret_cast<u32x4*>(Kc + (e >> 3) * QLD + (e & 7) * 8) = ch.k[q];
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = tid + q * NT;
    *reinterpret_cast<u32x4*>(Vc + (e >> 4) * VLD + (e & 15) * 8) = ch.v[q];
  }
  __syncthreads();
}

// Causal attention of the block's queries for head group g: first the block's
// own keys (Ks / Vts), then the keys of earlier blocks from the cache, whose
// first chunk (in ch, loaded by the caller ahead of the group) is staged after the
// block's own keys are processed (the softmax is independent of the key order).  prime() issues the next weight phase's
// look-ahead, after the own keys (issued earlier, its registers would be copied
// around the wave-specific code, and the copies would wait for the loads).
// NM: the unmasked mode (a single block: every query sees every valid key).
template <int DH, bool NM, class Prime>
__device__ __forceinline__ void attend_group(int g, int p0, bf16_t* Qs, const bf16_t* Ks,
                                             const bf16_t* Vts, const bf16_t* kc,
                                             const bf16_t* vc, int tpad, bf16_t* Kc, bf16_t* Vc,
                                             CacheChunk& ch, const Prime& prime, int kvl) {
  constexpr int NH = 64 / DH;
  const int lane = otid() % WAVE;
  const int w = __builtin_amdgcn_readfirstlane(otid() / WAVE);
  const int qa = w, qb = 7 - w;      // qa < qb
#pragma unroll
  for (int hd = 0; hd < NH; ++hd) {
    AttnState<DH> sa, sb;
    attn_init<DH>(sa, Qs, hd * DH, qa);
    attn_init<DH>(sb, Qs, hd * DH, qb);
    if (hd > 0 && p0 > 0) cache_load(ch, kc, vc, tpad, g, 0);   // head 0: loaded ahead
    // the block's own keys (one specialisation per wave: its pair counts)
    if constexpr (NM)
      attn_segment2<DH, -2, -2, 4, 4, true>(sa, sb, Ks, QLD, Vts, VLD, hd * DH, lane, kvl);
    else if (w == 0)
      attn_own<DH, 0>(sa, sb, Ks, Vts, hd * DH, lane);
    else if (w == 1)
      attn_own<DH, 1>(sa, sb, Ks, Vts, hd * DH, lane);
    else if (w == 2)
      attn_own<DH, 2>(sa, sb, Ks, Vts, hd * DH, lane);
    else
      attn_own<DH, 3>(sa, sb, Ks, Vts, hd * DH, lane);
    if (hd == NH - 1) prime();
    for (int c0 = 0; c0 < p0; c0 += BT) {     // earlier blocks: every key visible
      if (c0 > 0) cache_load(ch, kc, vc, tpad, g, c0);
      cache_put(ch, Kc, Vc);
      attn_segment2<DH, -1, -1, 4, 4, false>(sa, sb, Kc, QLD, Vc, VLD, hd * DH, lane);
      __syncthreads();
    }
    attn_finish<DH>(sa, Qs, hd * DH, qa);
    attn_finish<DH>(sb, Qs, hd * DH, qb);
  }
  // the next group's first cached chunk, in flight during this group's output
  // projection and the next group's Q / K / V
  if (p0 > 0 && g + 1 < DM / 64) cache_load(ch, kc, vc, tpad, g + 1, 0);
}

__device__ __forceinline__ int64_t nl_of(const Args& A, int64_t n) { return n - A.c0; }

// ---------------------------------------------------------------- block input
// Feature encoding of block rows [p0, p0 + BT) (Eq. 4 with early fusion):
// acc = X0^T = cvec + W_in[:, :d] Xs^T + E_act^T onehot(act) + E_time^T
// onehot(time) + E_pos^T onehot(position), and Xs <- bf16(X0).  cvec (the
// candidate half of the projection plus b_in) comes from cand_proj_kernel.  Rows
// past the valid length get whatever these give (token rows of zeros): no valid
// row ever reads them (causal mask, per-token sublayers, pooling over valid rows).
__device__ __forceinline__ void encode_block_input(const Args& A, int64_t n, int p0, int Tv,
                                                   f32x16 (&acc)[2][4], bf16_t* Xs,
                                                   int* tinfo, const uint8_t** rowptr, Pre& pre,
                                                   const WSeg& nxt) {
  const int d = A.d;
  {
    const int tid = otid();
    if (tid < BT) {   // resolve each row once: its embedding row and act / time
      const int p = p0 + tid;
      const uint8_t* rp = nullptr;
      int info = 0;
      if (p < Tv) {
        const TokenRef t = resolve_token(A.s, n, p, d * 2);
        rp = t.emb;
        info = t.act | (t.time << 8) | (1 << 16);
      }
      rowptr[tid] = rp;
      tinfo[tid] = info;
    }
    __syncthreads();
  }
  {
    // all of the thread's row pieces in flight at once, then into LDS
    constexpr int PER = BT * (KIN / 8) / NT;
    const int tid = otid();
    u32x4 v[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int e = tid + q * NT;
      const int r = e / (KIN / 8), c = e % (KIN / 8);
      const uint8_t* rp = rowptr[r];
      v[q] = u32x4{0u, 0u, 0u, 0u};
      if (rp && c < d / 8) v[q] = reinterpret_cast<const u32x4*>(rp)[c];
    }
    {   // accumulators <- cvec
      FZ_LANE_VARS
      const float* cv = A.cvec + nl_of(A, n) * DM;
#pragma unroll
      for (int ft = 0; ft < 2; ++ft)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float4 c4 = *reinterpret_cast<const float4*>(cv + 64 * w + ft * 32 + 8 * j + 4 * hf);
#pragma unroll
          for (int tt = 0; tt < 4; ++tt) {
            acc[ft][tt][4 * j] = c4.x;
            acc[ft][tt][4 * j + 1] = c4.y;
            acc[ft][tt][4 * j + 2] = c4.z;
            acc[ft][tt][4 * j + 3] = c4.w;
          }
        }
    }
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int e = tid + q * NT;
      const int r = e / (KIN / 8), c = e % (KIN / 8);
      *reinterpret_cast<u32x4*>(Xs + r * XLD + c * 8) = v[q];
    }
    __syncthreads();
  }
  {
    const int w = __builtin_amdgcn_readfirstlane(otid() / WAVE);
    const WSeg s_at = seg_resid(A.pk_at, AT_COLS / 16, 0, w);
    const WSeg s_pos = seg_resid(A.pk_pos, A.pos_nkb, p0 / 16, w);
    // the position rows (many weight bytes per MFMA) right after the long token
    // projection, whose iterations have time to bring their look-ahead in
    resid_phase<ShEmb, ShPos>(acc, pre, seg_resid(A.pk_in, KIN / 16, 0, w), s_pos, Xs, XLD);
    pos_phase<ShTab>(acc, pre, s_pos, s_at);
    table_phase<ShQkv>(acc, pre, s_at, nxt, tinfo);
  }
  {
    FZ_LANE_VARS
    __syncthreads();   // every wave is past Xs (tokens) and tinfo
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int ft = 0; ft < 2; ++ft)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          st4(Xs + (tt * 32 + l32) * XLD + 64 * w + ft * 32 + 8 * j + 4 * hf,
              acc[ft][tt][4 * j], acc[ft][tt][4 * j + 1], acc[ft][tt][4 * j + 2],
              acc[ft][tt][4 * j + 3]);
    __syncthreads();
  }
}

// ---------------------------------------------------------------- sublayers
// Position of key k (0..31, a multiple of 4 here) inside its 32-key pair in a V^T
// row: the order of the P^T fragment of 16x16x32 products, where lane group gq
// holds keys 4 gq .. +3 and 16 + 4 gq .. +3 as k-rows 8 gq .. +7.
__device__ __forceinline__ int vpos(int k) {
  return 8 * ((k >> 2) & 3) + 4 * (k >> 4) + (k & 3);
}

// Q / K / V of head group g: wave w computes token tiles 2(w & 1), 2(w & 1) + 1 of
// the column tiles q_d, k_d, v_d (d = w >> 1, 32 dims each) — one tile of each,
// so every wave's epilogue writes the same amount; Q and K transposed
// ([dim][token]), V untransposed.  Leaves the look-ahead empty.
__device__ __forceinline__ void qkv_phase(Pre& pre, const WSeg& cur, const WSeg& nxt,
                                          const bf16_t* Xs, bf16_t* Qs, bf16_t* Ks, bf16_t* Vts) {
  FZ_LANE_VARS
  constexpr int NKB = ShQkv::NKB;
  const int tp = w & 1, dt = w >> 1;
  f32x16 qa[3][2];
#pragma unroll
  for (int t = 0; t < 3; ++t) qa[t][0] = qa[t][1] = f32x16{};
  bf16x8 wq[NKB][3];
  bf16x8 xq[NKB][2];
  const bf16_t* arow = Xs + (tp * 64 + l32) * XLD + 8 * hf;
  xq[0][0] = lfrag(arow);
  xq[0][1] = lfrag(arow + 32 * XLD);
#pragma unroll
  for (int j = 0; j < NKB; ++j) {
    if (j + 1 < ShQkv::NX) {
      xq[j + 1][0] = lfrag(arow + (j + 1) * 16);
      xq[j + 1][1] = lfrag(arow + 32 * XLD + (j + 1) * 16);
    } else if (j + 1 < NKB) {   // the bias k-block (also as the A operand of V)
      xq[j + 1][0] = xq[j + 1][1] = bias_ones();
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {   // q_d, k_d: transposed
      const bf16x8 a = stream_frag<ShQkv>(wq, pre, j, t);
      qa[t][0] = mfma32(a, xq[j][0], qa[t][0]);
      qa[t][1] = mfma32(a, xq[j][1], qa[t][1]);
    }
    {                               // v_d: untransposed
      const bf16x8 a = stream_frag<ShQkv>(wq, pre, j, 2);
      qa[2][0] = mfma32(xq[j][0], a, qa[2][0]);
      qa[2][1] = mfma32(xq[j][1], a, qa[2][1]);
    }
    stream_fetch<ShQkv, NoPhase>(wq, pre, cur, nxt, j, lane);
    sched_fence();
  }
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int tt = 2 * tp + u;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      bf16_t* dst = t == 0 ? Qs : Ks;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        st4(dst + (tt * 32 + l32) * QLD + dt * 32 + 8 * j + 4 * hf, qa[t][u][4 * j],
            qa[t][u][4 * j + 1], qa[t][u][4 * j + 2], qa[t][u][4 * j + 3]);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
      st4(Vts + (dt * 32 + l32) * VLD + tt * 32 + vpos(8 * j + 4 * hf), qa[2][u][4 * j],
          qa[2][u][4 * j + 1], qa[2][u][4 * j + 2], qa[2][u][4 * j + 3]);
  }
}

// FFN first layer, chunk c: H^T = ReLU(W_1[chunk] Xs^T + b_1) into Hs; wave w
// computes hidden tiles 2w, 2w + 1 of the chunk for all 4 token tiles, so each
// weight fragment is loaded by one wave; the last k-block adds the biases.  ReLU
// acts on the packed bf16 pairs (for bf16 bit patterns the signed 16-bit max with
// zero is exactly ReLU, and rounding commutes with it).
typedef short s16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t relu2(uint32_t x) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(s16x2, x), s16x2{0, 0}));
}
template <class Nxt>
__device__ __forceinline__ void ffn1_phase(Pre& pre, const WSeg& cur, const WSeg& nxt,
                                           const bf16_t* Xs, bf16_t* Hs) {
  FZ_LANE_VARS
  constexpr int NKB = ShF1::NKB;
  f32x16 ha[2][4];
  bf16x8 wq[NKB][2];
  bf16x8 xq[NKB][4];
  const bf16_t* arow = Xs + l32 * XLD + 8 * hf;
#pragma unroll
  for (int tt = 0; tt < 4; ++tt) xq[0][tt] = lfrag(arow + 32 * tt * XLD);
#pragma unroll
  for (int j = 0; j < NKB; ++j) {
    if (j + 1 < ShF1::NX) {
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) xq[j + 1][tt] = lfrag(arow + 32 * tt * XLD + (j + 1) * 16);
    } else if (j + 1 < NKB) {   // the bias k-block
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) xq[j + 1][tt] = bias_ones();
    }
    {   // token tile by token tile (as in resid_phase)
      const bf16x8 a0 = stream_frag<ShF1>(wq, pre, j, 0), a1 = stream_frag<ShF1>(wq, pre, j, 1);
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        ha[0][tt] = mfma32(a0, xq[j][tt], j == 0 ? f32x16{} : ha[0][tt]);
        ha[1][tt] = mfma32(a1, xq[j][tt], j == 0 ? f32x16{} : ha[1][tt]);
      }
    }
    stream_fetch<ShF1, Nxt>(wq, pre, cur, nxt, j, lane);
    sched_fence();
  }
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int hid = (2 * w + t) * 32 + 8 * j + 4 * hf;
        *reinterpret_cast<uint2*>(Hs + (tt * 32 + l32) * HLD + hid) =
            make_uint2(relu2(pack2(ha[t][tt][4 * j], ha[t][tt][4 * j + 1])),
                       relu2(pack2(ha[t][tt][4 * j + 2], ha[t][tt][4 * j + 3])));
      }
}

// This block's K and V^T of head group g into the candidate's cache (read by the
// candidate's later blocks), carried along by the output projection: piece q
// (one 16-byte chunk of K and one of V^T per thread) is read from LDS at k-block
// q and stored at k-block q + 1.  Buffer stores whose range is empty when the
// block keeps nothing, so the phase has no branch.
struct CacheStore {
  __amdgpu_buffer_rsrc_t rk, rv;
  const bf16_t* ks;   // this thread's piece 0 in Ks / Vts
  const bf16_t* vs;
  int ko, vo;         // its byte offsets in the cache slices
  int vstep;          // bytes between V^T pieces (16 rows of the cache)
  u32x4 k, v;         // the piece in flight
  __device__ __forceinline__ void read(int q) {
    k = *reinterpret_cast<const u32x4*>(ks + q * 32 * QLD);
    v = *reinterpret_cast<const u32x4*>(vs + q * 16 * VLD);
  }
  __device__ __forceinline__ void write(int q) {
    __builtin_amdgcn_raw_buffer_store_b128(k, rk, ko, q * 32 * DM * 2, 0);
    __builtin_amdgcn_raw_buffer_store_b128(v, rv, vo, q * vstep, 0);
  }
  __device__ __forceinline__ void step(int j) {
    if (j >= 1 && j <= 4) write(j - 1);
    if (j <= 3) read(j);
  }
  __device__ __forceinline__ void finish() {}
};
template <int NKB>
struct CacheStoreTail : CacheStore {   // a phase of 4 k-blocks stores the last piece after it
  __device__ __forceinline__ void finish() {
    if constexpr (NKB == 4) write(3);
  }
};
template <int NKB>
__device__ __forceinline__ CacheStoreTail<NKB> cache_store(const Args& A, int g, int p0,
                                                           const bf16_t* Ks, const bf16_t* Vts,
                                                           bf16_t* kc, bf16_t* vc, bool keep) {
  static_assert(NKB == 4 || NKB == 5, "four pieces over the output projection's k-blocks");
  const int tid = otid();
  // (offsets in 32 bits: one candidate's cache holds at most DM x 1024 positions)
  const int bytes = keep ? A.tpad * DM * 2 : 0;
  CacheStoreTail<NKB> c;
  c.rk = __builtin_amdgcn_make_buffer_rsrc(kc, (short)0, bytes, 0x00020000);
  c.rv = __builtin_amdgcn_make_buffer_rsrc(vc, (short)0, bytes, 0x00020000);
  c.ks = Ks + (tid >> 3) * QLD + (tid & 7) * 8;
  c.vs = Vts + (tid >> 4) * VLD + (tid & 15) * 8;
  c.ko = ((p0 + (tid >> 3)) * DM + g * 64 + (tid & 7) * 8) * 2;
  c.vo = ((g * 64 + (tid >> 4)) * A.tpad + p0 + (tid & 15) * 8) * 2;
  c.vstep = 16 * A.tpad * 2;
  return c;
}

// Attention sublayer of one layer for the block: per 64-dim head group, Q / K /
// V^T into LDS (and K / V^T into the cache for later blocks), causal attention
// per head, and acc += O_g W_o[:, group]^T.  The stream leaves primed with the
// first FFN chunk of the layer.  NM: unmasked (keys at or past kvl are padding).
template <bool LAST, bool NM>
__device__ __forceinline__ void attention_group(const Args& A, const tav2_layer& L,
                                                const LayerPk& pk, f32x16 (&acc)[2][4], Pre& pre,
                                                bf16_t* Xs, bf16_t* Qs, bf16_t* Ks, bf16_t* Vts,
                                                bf16_t* Kc, bf16_t* Vc, bf16_t* kc, bf16_t* vc,
                                                int p0, bool keep, int g, CacheChunk& ch, int kvl) {
  const int w = __builtin_amdgcn_readfirstlane(otid() / WAVE);
  // (the last group's output projection also adds b_o: its bias k-block follows
  // the group's 4 k-blocks)
  using Wo = typename std::conditional<LAST, ShWoL, ShWo>::type;
  const WSeg so = seg_resid(pk.o, NKB_W, 4 * g, w);
  qkv_phase(pre, seg_qkv(pk.qkv, g, w), so, Xs, Qs, Ks, Vts);
  __syncthreads();
  // the output projection's look-ahead is loaded during the attention
  const auto prime = [&] { seg_prime<Wo>(pre, so, otid() % WAVE); };
  if (A.dh == 64)
    attend_group<64, NM>(g, p0, Qs, Ks, Vts, kc, vc, A.tpad, Kc, Vc, ch, prime, kvl);
  else
    attend_group<32, NM>(g, p0, Qs, Ks, Vts, kc, vc, A.tpad, Kc, Vc, ch, prime, kvl);
  __syncthreads();
  // the output projection carries the cache stores (after its first k-block's
  // weight loads, so the next phase's first wait on its weights does not also wait
  // for a store)
  if constexpr (!LAST) {
    resid_phase<ShWo, ShQkv>(acc, pre, so, seg_qkv(pk.qkv, g + 1, w), Qs, QLD,
                             cache_store<ShWo::NKB>(A, g, p0, Ks, Vts, kc, vc, keep));
  } else {   // the staging area is free now: it receives the LayerNorm parameters
    const LnParams q = ln_params_load(L.ln1_g, L.ln1_b);
    resid_phase<ShWoL, ShF1>(acc, pre, so, seg_ffn1(pk.w1, 0, w), Qs, QLD,
                             cache_store<ShWoL::NKB>(A, g, p0, Ks, Vts, kc, vc, keep));
    ln_params_store(q, reinterpret_cast<float*>(Kc));
  }
  __syncthreads();   // Qs (O) and Ks / Vts are rewritten by the next group
}
// The last head group is peeled out of the loop: the code after it (LayerNorm)
// then sees exactly which weight loads are still in flight.
template <bool NM>
__device__ __forceinline__ void attention_sublayer(const Args& A, const tav2_layer& L,
                                                   const LayerPk& pk, f32x16 (&acc)[2][4],
                                                   Pre& pre, bf16_t* Xs,
                                                   bf16_t* Qs, bf16_t* Ks, bf16_t* Vts, bf16_t* Kc,
                                                   bf16_t* Vc, bf16_t* kc, bf16_t* vc, int p0,
                                                   bool keep, int kvl) {
  CacheChunk ch;   // first cached chunk of the group about to attend
  if (p0 > 0) cache_load(ch, kc, vc, A.tpad, 0, 0);
  for (int g = 0; g + 1 < DM / 64; ++g)
    attention_group<false, NM>(A, L, pk, acc, pre, Xs, Qs, Ks, Vts, Kc, Vc, kc, vc, p0, keep, g,
                               ch, kvl);
  attention_group<true, NM>(A, L, pk, acc, pre, Xs, Qs, Ks, Vts, Kc, Vc, kc, vc, p0, keep,
                            DM / 64 - 1, ch, kvl);
}

// FFN sublayer: per chunk of FC hidden units, H^T into LDS, then
// acc += W_2[:, chunk] H^T (the last chunk also adds b_2).  The stream enters
// primed with chunk 0 and leaves primed with `after`: the next layer's first
// Q / K / V phase, or (last layer) the pooling projection (shape After).  The
// last chunk is peeled out of the loop (see attention_sublayer).
template <bool LAST, class After>
__device__ __forceinline__ void ffn_chunk(const Args& A, const tav2_layer& L, const LayerPk& pk,
                                          f32x16 (&acc)[2][4], Pre& pre, const WSeg& after,
                                          const bf16_t* Xs, bf16_t* Hs, int c) {
  using F2 = typename std::conditional<LAST, ShF2L, ShF2>::type;
  const int w = __builtin_amdgcn_readfirstlane(otid() / WAVE);
  const WSeg s2 = seg_resid(pk.w2, A.ffn / 16 + 1, c * (FC / 16), w);
  // last chunk: the LayerNorm parameters are loaded ahead of the first layer's
  // weight loads and go past the hidden chunk before the second layer
  LnParams q;
  if constexpr (LAST) q = ln_params_load(L.ln2_g, L.ln2_b);
  ffn1_phase<F2>(pre, seg_ffn1(pk.w1, c, w), s2, Xs, Hs);
  if constexpr (LAST)
    ln_params_store(q, reinterpret_cast<float*>(reinterpret_cast<uint8_t*>(Hs) + BT * HLD * 2));
  __syncthreads();
  if constexpr (!LAST)
    resid_phase<F2, ShF1>(acc, pre, s2, seg_ffn1(pk.w1, c + 1, w), Hs, HLD);
  else
    resid_phase<F2, After>(acc, pre, s2, after, Hs, HLD);
  __syncthreads();   // Hs is rewritten by the next chunk
}
template <class After>
__device__ __forceinline__ void ffn_sublayer(const Args& A, const tav2_layer& L,
                                             const LayerPk& pk, f32x16 (&acc)[2][4], Pre& pre,
                                             const WSeg& after, bf16_t* Xs, bf16_t* Hs) {
  const int nch = A.ffn / FC;
  for (int c = 0; c + 1 < nch; ++c)
    ffn_chunk<false, After>(A, L, pk, acc, pre, after, Xs, Hs, c);
  ffn_chunk<true, After>(A, L, pk, acc, pre, after, Xs, Hs, nch - 1);
}

// One encoder layer of the block: attention, LayerNorm 1, FFN, LayerNorm 2.  The
// last layer is a separate instance (its FFN leaves the stream primed with the
// pooling projection instead of the next layer's Q / K / V), so that no code
// joins two different look-ahead states.
template <bool LASTL, bool NM>
__device__ __forceinline__ void encoder_layer(const Args& A, int li, f32x16 (&acc)[2][4],
                                              Pre& pre, uint8_t* smem, int64_t nl, int p0,
                                              bool keep, int kvl) {
  const Args* AK = (const Args*)(__builtin_amdgcn_kernarg_segment_ptr());
  const int w = __builtin_amdgcn_readfirstlane(otid() / WAVE);
  bf16_t* Xs = reinterpret_cast<bf16_t*>(smem);
  uint8_t* Sc = smem + XS_BYTES;
  bf16_t* Kc = reinterpret_cast<bf16_t*>(smem + XS_BYTES + SC_BYTES);
  bf16_t* Vc = reinterpret_cast<bf16_t*>(smem + XS_BYTES + SC_BYTES + QS_BYTES);
  bf16_t* Qs = reinterpret_cast<bf16_t*>(Sc);                    // [BT][QLD], then O
  bf16_t* Ks = reinterpret_cast<bf16_t*>(Sc + QS_BYTES);         // [BT][QLD]
  bf16_t* Vts = reinterpret_cast<bf16_t*>(Sc + 2 * QS_BYTES);    // [64][VLD]
  bf16_t* Hs = reinterpret_cast<bf16_t*>(Sc);                    // [BT][HLD]
  float* red = reinterpret_cast<float*>(Sc);                     // reductions
  float* lnp1 = reinterpret_cast<float*>(Kc);                    // LayerNorm 1 parameters
  float* lnp2 = reinterpret_cast<float*>(Sc + BT * HLD * 2);     // LayerNorm 2 parameters
  // layer records are read through the kernel-argument segment so the runtime
  // layer index stays a scalar load instead of a private copy of the array
  const tav2_layer L = AK->layers[li];
  const LayerPk pk = AK->pk[li];
  bf16_t* kc = A.kcache ? A.kcache + (nl * A.n_layers + li) * int64_t(A.tpad) * DM : nullptr;
  bf16_t* vc = A.vcache ? A.vcache + (nl * A.n_layers + li) * int64_t(DM) * A.tpad : nullptr;
  attention_sublayer<NM>(A, L, pk, acc, pre, Xs, Qs, Ks, Vts, Kc, Vc, kc, vc, p0, keep, kvl);
  layer_norm(acc, lnp1, red, Xs);
  if constexpr (LASTL)
    ffn_sublayer<ShPool>(A, L, pk, acc, pre, seg_resid(A.pk_pool, DM / 16, 0, w), Xs, Hs);
  else
    ffn_sublayer<ShQkv>(A, L, pk, acc, pre, seg_qkv(AK->pk[li + 1].qkv, 0, w), Xs, Hs);
  layer_norm(acc, lnp2, red, Xs);
}

// ---------------------------------------------------------------- the kernel
// NM: the unmasked mode (every valid position sees every valid position; the
// host allows it only when T fits one 128-position block).
template <bool NM>
__global__ __launch_bounds__(NT) void encoder_fused_kernel(Args A) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[LDS_BYTES];
  bf16_t* Xs = reinterpret_cast<bf16_t*>(smem);
  uint8_t* Sc = smem + XS_BYTES;
  int* tinfo = reinterpret_cast<int*>(Sc);                       // [BT] during encoding
  const uint8_t** rowptr = reinterpret_cast<const uint8_t**>(Sc + BT * 8);   // [BT]

  const int64_t nl = blockIdx.x;
  const int64_t n = A.c0 + nl;
  const int Tv = token_valid_len(A.s, n);
  float* out = A.out + n * 2 * DM;
  if (Tv == 0) {
    for (int c = threadIdx.x; c < 2 * DM; c += NT) out[c] = 0.f;
    return;
  }
  const int nblk = (Tv + BT - 1) / BT;
  const Args* AK = (const Args*)(__builtin_amdgcn_kernarg_segment_ptr());
  const int wv = __builtin_amdgcn_readfirstlane(otid() / WAVE);
  const WSeg s_embed = seg_resid(A.pk_in, KIN / 16, 0, wv);
  const WSeg s_pool = seg_resid(A.pk_pool, DM / 16, 0, wv);
  Pre pre;
  seg_prime<ShEmb>(pre, s_embed, otid() % WAVE);
  f32x16 acc[2][4];
  float pm = -__builtin_inff();   // running pooled max of feature pool_feature()
  for (int blk = 0; blk < nblk; ++blk) {
    const int p0 = blk * BT;
    __syncthreads();
    encode_block_input(A, n, p0, Tv, acc, Xs, tinfo, rowptr, pre,
                       seg_qkv(AK->pk[0].qkv, 0, wv));
    for (int li = 0; li + 1 < A.n_layers; ++li)
      encoder_layer<false, NM>(A, li, acc, pre, smem, nl, p0, blk + 1 < nblk, Tv - p0);
    encoder_layer<true, NM>(A, A.n_layers - 1, acc, pre, smem, nl, p0, blk + 1 < nblk, Tv - p0);
    // ---- head: out[DM:] = X of the last valid token; running max of the pool
    {
      FZ_LANE_VARS
      const int last = Tv - 1 - p0;
      if (last >= 0 && last < BT) {
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
          if (tt * 32 + l32 == last) {
#pragma unroll
            for (int ft = 0; ft < 2; ++ft)
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                const int f = 64 * w + ft * 32 + 8 * j + 4 * hf;
                *reinterpret_cast<float4*>(out + DM + f) =
                    make_float4(acc[ft][tt][4 * j], acc[ft][tt][4 * j + 1],
                                acc[ft][tt][4 * j + 2], acc[ft][tt][4 * j + 3]);
              }
          }
      }
    }
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = f32x16{};
    // the pool phase prefetches the next block's input projection (also after the
    // last block, where the loads are simply unused)
    resid_phase<ShPool, ShEmb>(acc, pre, s_pool, s_embed, Xs, XLD);
    pm = pool_block(acc, pm, Tv - p0);
  }
  {
    const int f = pool_feature();
    out[f] = pm + A.b_pool[f];
  }
}

}  // namespace fz

// Launch of the unmasked instantiation (encoder_fused_unmasked.hip: a translation
// unit of its own, so that the causal kernel's code is generated as if it were
// the only instantiation).
hipError_t launch_encoder_fused_unmasked(const fz::Args& a, unsigned grid, hipStream_t st);

}  // namespace tav2
