// Fused bf16 encoder: one workgroup runs one candidate through feature encoding
// (Eq. 4, early fusion), every causal post-LN layer and the linear + max-pool head
// (Sec. 3.2.2) without writing activations to HBM.
//
// Layout of the work:
//  * The candidate's positions are processed in blocks of 128 tokens.  Under the
//    causal mask a block depends on earlier blocks only through their keys and
//    values, so each block runs through all layers in turn and leaves its K/V in a
//    per-candidate cache (workspace) for the blocks after it.
//  * 8 waves.  The fp32 residual stream of the block lives in registers as the
//    transposed product X^T [feature x token] (MFMA accumulator layout: one token
//    per lane, 4 consecutive features per register group), so LayerNorm over
//    features is an in-lane sum, one cross-half exchange and a 4-way exchange
//    between waves through LDS.
//  * The bf16 copy of the block's activations (MFMA operand), the per-head-group
//    Q / K / V^T, the attention output and the FFN hidden chunk live in LDS; weight
//    tiles [rows x 32] stream from L2 through a double-buffered LDS stage with a
//    register prefetch two steps ahead.
//  * Every LDS write of an activation is 4 consecutive bf16 of one row (8 bytes):
//    products whose consumer needs [token][feature] are computed transposed
//    (weights as MFMA A operand); V is computed untransposed to give V^T [dim][token].
//  * Attention: 16x16x32 MFMAs, wave w owns queries 16w .. 16w+15 of the block;
//    S^T = K Q^T puts one query per lane column, and P^T goes back into
//    O^T = V^T P^T from its accumulator registers with the matching key order.
#include "common.h"
#include "internal.h"
#include "token_source.h"

namespace tav2 {
namespace fz {

constexpr int DM = 256;          // d_model
constexpr int BT = 128;          // tokens per block
constexpr int NT = 512;          // threads (8 waves)
constexpr int KS = 32;           // k extent of one weight stage
constexpr int XLD = DM + 8;      // Xs row stride (bf16 elements)
constexpr int WLD = KS + 8;      // weight stage row stride
constexpr int WROWS = 256;       // rows per weight stage
constexpr int QLD = 64 + 8;      // Qs / Ks / Os row stride (one 64-dim head group)
constexpr int VLD = BT + 8;      // Vts row stride
constexpr int FC = 128;          // FFN hidden units per chunk
constexpr int HLD = FC + 8;      // Hs row stride
constexpr int MAX_LAYERS = 8;

constexpr int XS_BYTES = BT * XLD * 2;                 // 67584
constexpr int WS_BYTES = 2 * WROWS * WLD * 2;          // 40960
constexpr int QS_BYTES = BT * QLD * 2;                 // 18432
constexpr int VS_BYTES = 64 * VLD * 2;                 // 17408
constexpr int SC_BYTES = 2 * QS_BYTES + VS_BYTES;      // 54272
constexpr int PM_BYTES = DM * 4;                       // running pooled max
constexpr int LDS_BYTES = XS_BYTES + WS_BYTES + SC_BYTES + PM_BYTES;
static_assert(LDS_BYTES <= 163840, "fused encoder exceeds the 160 KiB of LDS");
static_assert(BT * HLD * 2 <= SC_BYTES, "FFN chunk does not fit the scratch region");
static_assert(2 * BT * 4 * 4 + 2 * DM * 4 <= SC_BYTES, "reduction buffers do not fit");

typedef float f32x4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4v mfma16(const bf16x8& a, const bf16x8& b, const f32x4v& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// The thread index through an empty asm: index and address arithmetic derived from
// it is recomputed inside each phase instead of being hoisted out of the block and
// layer loops (which would keep it live, and spilled, across the whole kernel).
__device__ __forceinline__ int otid() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

// Per-phase lane coordinates: lane, wave (uniform), half, column-in-half, and the
// residual tile coordinates fq (feature quarter) and th (token half).
#define FZ_LANE_VARS                                                      \
  const int tid_ = otid();                                                \
  const int lane = tid_ % WAVE;                                           \
  const int w = __builtin_amdgcn_readfirstlane(tid_ / WAVE);              \
  const int hf = lane / 32, l32 = lane % 32;                              \
  const int fq = w & 3, th = w >> 2;                                      \
  (void)hf; (void)l32; (void)fq; (void)th;

__device__ __forceinline__ bf16x8 frag(const bf16_t* p) {
  return as_bf16x8(*reinterpret_cast<const uint4*>(p));
}
__device__ __forceinline__ void st4(bf16_t* p, float a, float b, float c, float d) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack2(a, b), pack2(c, d));
}

struct Args {
  TokenSource s;
  const bf16_t* cand;       // [total, d]
  const bf16_t* W_in;       // [DM, 2d]
  const float* b_in;
  const bf16_t* E_act;
  const bf16_t* E_time;     // may be null
  const bf16_t* E_pos;
  const bf16_t* W_pool;
  const float* b_pool;
  tav2_layer layers[MAX_LAYERS];
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

// ---------------------------------------------------------------- weight staging
// A [R x 32] bf16 tile moves as 16-byte items, 4 per row; thread t owns items t
// and t + NT.  Items travel in native vector registers (no arrays, no references)
// so they stay in VGPRs while the loads are in flight.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

#define FZ_WLOAD(RA, RB, ROWS, R, K0)                                                   \
  do {                                                                                  \
    if (wt_ < (R) * 4)                                                                  \
      RA = *reinterpret_cast<const u32x4*>(ROWS(wt_ >> 2) + (K0) + (wt_ & 3) * 8);      \
    if (wt_ + NT < (R) * 4)                                                             \
      RB = *reinterpret_cast<const u32x4*>(ROWS((wt_ + NT) >> 2) + (K0) + (wt_ & 3) * 8); \
  } while (0)

#define FZ_WSTORE(RA, RB, BUF, R)                                                       \
  do {                                                                                  \
    if (wt_ < (R) * 4)                                                                  \
      *reinterpret_cast<u32x4*>(Ws + ((BUF) * WROWS + (wt_ >> 2)) * WLD + (wt_ & 3) * 8) = RA; \
    if (wt_ + NT < (R) * 4)                                                             \
      *reinterpret_cast<u32x4*>(Ws + ((BUF) * WROWS + ((wt_ + NT) >> 2)) * WLD + (wt_ & 3) * 8) = RB; \
  } while (0)

// Streams R weight rows x K columns through the two LDS stages.  BODY runs once
// per 32-wide k step with `stage` (the resident [R x 32] tile) and `k0` defined.
// The register prefetch runs two steps ahead; the loop is unrolled by two so the
// two register sets alternate without copies.  Ends with a barrier.
#define FZ_STREAM(ROWS, R, K, BODY)                                             \
  do {                                                                          \
    const int nks_ = (K) / KS;                                                  \
    const int wt_ = otid();                                                     \
    u32x4 r0a_ = {}, r0b_ = {}, r1a_ = {}, r1b_ = {};                           \
    FZ_WLOAD(r1a_, r1b_, ROWS, R, 0);                                           \
    if (nks_ > 1) FZ_WLOAD(r0a_, r0b_, ROWS, R, KS);                            \
    FZ_WSTORE(r1a_, r1b_, 0, R);                                                \
    __syncthreads();                                                            \
    for (int ks_ = 0; ks_ < nks_; ks_ += 2) {                                   \
      if (ks_ + 2 < nks_) FZ_WLOAD(r1a_, r1b_, ROWS, R, (ks_ + 2) * KS);        \
      {                                                                         \
        const bf16_t* stage = Ws + (ks_ & 1) * WROWS * WLD;                     \
        const int k0 = ks_ * KS;                                                \
        BODY                                                                    \
      }                                                                         \
      if (ks_ + 1 < nks_) FZ_WSTORE(r0a_, r0b_, (ks_ + 1) & 1, R);              \
      __syncthreads();                                                          \
      if (ks_ + 1 >= nks_) break;                                               \
      if (ks_ + 3 < nks_) FZ_WLOAD(r0a_, r0b_, ROWS, R, (ks_ + 3) * KS);        \
      {                                                                         \
        const bf16_t* stage = Ws + ((ks_ + 1) & 1) * WROWS * WLD;               \
        const int k0 = (ks_ + 1) * KS;                                          \
        BODY                                                                    \
      }                                                                         \
      if (ks_ + 2 < nks_) FZ_WSTORE(r1a_, r1b_, (ks_ + 2) & 1, R);              \
      __syncthreads();                                                          \
    }                                                                           \
  } while (0)

// C^T[256 feature x 128 token] += W[256 x K] . ACT[128 x K]^T; wave tile
// 64 features (fq) x 64 tokens (th) as acc[feature tile][token tile].
#define FZ_RESID_BODY(ACT, ALD)                                                          \
  _Pragma("unroll") for (int kb = 0; kb < KS / 16; ++kb) {                                \
    bf16x8 wa_[2], xb_[2];                                                                \
    _Pragma("unroll") for (int t = 0; t < 2; ++t) {                                       \
      wa_[t] = frag(stage + (fq * 64 + t * 32 + l32) * WLD + kb * 16 + 8 * hf);           \
      xb_[t] = frag((ACT) + (th * 64 + t * 32 + l32) * (ALD) + k0 + kb * 16 + 8 * hf);    \
    }                                                                                     \
    _Pragma("unroll") for (int a = 0; a < 2; ++a)                                         \
      _Pragma("unroll") for (int b = 0; b < 2; ++b) acc[a][b] = mfma32(wa_[a], xb_[b], acc[a][b]); \
  }

// ---------------------------------------------------------------- LayerNorm
// acc holds C^T (features x tokens) of the block without the sublayer bias.
// x <- LN(acc + bias) with gain g and offset b; Xs <- bf16(x).  Ends with a barrier.
__device__ __forceinline__ void layer_norm(f32x16 (&acc)[2][2], const float* bias,
                                           const float* g, const float* b, float* red,
                                           bf16_t* Xs) {
  FZ_LANE_VARS
  float s[2] = {0.f, 0.f}, ss[2] = {0.f, 0.f};
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int ft = 0; ft < 2; ++ft)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 bi = *reinterpret_cast<const float4*>(bias + fq * 64 + ft * 32 + 8 * j + 4 * hf);
        const float v0 = acc[ft][tt][4 * j] + bi.x;
        const float v1 = acc[ft][tt][4 * j + 1] + bi.y;
        const float v2 = acc[ft][tt][4 * j + 2] + bi.z;
        const float v3 = acc[ft][tt][4 * j + 3] + bi.w;
        acc[ft][tt][4 * j] = v0;
        acc[ft][tt][4 * j + 1] = v1;
        acc[ft][tt][4 * j + 2] = v2;
        acc[ft][tt][4 * j + 3] = v3;
        s[tt] += (v0 + v1) + (v2 + v3);
        ss[tt] += (v0 * v0 + v1 * v1) + (v2 * v2 + v3 * v3);
      }
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    s[tt] += __shfl_xor(s[tt], 32, WAVE);
    ss[tt] += __shfl_xor(ss[tt], 32, WAVE);
  }
  // red[tok][fq] = (sum, sumsq) over this wave's 64 features
  if (hf == 0) {
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const int tok = th * 64 + tt * 32 + l32;
      red[(tok * 4 + fq) * 2] = s[tt];
      red[(tok * 4 + fq) * 2 + 1] = ss[tt];
    }
  }
  __syncthreads();
  float mean[2], rstd[2];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    const int tok = th * 64 + tt * 32 + l32;
    const float4 a = *reinterpret_cast<const float4*>(red + tok * 8);
    const float4 c = *reinterpret_cast<const float4*>(red + tok * 8 + 4);
    const float sum = (a.x + a.z) + (c.x + c.z);
    const float sq = (a.y + a.w) + (c.y + c.w);
    mean[tt] = sum * (1.f / DM);
    const float var = fmaxf(sq * (1.f / DM) - mean[tt] * mean[tt], 0.f);
    rstd[tt] = rsqrtf(var + 1e-5f);
  }
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int ft = 0; ft < 2; ++ft)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int f = fq * 64 + ft * 32 + 8 * j + 4 * hf;
        const float4 gg = *reinterpret_cast<const float4*>(g + f);
        const float4 bb = *reinterpret_cast<const float4*>(b + f);
        const float v0 = (acc[ft][tt][4 * j] - mean[tt]) * rstd[tt] * gg.x + bb.x;
        const float v1 = (acc[ft][tt][4 * j + 1] - mean[tt]) * rstd[tt] * gg.y + bb.y;
        const float v2 = (acc[ft][tt][4 * j + 2] - mean[tt]) * rstd[tt] * gg.z + bb.z;
        const float v3 = (acc[ft][tt][4 * j + 3] - mean[tt]) * rstd[tt] * gg.w + bb.w;
        acc[ft][tt][4 * j] = v0;
        acc[ft][tt][4 * j + 1] = v1;
        acc[ft][tt][4 * j + 2] = v2;
        acc[ft][tt][4 * j + 3] = v3;
        st4(Xs + (th * 64 + tt * 32 + l32) * XLD + fq * 64 + ft * 32 + 8 * j + 4 * hf, v0, v1, v2,
            v3);
      }
  __syncthreads();
}

// ---------------------------------------------------------------- pooling
// Max over the block's valid tokens (token < nvalid) of Y^T = acc + b_pool, folded
// into pmax.  The 32 per-lane features are max-reduced across the 32 lanes of a
// half with a transposing butterfly, so lane l32 ends with feature index
// bitrev5(l32) of its half.  Ends with a barrier.
#define FZ_TMAX(HALF, MASK)                                                   \
  _Pragma("unroll") for (int k = 0; k < (HALF); ++k) {                        \
    const bool up = (l32 & (MASK)) != 0;                                      \
    const float keep = up ? v[k + (HALF)] : v[k];                             \
    const float send = up ? v[k] : v[k + (HALF)];                             \
    v[k] = fmaxf(keep, __shfl_xor(send, (MASK), WAVE));                       \
  }

__device__ __forceinline__ void pool_block(f32x16 (&acc)[2][2], const float* b_pool, float* pmax,
                                           float* red, int nvalid) {
  FZ_LANE_VARS
  float v[32];
#pragma unroll
  for (int ft = 0; ft < 2; ++ft)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float m = -__builtin_inff();
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
        if (th * 64 + tt * 32 + l32 < nvalid) m = fmaxf(m, acc[ft][tt][r]);
      v[ft * 16 + r] = m;
    }
  FZ_TMAX(16, 1)
  FZ_TMAX(8, 2)
  FZ_TMAX(4, 4)
  FZ_TMAX(2, 8)
  FZ_TMAX(1, 16)
  const int k = ((l32 & 1) << 4) | ((l32 & 2) << 2) | (l32 & 4) | ((l32 & 8) >> 2) | ((l32 & 16) >> 4);
  const int f = fq * 64 + (k >> 4) * 32 + 8 * ((k & 15) >> 2) + 4 * hf + (k & 3);
  red[th * DM + f] = v[0] + b_pool[f];
  __syncthreads();
  if (tid_ < DM) {
    const int c = tid_;
    pmax[c] = fmaxf(pmax[c], fmaxf(red[c], red[DM + c]));
  }
  __syncthreads();
}

// ---------------------------------------------------------------- attention
// Causal attention of one head (columns col0 .. col0 + DH of the 64-dim group)
// for the block's 128 queries; wave w owns queries 16w .. 16w+15.  Keys before
// the block come from the cache, keys of the block from Ks / Vts.  The output
// overwrites the wave's own rows of Qs (already read into registers).
template <int DH>
__device__ __forceinline__ void attend_head(int g, int col0, int p0, bf16_t* Qs, const bf16_t* Ks,
                                            const bf16_t* Vts, const bf16_t* kc,
                                            const bf16_t* vc, int tpad) {
  FZ_LANE_VARS
  const int gq = lane / 16, c16 = lane % 16;
  const int qrow = 16 * w + c16;
  bf16x8 qf[DH / 32];
#pragma unroll
  for (int kb = 0; kb < DH / 32; ++kb) qf[kb] = frag(Qs + qrow * QLD + col0 + 32 * kb + 8 * gq);
  f32x4v o[DH / 16];
#pragma unroll
  for (int t = 0; t < DH / 16; ++t) o[t] = f32x4v{0.f, 0.f, 0.f, 0.f};
  float mrun = -__builtin_inff(), lrun = 0.f;
  const float sc = rsqrtf(float(DH)) * 1.4426950408889634f;

  // keys cached from earlier blocks: all visible
  for (int k0 = 0; k0 < p0; k0 += 32) {
    f32x4v s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      s[t] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < DH / 32; ++kb) {
        const bf16x8 kf = frag(kc + int64_t(k0 + 16 * t + c16) * DM + g * 64 + col0 + 32 * kb + 8 * gq);
        s[t] = mfma16(kf, qf[kb], s[t]);
      }
    }
    float mx = -__builtin_inff();
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s[t][i] *= sc;
        mx = fmaxf(mx, s[t][i]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, WAVE));
    mx = fmaxf(mx, __shfl_xor(mx, 32, WAVE));
    const float mnew = fmaxf(mrun, mx);
    const float alpha = exp2f(mrun - mnew);
    bf16x8 pb;
    float psum = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = exp2f(s[t][i] - mnew);
        psum += p;
        pb[4 * t + i] = static_cast<__bf16>(p);
      }
    lrun = lrun * alpha + psum;
    mrun = mnew;
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) {
      o[dt] *= alpha;
      const bf16_t* vr = vc + int64_t(g * 64 + col0 + 16 * dt + c16) * tpad + k0 + 4 * gq;
      const uint2 lo = *reinterpret_cast<const uint2*>(vr);
      const uint2 hi = *reinterpret_cast<const uint2*>(vr + 16);
      o[dt] = mfma16(as_bf16x8(lo, hi), pb, o[dt]);
    }
  }
  // keys of this block up to the wave's last query, causal mask inside
  const int kend = 16 * w + 16;
  for (int k0 = 0; k0 < kend; k0 += 32) {
    f32x4v s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      s[t] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < DH / 32; ++kb) {
        const bf16x8 kf = frag(Ks + (k0 + 16 * t + c16) * QLD + col0 + 32 * kb + 8 * gq);
        s[t] = mfma16(kf, qf[kb], s[t]);
      }
    }
    float mx = -__builtin_inff();
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = k0 + 16 * t + 4 * gq + i;
        s[t][i] = key > qrow ? -__builtin_inff() : s[t][i] * sc;
        mx = fmaxf(mx, s[t][i]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, WAVE));
    mx = fmaxf(mx, __shfl_xor(mx, 32, WAVE));
    const float mnew = fmaxf(mrun, mx);
    const float alpha = exp2f(mrun - mnew);
    bf16x8 pb;
    float psum = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = exp2f(s[t][i] - mnew);
        psum += p;
        pb[4 * t + i] = static_cast<__bf16>(p);
      }
    lrun = lrun * alpha + psum;
    mrun = mnew;
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) {
      o[dt] *= alpha;
      const bf16_t* vr = Vts + (col0 + 16 * dt + c16) * VLD + k0 + 4 * gq;
      const uint2 lo = *reinterpret_cast<const uint2*>(vr);
      const uint2 hi = *reinterpret_cast<const uint2*>(vr + 16);
      o[dt] = mfma16(as_bf16x8(lo, hi), pb, o[dt]);
    }
  }
  float l = lrun + __shfl_xor(lrun, 16, WAVE);
  l += __shfl_xor(l, 32, WAVE);
  const float inv = 1.f / l;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt)
    st4(Qs + qrow * QLD + col0 + 16 * dt + 4 * gq, o[dt][0] * inv, o[dt][1] * inv, o[dt][2] * inv,
        o[dt][3] * inv);
}

// ---------------------------------------------------------------- the kernel
// Feature encoding of block rows [p0, p0 + BT): token rows into Xs, then
// acc = X0^T = W_in[:, :d] Xs^T + c W_in[:, d:]^T + b_in + E_act + E_time + E_pos
// (zero for positions past the valid length), and Xs <- bf16(X0).
__device__ __forceinline__ void encode_block_input(const Args& A, int64_t n, int p0, int Tv,
                                                   f32x16 (&acc)[2][2], bf16_t* Xs, bf16_t* Ws,
                                                   float* cvec, int* tinfo) {
  const int d = A.d;
  {
    const int tid = otid();
    for (int e = tid; e < BT * (d / 8); e += NT) {
      const int r = e / (d / 8), c = e % (d / 8);
      const int p = p0 + r;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (p < Tv) {
        const TokenRef t = resolve_token(A.s, n, p, d * 2);
        if (t.emb) v = reinterpret_cast<const uint4*>(t.emb)[c];
        if (c == 0) tinfo[r] = t.act | (t.time << 8) | (1 << 16);
      } else if (c == 0) {
        tinfo[r] = 0;
      }
      *reinterpret_cast<uint4*>(Xs + r * XLD + c * 8) = v;
    }
    if (tid < DM) {   // candidate half of the input projection: c W_in[:, d:]^T + b_in
      const bf16_t* wr = A.W_in + int64_t(tid) * 2 * d + d;
      const bf16_t* cr = A.cand + n * d;
      float s = A.b_in[tid];
      for (int j = 0; j < d; j += 8) {
        const uint4 wv = *reinterpret_cast<const uint4*>(wr + j);
        const uint4 cv = *reinterpret_cast<const uint4*>(cr + j);
        const bf16_t* wp = reinterpret_cast<const bf16_t*>(&wv);
        const bf16_t* cp = reinterpret_cast<const bf16_t*>(&cv);
#pragma unroll
        for (int u = 0; u < 8; ++u) s = fmaf(bf2f(wp[u]), bf2f(cp[u]), s);
      }
      cvec[tid] = s;
    }
  }
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};
  {
    FZ_LANE_VARS
    const bf16_t* W_in = A.W_in;
    auto rows = [W_in, d](int i) { return W_in + int64_t(i) * 2 * d; };
    FZ_STREAM(rows, DM, d, FZ_RESID_BODY(Xs, XLD));
  }
  {
    FZ_LANE_VARS
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const int r = th * 64 + tt * 32 + l32;
      const int info = tinfo[r];
      const bool valid = (info >> 16) & 1;
      const int act = info & 0xFF, tim = (info >> 8) & 0xFF;
      const int p = valid ? p0 + r : 0;
#pragma unroll
      for (int ft = 0; ft < 2; ++ft)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int f = fq * 64 + ft * 32 + 8 * j + 4 * hf;
          const uint2 ea = *reinterpret_cast<const uint2*>(A.E_act + act * DM + f);
          const uint2 ep = *reinterpret_cast<const uint2*>(A.E_pos + int64_t(p) * DM + f);
          uint2 et = make_uint2(0, 0);
          if (A.E_time) et = *reinterpret_cast<const uint2*>(A.E_time + tim * DM + f);
          const bf16_t* eap = reinterpret_cast<const bf16_t*>(&ea);
          const bf16_t* epp = reinterpret_cast<const bf16_t*>(&ep);
          const bf16_t* etp = reinterpret_cast<const bf16_t*>(&et);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float v = acc[ft][tt][4 * j + i];
            acc[ft][tt][4 * j + i] =
                valid ? v + cvec[f + i] + bf2f(eap[i]) + bf2f(epp[i]) + bf2f(etp[i]) : 0.f;
          }
        }
    }
    __syncthreads();   // every wave is past Xs (tokens), cvec and tinfo
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int ft = 0; ft < 2; ++ft)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          st4(Xs + (th * 64 + tt * 32 + l32) * XLD + fq * 64 + ft * 32 + 8 * j + 4 * hf,
              acc[ft][tt][4 * j], acc[ft][tt][4 * j + 1], acc[ft][tt][4 * j + 2],
              acc[ft][tt][4 * j + 3]);
    __syncthreads();
  }
}

// Attention sublayer of one layer for the block: per 64-dim head group, the
// group's Q / K / V^T into LDS (and K / V^T into the cache for later blocks),
// causal attention per head, and acc += O_g W_o[:, group]^T.
__device__ __forceinline__ void attention_sublayer(const Args& A, const tav2_layer& L,
                                                   f32x16 (&acc)[2][2], bf16_t* Xs, bf16_t* Ws,
                                                   bf16_t* Qs, bf16_t* Ks, bf16_t* Vts,
                                                   bf16_t* kc, bf16_t* vc, int p0, bool keep) {
  const bf16_t* Wqkv = static_cast<const bf16_t*>(L.W_qkv);
  const bf16_t* Wo = static_cast<const bf16_t*>(L.W_o);
  for (int g = 0; g < DM / 64; ++g) {
    {
      // wave w: token tile w & 3; column tiles 3(w >> 2) .. +2 of q0 q1 k0 k1 v0 v1
      FZ_LANE_VARS
      const int tt = w & 3;
      f32x16 qa[3];
#pragma unroll
      for (int t = 0; t < 3; ++t) qa[t] = f32x16{};
      auto rows = [Wqkv, g](int i) { return Wqkv + int64_t((i >> 6) * DM + g * 64 + (i & 63)) * DM; };
      if (w < 4) {   // q0 q1 k0: transposed
        FZ_STREAM(rows, 192, DM, {
          _Pragma("unroll") for (int kb = 0; kb < KS / 16; ++kb) {
            const bf16x8 xf = frag(Xs + (tt * 32 + l32) * XLD + k0 + kb * 16 + 8 * hf);
            _Pragma("unroll") for (int t = 0; t < 3; ++t) {
              const bf16x8 wf = frag(stage + (t * 32 + l32) * WLD + kb * 16 + 8 * hf);
              qa[t] = mfma32(wf, xf, qa[t]);
            }
          }
        });
      } else {       // k1 transposed; v0 v1 untransposed
        FZ_STREAM(rows, 192, DM, {
          _Pragma("unroll") for (int kb = 0; kb < KS / 16; ++kb) {
            const bf16x8 xf = frag(Xs + (tt * 32 + l32) * XLD + k0 + kb * 16 + 8 * hf);
            const bf16x8 w3 = frag(stage + (3 * 32 + l32) * WLD + kb * 16 + 8 * hf);
            const bf16x8 w4 = frag(stage + (4 * 32 + l32) * WLD + kb * 16 + 8 * hf);
            const bf16x8 w5 = frag(stage + (5 * 32 + l32) * WLD + kb * 16 + 8 * hf);
            qa[0] = mfma32(w3, xf, qa[0]);
            qa[1] = mfma32(xf, w4, qa[1]);
            qa[2] = mfma32(xf, w5, qa[2]);
          }
        });
      }
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const int ct = (w >> 2) * 3 + t;
        const int part = ct >> 1;                 // 0 q, 1 k, 2 v
        const int dt = ct & 1;
        const float* bias = L.b_qkv + part * DM + g * 64 + dt * 32;
        if (part < 2) {
          bf16_t* dst = part == 0 ? Qs : Ks;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int dim = 8 * j + 4 * hf;
            const float4 bv = *reinterpret_cast<const float4*>(bias + dim);
            st4(dst + (tt * 32 + l32) * QLD + dt * 32 + dim, qa[t][4 * j] + bv.x,
                qa[t][4 * j + 1] + bv.y, qa[t][4 * j + 2] + bv.z, qa[t][4 * j + 3] + bv.w);
          }
        } else {
          const float bv = bias[l32];
#pragma unroll
          for (int j = 0; j < 4; ++j)
            st4(Vts + (dt * 32 + l32) * VLD + tt * 32 + 8 * j + 4 * hf, qa[t][4 * j] + bv,
                qa[t][4 * j + 1] + bv, qa[t][4 * j + 2] + bv, qa[t][4 * j + 3] + bv);
        }
      }
    }
    __syncthreads();
    if (keep) {   // this block's K and V^T for the later blocks of the candidate
      const int tid = otid();
      for (int e = tid; e < BT * 8; e += NT) {
        const int r = e >> 3, c = (e & 7) * 8;
        *reinterpret_cast<uint4*>(kc + int64_t(p0 + r) * DM + g * 64 + c) =
            *reinterpret_cast<const uint4*>(Ks + r * QLD + c);
      }
      for (int e = tid; e < 64 * (BT / 8); e += NT) {
        const int r = e / (BT / 8), c = (e % (BT / 8)) * 8;
        *reinterpret_cast<uint4*>(vc + int64_t(g * 64 + r) * A.tpad + p0 + c) =
            *reinterpret_cast<const uint4*>(Vts + r * VLD + c);
      }
    }
    if (A.dh == 64) {
      attend_head<64>(g, 0, p0, Qs, Ks, Vts, kc, vc, A.tpad);
    } else {
      attend_head<32>(g, 0, p0, Qs, Ks, Vts, kc, vc, A.tpad);
      attend_head<32>(g, 32, p0, Qs, Ks, Vts, kc, vc, A.tpad);
    }
    __syncthreads();
    {   // acc += O_g W_o[:, 64g : 64g + 64]^T
      FZ_LANE_VARS
      auto rows = [Wo, g](int i) { return Wo + int64_t(i) * DM + g * 64; };
      FZ_STREAM(rows, DM, 64, FZ_RESID_BODY(Qs, QLD));
    }
  }
}

// FFN sublayer: per chunk of 128 hidden units, H^T = ReLU(W_1[chunk] Xs^T + b_1)
// into LDS, then acc += W_2[:, chunk] H^T.
__device__ __forceinline__ void ffn_sublayer(const Args& A, const tav2_layer& L,
                                             f32x16 (&acc)[2][2], bf16_t* Xs, bf16_t* Ws,
                                             bf16_t* Hs) {
  const bf16_t* W1 = static_cast<const bf16_t*>(L.W_1);
  const bf16_t* W2 = static_cast<const bf16_t*>(L.W_2);
  const int ffn = A.ffn;
  for (int c = 0; c < ffn / FC; ++c) {
    {
      // wave w: hidden tile w & 3, token tiles 2(w >> 2) and 2(w >> 2) + 1
      FZ_LANE_VARS
      const int ht = w & 3, tp = w >> 2;
      f32x16 ha[2];
      ha[0] = f32x16{};
      ha[1] = f32x16{};
      auto rows = [W1, c](int i) { return W1 + int64_t(c * FC + i) * DM; };
      FZ_STREAM(rows, FC, DM, {
        _Pragma("unroll") for (int kb = 0; kb < KS / 16; ++kb) {
          const bf16x8 wf = frag(stage + (ht * 32 + l32) * WLD + kb * 16 + 8 * hf);
          _Pragma("unroll") for (int t = 0; t < 2; ++t) {
            const bf16x8 xf = frag(Xs + ((2 * tp + t) * 32 + l32) * XLD + k0 + kb * 16 + 8 * hf);
            ha[t] = mfma32(wf, xf, ha[t]);
          }
        }
      });
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int hid = ht * 32 + 8 * j + 4 * hf;
          const float4 bv = *reinterpret_cast<const float4*>(L.b_1 + c * FC + hid);
          st4(Hs + ((2 * tp + t) * 32 + l32) * HLD + hid, fmaxf(ha[t][4 * j] + bv.x, 0.f),
              fmaxf(ha[t][4 * j + 1] + bv.y, 0.f), fmaxf(ha[t][4 * j + 2] + bv.z, 0.f),
              fmaxf(ha[t][4 * j + 3] + bv.w, 0.f));
        }
    }
    __syncthreads();
    {
      FZ_LANE_VARS
      auto rows = [W2, c, ffn](int i) { return W2 + int64_t(i) * ffn + c * FC; };
      FZ_STREAM(rows, DM, FC, FZ_RESID_BODY(Hs, HLD));
    }
  }
}

__global__ __launch_bounds__(NT) void encoder_fused_kernel(Args A) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[LDS_BYTES];
  bf16_t* Xs = reinterpret_cast<bf16_t*>(smem);
  bf16_t* Ws = reinterpret_cast<bf16_t*>(smem + XS_BYTES);
  uint8_t* Sc = smem + XS_BYTES + WS_BYTES;
  float* pmax = reinterpret_cast<float*>(smem + XS_BYTES + WS_BYTES + SC_BYTES);
  bf16_t* Qs = reinterpret_cast<bf16_t*>(Sc);                    // [BT][QLD], then O
  bf16_t* Ks = reinterpret_cast<bf16_t*>(Sc + QS_BYTES);         // [BT][QLD]
  bf16_t* Vts = reinterpret_cast<bf16_t*>(Sc + 2 * QS_BYTES);    // [64][VLD]
  bf16_t* Hs = reinterpret_cast<bf16_t*>(Sc);                    // [BT][HLD]
  float* red = reinterpret_cast<float*>(Sc);                     // reductions
  float* cvec = reinterpret_cast<float*>(Sc);                    // [DM] during encoding
  int* tinfo = reinterpret_cast<int*>(Sc + DM * 4);              // [BT] during encoding

  const int64_t nl = blockIdx.x;
  const int64_t n = A.c0 + nl;
  const int Tv = token_valid_len(A.s, n);
  float* out = A.out + n * 2 * DM;
  if (Tv == 0) {
    for (int c = threadIdx.x; c < 2 * DM; c += NT) out[c] = 0.f;
    return;
  }
  const int nblk = (Tv + BT - 1) / BT;
  for (int c = threadIdx.x; c < DM; c += NT) pmax[c] = -__builtin_inff();
  // layer records are read through the kernel-argument segment so the runtime
  // layer index stays a scalar load instead of a private copy of the array
  const Args* AK = (const Args*)(__builtin_amdgcn_kernarg_segment_ptr());

  f32x16 acc[2][2];
  for (int blk = 0; blk < nblk; ++blk) {
    const int p0 = blk * BT;
    __syncthreads();
    encode_block_input(A, n, p0, Tv, acc, Xs, Ws, cvec, tinfo);
    for (int li = 0; li < A.n_layers; ++li) {
      const tav2_layer L = AK->layers[li];
      bf16_t* kc = A.kcache ? A.kcache + (nl * A.n_layers + li) * int64_t(A.tpad) * DM : nullptr;
      bf16_t* vc = A.vcache ? A.vcache + (nl * A.n_layers + li) * int64_t(DM) * A.tpad : nullptr;
      attention_sublayer(A, L, acc, Xs, Ws, Qs, Ks, Vts, kc, vc, p0, blk + 1 < nblk);
      layer_norm(acc, L.b_o, L.ln1_g, L.ln1_b, red, Xs);
      ffn_sublayer(A, L, acc, Xs, Ws, Hs);
      layer_norm(acc, L.b_2, L.ln2_g, L.ln2_b, red, Xs);
    }
    // ---- head: out[DM:] = X of the last valid token; running max of the pool
    {
      FZ_LANE_VARS
      const int last = Tv - 1 - p0;
      if (last >= 0 && last < BT) {
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
          if (th * 64 + tt * 32 + l32 == last) {
#pragma unroll
            for (int ft = 0; ft < 2; ++ft)
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                const int f = fq * 64 + ft * 32 + 8 * j + 4 * hf;
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
      for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};
    {
      FZ_LANE_VARS
      const bf16_t* Wp = A.W_pool;
      auto rows = [Wp](int i) { return Wp + int64_t(i) * DM; };
      FZ_STREAM(rows, DM, DM, FZ_RESID_BODY(Xs, XLD));
    }
    pool_block(acc, A.b_pool, pmax, red, Tv - p0);
  }
  for (int c = threadIdx.x; c < DM; c += NT) out[c] = pmax[c];
}

}  // namespace fz

// ---------------------------------------------------------------- host side
namespace {
constexpr size_t CACHE_BUDGET = size_t(2) << 30;   // bytes of K/V cache per launch

int64_t fused_tpad(int T) { return (T + fz::BT - 1) / fz::BT * fz::BT; }

size_t per_candidate_cache(int T, const tav2_weights& w) {
  if (T <= fz::BT) return 0;
  return size_t(w.n_layers) * 2 * size_t(fused_tpad(T)) * fz::DM * 2;
}

int64_t fused_chunk(int64_t total, int T, const tav2_weights& w) {
  const size_t per = per_candidate_cache(T, w);
  if (per == 0) return total > 0 ? total : 1;
  int64_t c = int64_t(CACHE_BUDGET / per);
  if (c < 1) c = 1;
  return c < total ? c : (total > 0 ? total : 1);
}
}  // namespace

bool encode_fused_supported(int d, const tav2_weights& w) {
  const int dh = w.d_model / w.n_heads;
  return w.d_model == fz::DM && (dh == 32 || dh == 64) && w.d_ffn % fz::FC == 0 &&
         d % 32 == 0 && d <= fz::DM && w.n_layers <= fz::MAX_LAYERS;
}

size_t encode_fused_workspace(int64_t total, int T, const tav2_weights& w) {
  const size_t per = per_candidate_cache(T, w);
  return per * size_t(fused_chunk(total, T, w));
}

hipError_t launch_encode_fused(const TokenSource& src, const void* cand_emb, int64_t total,
                               const tav2_weights& w, float* out, void* ws, hipStream_t st) {
  if (total == 0) return hipSuccess;
  fz::Args a{};
  a.s = src;
  a.cand = static_cast<const bf16_t*>(cand_emb);
  a.W_in = static_cast<const bf16_t*>(w.W_in);
  a.b_in = w.b_in;
  a.E_act = static_cast<const bf16_t*>(w.E_act);
  a.E_time = static_cast<const bf16_t*>(w.E_time);
  a.E_pos = static_cast<const bf16_t*>(w.E_pos);
  a.W_pool = static_cast<const bf16_t*>(w.W_pool);
  a.b_pool = w.b_pool;
  for (int i = 0; i < w.n_layers; ++i) a.layers[i] = w.layers[i];
  a.n_layers = w.n_layers;
  a.d = src.d;
  a.dh = w.d_model / w.n_heads;
  a.ffn = w.d_ffn;
  a.tpad = int(fused_tpad(src.T));
  a.out = out;
  const size_t per = per_candidate_cache(src.T, w);
  const int64_t chunk = fused_chunk(total, src.T, w);
  for (int64_t c0 = 0; c0 < total; c0 += chunk) {
    const int64_t nc = total - c0 < chunk ? total - c0 : chunk;
    a.c0 = c0;
    if (per) {
      a.kcache = static_cast<bf16_t*>(ws);
      a.vcache = reinterpret_cast<bf16_t*>(static_cast<uint8_t*>(ws) + per / 2 * size_t(chunk));
    }
    ProfScope prof("encoder_fused", st);
    fz::encoder_fused_kernel<<<unsigned(nc), fz::NT, 0, st>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace tav2
