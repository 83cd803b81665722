// Single-kernel encoder for the paper's production encoder shape: d_model 64,
// one or two heads, a narrow FFN, a few layers (Sec. 3.2.2 'Transformer
// Encoder'; the fused transformer of Sec. 3.4.2 keeps every transformer weight
// on chip next to the activations).  One workgroup runs Eq. 4's feature
// encoding, every causal post-LN layer and the linear + max-pool head for one
// candidate at a time, with all layer weights resident in LDS.
//
// Layout of the work:
//  * The workgroup is persistent: it loads every weight into LDS once and then
//    takes candidates blockIdx.x, blockIdx.x + gridDim.x, ...
//  * A candidate's positions are processed in blocks of 64; under the causal
//    mask a block depends on earlier blocks only through their keys and values,
//    which each block leaves in a per-workgroup cache in global memory.
//  * 4 waves; wave w owns tokens 16 w .. +15 of the block in every phase except
//    attention's key loop.  The fp32 residual stream of those tokens stays in
//    registers as X^T tiles (16x16x32 MFMA accumulator layout: lane l holds
//    token l % 16, features 16 f + 4 (l / 16) + i), so LayerNorm is an in-lane sum
//    plus two lane exchanges.
//  * Products whose consumer wants [token][feature] rows are computed
//    transposed (weights as the A operand), so every LDS write is 4 consecutive
//    bf16 of one row; V is computed untransposed to give V^T [dim][key], with
//    each 32-key pair's keys in the order of the P^T fragment.
//  * Attention: S^T = K Q^T (one query per lane column), online softmax over
//    32-key pairs in registers, O^T += V^T P^T; keys of earlier blocks are read
//    from the cache straight into MFMA operands.
#include <atomic>

#include "common.h"
#include "internal.h"
#include "token_source.h"

namespace tav2 {
namespace sm {

constexpr int DM = 64;          // d_model
constexpr int BT = 64;          // tokens per block
constexpr int NT = 256;         // threads (4 waves, 16 tokens each)
constexpr int RLD = DM + 8;     // row stride (bf16) of [*][64] activations and weights
constexpr int MAX_LAYERS = 4;

typedef float f32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f32x4 mma(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// 16x16x32 operands: A[16 x 32] lane l: row l % 16, k = 8 (l / 16) .. +7;
// B[32 x 16] lane l: column l % 16, same k; D[16 x 16] lane l: column l % 16,
// rows 4 (l / 16) + i in register i.
__device__ __forceinline__ bf16x8 frag(const bf16_t* p) {
  return as_bf16x8(*reinterpret_cast<const uint4*>(p));
}
__device__ __forceinline__ void put4(bf16_t* p, float a, float b, float c, float d) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack2(a, b), pack2(c, d));
}
// Position of key k (0..31) of a 32-key pair in a V^T row: the P^T fragment's
// order, where lane group g holds keys 4 g .. +3 and 16 + 4 g .. +3 as k-rows
// 8 g .. +7.
__device__ __forceinline__ int vpos(int k) { return 8 * ((k >> 2) & 3) + 4 * (k >> 4) + (k & 3); }

struct LayerW {   // LDS offsets (bytes) of one layer's weights
  int qkv, o, w1, w2, vec;
};
struct Args {
  TokenSource s;
  const bf16_t* cand;        // [total, d]
  const bf16_t* W_in;        // [DM, 2 d]
  const float* b_in;
  const bf16_t* E_act;       // [8, DM]
  const bf16_t* E_time;      // [64, DM] or null
  const bf16_t* E_pos;       // [max_pos, DM]
  const bf16_t* W_pool;      // [DM, DM]
  const float* b_pool;
  tav2_layer layers[MAX_LAYERS];
  int n_layers, d, dh, ffn;
  int64_t total;
  int tpad;                  // cache stride in positions (T rounded up to BT)
  bf16_t* kcache;            // [grid][layers][tpad][DM]
  bf16_t* vcache;            // [grid][layers][DM][tpad]
  float* out;                // [total, 2 DM]
  // LDS layout (bytes)
  LayerW lw[MAX_LAYERS];
  int win, wpool, xb, q, k, vt, h, cvec, pool, tinfo, rowp, lds_bytes;
  int unmasked;
};

// LDS layout: weights first (loaded once), then the block's activations.
__host__ __device__ inline void plan_lds(Args& a) {
  int off = 0;
  auto take = [&](int bytes) {
    const int at = off;
    off += (bytes + 15) / 16 * 16;
    return at;
  };
  const int fld = a.ffn + 8;   // row stride of [*][ffn] matrices
  for (int l = 0; l < a.n_layers; ++l) {
    a.lw[l].qkv = take(3 * DM * RLD * 2);
    a.lw[l].o = take(DM * RLD * 2);
    a.lw[l].w1 = take(a.ffn * RLD * 2);
    a.lw[l].w2 = take(DM * fld * 2);
    a.lw[l].vec = take((3 * DM + DM + 2 * DM + a.ffn + DM + 2 * DM) * 4);
  }
  a.win = take(DM * (a.d + 8) * 2);
  a.wpool = take(DM * RLD * 2);
  a.xb = take(BT * RLD * 2);
  a.q = take(BT * RLD * 2);    // Q, then the attention output O
  a.k = take(BT * RLD * 2);
  a.vt = take(DM * RLD * 2);   // V^T [dim][key]
  a.h = take(BT * fld * 2);
  a.cvec = take(DM * 4);
  a.pool = take(5 * DM * 4);   // running maxima, then one partial per wave
  a.tinfo = take(BT * 4);
  a.rowp = take(BT * 8);
  a.lds_bytes = off;
}
// Offsets of the layer vectors inside lw.vec (floats).
constexpr int V_BQKV = 0, V_BO = 3 * DM, V_LN1G = 4 * DM, V_LN1B = 5 * DM, V_B1 = 6 * DM;
__device__ __forceinline__ int v_b2(int ffn) { return 6 * DM + ffn; }
__device__ __forceinline__ int v_ln2g(int ffn) { return 7 * DM + ffn; }
__device__ __forceinline__ int v_ln2b(int ffn) { return 8 * DM + ffn; }

// Orders a wave's LDS writes before its later LDS reads of rows other lanes wrote
// (the wave's own token rows: no workgroup barrier is needed for them).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Copy a row-major [rows][cols] bf16 matrix into LDS rows of stride ld.
__device__ __forceinline__ void copy_matrix(bf16_t* dst, int ld, const bf16_t* src, int rows,
                                            int cols) {
  const int per = cols / 8;
  for (int e = threadIdx.x; e < rows * per; e += NT) {
    const int r = e / per, c = e % per;
    *reinterpret_cast<uint4*>(dst + r * ld + c * 8) =
        *reinterpret_cast<const uint4*>(src + int64_t(r) * cols + c * 8);
  }
}
__device__ __forceinline__ void copy_floats(float* dst, const float* src, int n) {
  for (int e = threadIdx.x; e < n; e += NT) dst[e] = src[e];
}

// ---------------------------------------------------------------- LayerNorm
// acc[f] (f = feature tile) holds X^T of the lane's token: features 16 f + 4 g + i.
// Normalises over the 64 features (two passes: mean, then the centred squares).
__device__ __forceinline__ void layer_norm(f32x4 (&x)[4], const float* g, const float* b) {
  const int lane = threadIdx.x % WAVE, grp = lane / 16;
  float s = 0.f;
#pragma unroll
  for (int f = 0; f < 4; ++f) s += (x[f][0] + x[f][1]) + (x[f][2] + x[f][3]);
  s += __shfl_xor(s, 16, WAVE);
  s += __shfl_xor(s, 32, WAVE);
  const float mean = s * (1.f / DM);
  float v = 0.f;
#pragma unroll
  for (int f = 0; f < 4; ++f)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float c = x[f][i] - mean;
      v = fmaf(c, c, v);
    }
  v += __shfl_xor(v, 16, WAVE);
  v += __shfl_xor(v, 32, WAVE);
  const float rstd = rsqrtf(v * (1.f / DM) + 1e-5f);
#pragma unroll
  for (int f = 0; f < 4; ++f) {
    const float4 gg = *reinterpret_cast<const float4*>(g + 16 * f + 4 * grp);
    const float4 bb = *reinterpret_cast<const float4*>(b + 16 * f + 4 * grp);
    x[f][0] = fmaf((x[f][0] - mean) * rstd, gg.x, bb.x);
    x[f][1] = fmaf((x[f][1] - mean) * rstd, gg.y, bb.y);
    x[f][2] = fmaf((x[f][2] - mean) * rstd, gg.z, bb.z);
    x[f][3] = fmaf((x[f][3] - mean) * rstd, gg.w, bb.w);
  }
}
// Xb rows of the wave's tokens <- bf16(x).
__device__ __forceinline__ void store_xb(bf16_t* Xb, const f32x4 (&x)[4]) {
  const int lane = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
  bf16_t* row = Xb + (16 * w + lane % 16) * RLD + 4 * (lane / 16);
#pragma unroll
  for (int f = 0; f < 4; ++f) put4(row + 16 * f, x[f][0], x[f][1], x[f][2], x[f][3]);
  wave_lds_sync();
}
// The 4 bf16 at p (8-byte aligned) added to v.
__device__ __forceinline__ void add4(float (&v)[4], const bf16_t* p) {
  const uint2 r = *reinterpret_cast<const uint2*>(p);
  v[0] += __uint_as_float(r.x << 16);
  v[1] += __uint_as_float(r.x & 0xFFFF0000u);
  v[2] += __uint_as_float(r.y << 16);
  v[3] += __uint_as_float(r.y & 0xFFFF0000u);
}

// acc[f] += W[16 f + .., :K] X^T for the wave's tokens: A = W rows (LDS, stride
// wld), B = the tokens' rows of ACT (LDS, stride ald), K a multiple of 32.
template <int NF>
__device__ __forceinline__ void wt_product(f32x4 (&acc)[NF], const bf16_t* W, int wld,
                                           const bf16_t* ACT, int ald, int K) {
  const int lane = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
  const int c16 = lane % 16, g = lane / 16;
  const bf16_t* arow = W + c16 * wld + 8 * g;
  const bf16_t* brow = ACT + (16 * w + c16) * ald + 8 * g;
  for (int k0 = 0; k0 < K; k0 += 32) {
    const bf16x8 b = frag(brow + k0);
#pragma unroll
    for (int f = 0; f < NF; ++f) acc[f] = mma(frag(arow + 16 * f * wld + k0), b, acc[f]);
  }
}

// ---------------------------------------------------------------- attention
// Online softmax state of one 16-query tile and head (queries in lane columns).
template <int DH>
struct Att {
  bf16x8 qf[DH / 32];   // Q^T fragments
  f32x4 o[DH / 16];     // O^T accumulators
  float m, l;           // running max (log2 units), this lane's partial row sum
};

// One 32-key pair: keys from K rows (A operand rows: key, k = dims) and V^T
// columns (A operand of O^T += V^T P^T: rows dims, k = keys in vpos order).  Key
// j of the pair is visible to the lane's query iff j < lim (32: all).  Before the
// first visible key the running max is -inf: the exponents then use 0 as
// reference, which gives zero weights and a zero rescale of the (zero) sums.
template <int DH>
__device__ __forceinline__ void att_pair(Att<DH>& st, const bf16_t* K, int kld, const bf16_t* Vt,
                                         int vld, int col0, int lim, float scale_l2) {
  const int lane = threadIdx.x % WAVE;
  const int c16 = lane % 16, g = lane / 16;
  f32x4 s[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < DH / 32; ++kb)
      a = mma(frag(K + (16 * t + c16) * kld + col0 + 32 * kb + 8 * g), st.qf[kb], a);
    s[t] = a;
  }
  // key 16 t + 4 g + i of the pair
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (4 * g + i >= lim) s[0][i] = -__builtin_inff();
    if (16 + 4 * g + i >= lim) s[1][i] = -__builtin_inff();
  }
  float mx = -__builtin_inff();
#pragma unroll
  for (int t = 0; t < 2; ++t)
    mx = fmaxf(mx, fmaxf(fmaxf(s[t][0], s[t][1]), fmaxf(s[t][2], s[t][3])));
  mx = fmaxf(mx, __shfl_xor(mx, 16, WAVE));
  mx = fmaxf(mx, __shfl_xor(mx, 32, WAVE));
  const float mnew = fmaxf(st.m, mx * scale_l2);
  const float mref = mnew == -__builtin_inff() ? 0.f : mnew;
  const float alpha = exp2f(st.m - mref);
  st.l *= alpha;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) st.o[dt] *= alpha;
  st.m = mnew;
  bf16x8 pb;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = exp2f(fmaf(s[t][i], scale_l2, -mref));
      st.l += p;
      pb[4 * t + i] = static_cast<__bf16>(p);
    }
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt)
    st.o[dt] = mma(frag(Vt + (col0 + 16 * dt + c16) * vld + 8 * g), pb, st.o[dt]);
}

// Attention of the wave's 16 queries (block positions 16 w ..) for one head: the
// block's own keys 0 .. 16 w + 15 (causal; unmasked: 0 .. nkv - 1), then earlier
// blocks' keys from the cache.  Leaves O = softmax(S) V in the Q rows.
template <int DH>
__device__ __forceinline__ void attend(bf16_t* Qs, const bf16_t* Ks, const bf16_t* Vts,
                                       const bf16_t* kc, const bf16_t* vc, int tpad, int p0,
                                       int col0, int nkv, bool unmasked) {
  const int lane = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
  const int c16 = lane % 16, g = lane / 16;
  constexpr float scale_l2 = (DH == 64 ? 0.125f : 0.17677669529663688f) * 1.4426950408889634f;
  Att<DH> st;
#pragma unroll
  for (int kb = 0; kb < DH / 32; ++kb) st.qf[kb] = frag(Qs + (16 * w + c16) * RLD + col0 + 32 * kb + 8 * g);
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) st.o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -__builtin_inff();
  st.l = 0.f;
  // earlier blocks: every key visible
  for (int c0 = 0; c0 < p0; c0 += 32)
    att_pair<DH>(st, kc + int64_t(c0) * DM, DM, vc + c0, tpad, col0, 32, scale_l2);
  // own block: query 16 w + c16 sees keys <= itself (causal) or < nkv (unmasked)
  const int q = 16 * w + c16;
  const int kend = unmasked ? nkv : 16 * (w + 1);
  for (int k0 = 0; k0 < kend; k0 += 32) {
    const int lim = unmasked ? nkv - k0 : q + 1 - k0;   // keys k0 + j visible iff j < lim
    att_pair<DH>(st, Ks + k0 * RLD, RLD, Vts + k0, RLD, col0, lim, scale_l2);
  }
  float l = st.l;
  l += __shfl_xor(l, 16, WAVE);
  l += __shfl_xor(l, 32, WAVE);
  const float inv = 1.f / l;
  // O^T tile dt: lane holds query c16, dims 16 dt + 4 g + i
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt)
    put4(Qs + (16 * w + c16) * RLD + col0 + 16 * dt + 4 * g, st.o[dt][0] * inv,
         st.o[dt][1] * inv, st.o[dt][2] * inv, st.o[dt][3] * inv);
  wave_lds_sync();
}

// ---------------------------------------------------------------- the kernel
__global__ __launch_bounds__(NT) void encoder_small_kernel(Args A) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int tid = threadIdx.x, lane = tid % WAVE, w = tid / WAVE;
  const int c16 = lane % 16, g = lane / 16;
  const int d = A.d, ffn = A.ffn, fld = ffn + 8;
  // ---- weights into LDS, once
  for (int l = 0; l < A.n_layers; ++l) {
    const tav2_layer& L = A.layers[l];
    copy_matrix(reinterpret_cast<bf16_t*>(smem + A.lw[l].qkv), RLD,
                static_cast<const bf16_t*>(L.W_qkv), 3 * DM, DM);
    copy_matrix(reinterpret_cast<bf16_t*>(smem + A.lw[l].o), RLD, static_cast<const bf16_t*>(L.W_o),
                DM, DM);
    copy_matrix(reinterpret_cast<bf16_t*>(smem + A.lw[l].w1), RLD,
                static_cast<const bf16_t*>(L.W_1), ffn, DM);
    copy_matrix(reinterpret_cast<bf16_t*>(smem + A.lw[l].w2), fld,
                static_cast<const bf16_t*>(L.W_2), DM, ffn);
    float* v = reinterpret_cast<float*>(smem + A.lw[l].vec);
    copy_floats(v + V_BQKV, L.b_qkv, 3 * DM);
    copy_floats(v + V_BO, L.b_o, DM);
    copy_floats(v + V_LN1G, L.ln1_g, DM);
    copy_floats(v + V_LN1B, L.ln1_b, DM);
    copy_floats(v + V_B1, L.b_1, ffn);
    copy_floats(v + v_b2(ffn), L.b_2, DM);
    copy_floats(v + v_ln2g(ffn), L.ln2_g, DM);
    copy_floats(v + v_ln2b(ffn), L.ln2_b, DM);
  }
  {   // token half of W_in: columns 0 .. d - 1 of [DM][2 d]
    bf16_t* dst = reinterpret_cast<bf16_t*>(smem + A.win);
    const int per = d / 8;
    for (int e = tid; e < DM * per; e += NT) {
      const int r = e / per, c = e % per;
      *reinterpret_cast<uint4*>(dst + r * (d + 8) + c * 8) =
          *reinterpret_cast<const uint4*>(A.W_in + int64_t(r) * 2 * d + c * 8);
    }
  }
  copy_matrix(reinterpret_cast<bf16_t*>(smem + A.wpool), RLD, A.W_pool, DM, DM);
  bf16_t* Xb = reinterpret_cast<bf16_t*>(smem + A.xb);
  bf16_t* Qs = reinterpret_cast<bf16_t*>(smem + A.q);
  bf16_t* Ks = reinterpret_cast<bf16_t*>(smem + A.k);
  bf16_t* Vts = reinterpret_cast<bf16_t*>(smem + A.vt);
  bf16_t* Hs = reinterpret_cast<bf16_t*>(smem + A.h);
  float* cvec = reinterpret_cast<float*>(smem + A.cvec);
  float* pool = reinterpret_cast<float*>(smem + A.pool);
  int* tinfo = reinterpret_cast<int*>(smem + A.tinfo);
  const uint8_t** rowp = reinterpret_cast<const uint8_t**>(smem + A.rowp);
  const bf16_t* Win = reinterpret_cast<const bf16_t*>(smem + A.win);
  const bf16_t* Wpool = reinterpret_cast<const bf16_t*>(smem + A.wpool);
  bf16_t* kc_wg = A.kcache ? A.kcache + int64_t(blockIdx.x) * A.n_layers * A.tpad * DM : nullptr;
  bf16_t* vc_wg = A.vcache ? A.vcache + int64_t(blockIdx.x) * A.n_layers * DM * A.tpad : nullptr;

  for (int64_t n = blockIdx.x; n < A.total; n += gridDim.x) {
    __syncthreads();   // weights loaded; the previous candidate is done with the buffers
    const int Tv = token_valid_len(A.s, n);
    float* out = A.out + n * 2 * DM;
    if (Tv == 0) {
      for (int c = tid; c < 2 * DM; c += NT) out[c] = 0.f;
      continue;
    }
    // candidate half of the input projection and the pooled maxima
    if (tid < DM) {   // W_in[:, d:] c + b_in, 8 columns per load
      const uint4* wr = reinterpret_cast<const uint4*>(A.W_in + int64_t(tid) * 2 * d + d);
      const uint4* cr = reinterpret_cast<const uint4*>(A.cand + n * d);
      float acc = A.b_in[tid];
#pragma unroll 4
      for (int j = 0; j < d / 8; ++j) {
        const bf16x8 a = as_bf16x8(wr[j]), b = as_bf16x8(cr[j]);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = fmaf(float(a[u]), float(b[u]), acc);
      }
      cvec[tid] = acc;
    } else if (tid < 2 * DM) {
      pool[tid - DM] = -__builtin_inff();
    }
    const int nblk = (Tv + BT - 1) / BT;
    for (int blk = 0; blk < nblk; ++blk) {
      const int p0 = blk * BT;
      const int nv = Tv - p0 < BT ? Tv - p0 : BT;   // valid positions of the block
      // ---- resolve the block's tokens
      if (tid < BT) {
        const int p = p0 + tid;
        const uint8_t* rp = nullptr;
        int info = 0;
        if (p < Tv) {
          const TokenRef t = resolve_token(A.s, n, p, d * 2);
          rp = t.emb;
          info = t.act | (t.time << 8);
        }
        rowp[tid] = rp;
        tinfo[tid] = info;
      }
      __syncthreads();
      // ---- Eq. 4: X0^T = W_in[:, :d] E^T + cvec + E_act + E_time + E_pos
      f32x4 x[4];
      {
        const int tok = 16 * w + c16;          // this lane's token (B operand column)
        const uint8_t* rp = rowp[tok];
#pragma unroll
        for (int f = 0; f < 4; ++f) x[f] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int k0 = 0; k0 < d; k0 += 32) {
          bf16x8 b{};
          if (rp) b = frag(reinterpret_cast<const bf16_t*>(rp) + k0 + 8 * g);
#pragma unroll
          for (int f = 0; f < 4; ++f)
            x[f] = mma(frag(Win + (16 * f + c16) * (d + 8) + k0 + 8 * g), b, x[f]);
        }
        // D of the transposed product: lane holds token c16 (of the wave's tile),
        // features 16 f + 4 g + i
        const int info = tinfo[16 * w + c16];
        const int act = info & 0xFF, tim = (info >> 8) & 0xFF;
        const int p = p0 + 16 * w + c16;
        const bool valid = p < Tv;
#pragma unroll
        for (int f = 0; f < 4; ++f) {
          const int feat = 16 * f + 4 * g;
          float v[4] = {0.f, 0.f, 0.f, 0.f};
          if (valid) {
            add4(v, A.E_act + act * DM + feat);
            add4(v, A.E_pos + int64_t(p) * DM + feat);
            if (A.E_time) add4(v, A.E_time + tim * DM + feat);
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) x[f][i] += cvec[feat + i] + v[i];
        }
        store_xb(Xb, x);
      }
      // ---- layers
      for (int li = 0; li < A.n_layers; ++li) {
        const bf16_t* Wqkv = reinterpret_cast<const bf16_t*>(smem + A.lw[li].qkv);
        const bf16_t* Wo = reinterpret_cast<const bf16_t*>(smem + A.lw[li].o);
        const bf16_t* W1 = reinterpret_cast<const bf16_t*>(smem + A.lw[li].w1);
        const bf16_t* W2 = reinterpret_cast<const bf16_t*>(smem + A.lw[li].w2);
        const float* vec = reinterpret_cast<const float*>(smem + A.lw[li].vec);
        bf16_t* kc = kc_wg ? kc_wg + int64_t(li) * A.tpad * DM : nullptr;
        bf16_t* vc = vc_wg ? vc_wg + int64_t(li) * DM * A.tpad : nullptr;
        // Q and K transposed (rows of Wq / Wk as A), V untransposed (X as A)
        f32x4 qk[8];
#pragma unroll
        for (int f = 0; f < 8; ++f) qk[f] = f32x4{0.f, 0.f, 0.f, 0.f};
        wt_product<8>(qk, Wqkv, RLD, Xb, RLD, DM);
        f32x4 vv[4];
#pragma unroll
        for (int f = 0; f < 4; ++f) vv[f] = f32x4{0.f, 0.f, 0.f, 0.f};
        {
          const bf16_t* arow = Xb + (16 * w + c16) * RLD + 8 * g;   // A: the wave's tokens
          const bf16_t* brow = Wqkv + (2 * DM + c16) * RLD + 8 * g;  // B: W_v rows (columns of V)
          for (int k0 = 0; k0 < DM; k0 += 32) {
            const bf16x8 a = frag(arow + k0);
#pragma unroll
            for (int f = 0; f < 4; ++f) vv[f] = mma(a, frag(brow + 16 * f * RLD + k0), vv[f]);
          }
        }
        __syncthreads();   // every wave is past the previous layer's attention (K, V^T reads)
        {
          const int tok = 16 * w + c16;
#pragma unroll
          for (int f = 0; f < 8; ++f) {   // Q (f < 4) and K (f >= 4): lane token c16, dims 16 (f % 4) + 4 g + i
            const int dcol = 16 * (f % 4) + 4 * g;
            const float* bias = vec + V_BQKV + 16 * f + 4 * g;
            bf16_t* dst = (f < 4 ? Qs : Ks) + tok * RLD + dcol;
            put4(dst, qk[f][0] + bias[0], qk[f][1] + bias[1], qk[f][2] + bias[2], qk[f][3] + bias[3]);
          }
          // V: D[token][dim]: lane holds dim 16 f + c16, tokens 16 w + 4 g + i
#pragma unroll
          for (int f = 0; f < 4; ++f) {
            const int dim = 16 * f + c16;
            const float bv = vec[V_BQKV + 2 * DM + dim];
            const int t0 = 16 * w + 4 * g;   // 4 consecutive keys, inside one 32-key pair
            const int pair = t0 & ~31, kin = t0 & 31;
            put4(Vts + dim * RLD + pair + vpos(kin), vv[f][0] + bv, vv[f][1] + bv, vv[f][2] + bv,
                 vv[f][3] + bv);
          }
        }
        __syncthreads();
        if (kc && blk + 1 < nblk) {   // this block's K and V^T for later blocks
          for (int e = tid; e < BT * (DM / 8); e += NT) {
            const int r = e / (DM / 8), c = e % (DM / 8);
            *reinterpret_cast<uint4*>(kc + int64_t(p0 + r) * DM + c * 8) =
                *reinterpret_cast<const uint4*>(Ks + r * RLD + c * 8);
          }
          for (int e = tid; e < DM * (BT / 8); e += NT) {
            const int r = e / (BT / 8), c = e % (BT / 8);
            *reinterpret_cast<uint4*>(vc + int64_t(r) * A.tpad + p0 + c * 8) =
                *reinterpret_cast<const uint4*>(Vts + r * RLD + c * 8);
          }
        }
        // ---- attention (per head), O into the Q rows of the wave's tokens
        const bool nm = A.unmasked != 0;
        if (A.dh == 64) {
          attend<64>(Qs, Ks, Vts, kc, vc, A.tpad, p0, 0, nv, nm);
        } else {
          attend<32>(Qs, Ks, Vts, kc, vc, A.tpad, p0, 0, nv, nm);
          attend<32>(Qs, Ks, Vts, kc, vc, A.tpad, p0, 32, nv, nm);
        }
        // ---- x += O W_o^T + b_o; LayerNorm 1 (the wave's own O rows: no barrier)
        {
          f32x4 o[4];
#pragma unroll
          for (int f = 0; f < 4; ++f) o[f] = f32x4{0.f, 0.f, 0.f, 0.f};
          wt_product<4>(o, Wo, RLD, Qs, RLD, DM);
#pragma unroll
          for (int f = 0; f < 4; ++f)
#pragma unroll
            for (int i = 0; i < 4; ++i) x[f][i] += o[f][i] + vec[V_BO + 16 * f + 4 * g + i];
          layer_norm(x, vec + V_LN1G, vec + V_LN1B);
          store_xb(Xb, x);
        }
        // ---- FFN: H = ReLU(x W_1^T + b_1); x += H W_2^T + b_2; LayerNorm 2
        {
          for (int f0 = 0; f0 < ffn; f0 += 16) {
            f32x4 hh[1] = {f32x4{0.f, 0.f, 0.f, 0.f}};
            wt_product<1>(hh, W1 + f0 * RLD, RLD, Xb, RLD, DM);
            const float* b1 = vec + V_B1 + f0 + 4 * g;
            put4(Hs + (16 * w + c16) * fld + f0 + 4 * g, fmaxf(hh[0][0] + b1[0], 0.f),
                 fmaxf(hh[0][1] + b1[1], 0.f), fmaxf(hh[0][2] + b1[2], 0.f),
                 fmaxf(hh[0][3] + b1[3], 0.f));
          }
          wave_lds_sync();
          f32x4 o[4];
#pragma unroll
          for (int f = 0; f < 4; ++f) o[f] = f32x4{0.f, 0.f, 0.f, 0.f};
          wt_product<4>(o, W2, fld, Hs, fld, ffn);
#pragma unroll
          for (int f = 0; f < 4; ++f)
#pragma unroll
            for (int i = 0; i < 4; ++i) x[f][i] += o[f][i] + vec[v_b2(ffn) + 16 * f + 4 * g + i];
          layer_norm(x, vec + v_ln2g(ffn), vec + v_ln2b(ffn));
          store_xb(Xb, x);
        }
      }
      // ---- head: last token's X, running max of X W_pool^T over valid tokens
      {
        const int p = p0 + 16 * w + c16;
        if (p == Tv - 1) {
#pragma unroll
          for (int f = 0; f < 4; ++f)
            *reinterpret_cast<float4*>(out + DM + 16 * f + 4 * g) =
                make_float4(x[f][0], x[f][1], x[f][2], x[f][3]);
        }
        f32x4 y[4];
#pragma unroll
        for (int f = 0; f < 4; ++f) y[f] = f32x4{0.f, 0.f, 0.f, 0.f};
        wt_product<4>(y, Wpool, RLD, Xb, RLD, DM);
        const bool valid = p < Tv;
#pragma unroll
        for (int f = 0; f < 4; ++f)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float m = valid ? y[f][i] : -__builtin_inff();
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, WAVE));
            y[f][i] = m;   // max over the wave's 16 tokens of feature 16 f + 4 g + i
          }
        if (c16 == 0) {
#pragma unroll
          for (int f = 0; f < 4; ++f)
#pragma unroll
            for (int i = 0; i < 4; ++i) pool[DM + w * DM + 16 * f + 4 * g + i] = y[f][i];
        }
      }
      __syncthreads();
      if (tid < DM) {
        float m = pool[tid];
#pragma unroll
        for (int v = 0; v < 4; ++v) m = fmaxf(m, pool[DM + v * DM + tid]);
        pool[tid] = m;
      }
    }
    __syncthreads();
    if (tid < DM) out[tid] = pool[tid] + A.b_pool[tid];
  }
}

}  // namespace sm

// ---------------------------------------------------------------- host side
namespace {
constexpr size_t SM_CACHE_BUDGET = size_t(1) << 30;   // K/V cache bytes at most
constexpr int SM_LDS_MAX = 160 * 1024;

sm::Args small_args(const tav2_weights& w, int d) {
  sm::Args a{};
  a.n_layers = w.n_layers;
  a.d = d;
  a.ffn = w.d_ffn;
  a.dh = w.d_model / w.n_heads;
  sm::plan_lds(a);
  return a;
}
int64_t small_tpad(int T) { return (T + sm::BT - 1) / sm::BT * sm::BT; }
size_t small_per_wg_cache(int T, const tav2_weights& w) {
  if (T <= sm::BT) return 0;
  return size_t(w.n_layers) * 2 * size_t(small_tpad(T)) * sm::DM * 2;
}
int small_grid(int64_t total, int T, const tav2_weights& w) {
  int cus = 256;
  int dev = 0;
  if (hipGetDevice(&dev) == hipSuccess) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        v > 0)
      cus = v;
  }
  int64_t g = total < cus ? total : cus;
  const size_t per = small_per_wg_cache(T, w);
  if (per) {
    const int64_t cap = int64_t(SM_CACHE_BUDGET / per);
    if (g > cap) g = cap > 0 ? cap : 1;
  }
  return int(g > 0 ? g : 1);
}
}  // namespace

bool encode_small_supported(int d, const tav2_weights& w) {
  if (w.d_model != sm::DM || w.n_layers > sm::MAX_LAYERS) return false;
  const int dh = w.d_model / w.n_heads;
  if (dh != 32 && dh != 64) return false;
  if (w.d_ffn % 32 || w.d_ffn > 256 || d % 32 || d > 256) return false;
  return small_args(w, d).lds_bytes <= SM_LDS_MAX;
}

size_t encode_small_workspace(int64_t total, int T, const tav2_weights& w) {
  return small_per_wg_cache(T, w) * size_t(small_grid(total, T, w));
}

hipError_t launch_encode_small(const TokenSource& src, const void* cand_emb, int64_t total,
                               const tav2_weights& w, float* out, void* ws, bool unmasked,
                               hipStream_t st) {
  if (total == 0) return hipSuccess;
  sm::Args a = small_args(w, src.d);
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
  a.total = total;
  a.tpad = int(small_tpad(src.T));
  a.out = out;
  a.unmasked = unmasked ? 1 : 0;
  const int grid = small_grid(total, src.T, w);
  const size_t per = small_per_wg_cache(src.T, w);
  if (per) {
    a.kcache = static_cast<bf16_t*>(ws);
    a.vcache = reinterpret_cast<bf16_t*>(static_cast<uint8_t*>(ws) + per / 2 * size_t(grid));
  }
  static std::atomic<bool> done[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64 && !done[dev].load(std::memory_order_acquire)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(sm::encoder_small_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, SM_LDS_MAX);
    if (e != hipSuccess) return e;
    done[dev].store(true, std::memory_order_release);
  }
  ProfScope prof("encoder_small", st);
  sm::encoder_small_kernel<<<unsigned(grid), sm::NT, size_t(a.lds_bytes), st>>>(a);
  return hipGetLastError();
}

}  // namespace tav2
