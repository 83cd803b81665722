// Single-kernel encoder for the paper's production encoder shape: d_model 64,
// one or two heads, a narrow FFN, a few layers (Sec. 3.2.2 'Transformer
// Encoder'; the fused transformer of Sec. 3.4.2 keeps every transformer weight
// on chip next to the activations).  One workgroup runs Eq. 4's feature
// encoding, every causal post-LN layer and the linear + max-pool head for one
// candidate at a time, with all layer weights resident in LDS (W_pool in
// registers).
//
// Layout of the work:
//  * The workgroup is persistent: it loads every weight on chip once and then
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
//    32-key pairs in registers, O^T += V^T P^T; keys of earlier blocks come
//    from the cache through a one-pair LDS stage filled by the whole workgroup.
//  * The next block's token rows are resolved during the current block and
//    loaded after its last attention, so Eq. 4 finds them in registers.
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
constexpr int SLD = 32 + 8;     // row stride (bf16) of a staged V^T pair
constexpr int MAX_LAYERS = 4;
constexpr int MAX_DK = 8;       // token width d <= 256: at most 8 k-steps of 32 (kernels for 1, 2, 4, 8)

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
  const uint8_t* packed;     // the weights' LDS image (tav2_pack_weights), or null
  int n_layers, d, dh, ffn;
  int64_t total;
  int tpad;                  // cache stride in positions (T rounded up to BT)
  bf16_t* kcache;            // [grid][layers][tpad][DM]
  bf16_t* vcache;            // [grid][layers][DM][tpad]
  float* out;                // [total, 2 DM]
  // LDS layout (bytes): the weights' image [0, wbytes), then the activations
  LayerW lw[MAX_LAYERS];
  int win, wbytes, xb, q, k, vt, h, kst, vst, cvec, pool, lds_bytes;
  int unmasked;
};

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
  a.wbytes = off;
  a.xb = take(BT * RLD * 2);
  a.q = take(BT * RLD * 2);    // Q, then the attention output O
  a.k = take(BT * RLD * 2);
  a.vt = take(DM * RLD * 2);   // V^T [dim][key]
  a.h = take(BT * fld * 2);
  a.kst = take(32 * RLD * 2);  // one 32-key pair of an earlier block: K rows
  a.vst = take(DM * SLD * 2);  //   and V^T rows
  a.cvec = take(DM * 4);
  a.pool = take(4 * DM * 4);   // one row of pooled maxima per wave
  a.lds_bytes = off;
}
// Offsets of the layer vectors inside lw.vec (floats).
constexpr int V_BQKV = 0, V_BO = 3 * DM, V_LN1G = 4 * DM, V_LN1B = 5 * DM, V_B1 = 6 * DM;
__host__ __device__ constexpr int v_b2(int ffn) { return 6 * DM + ffn; }
__host__ __device__ constexpr int v_ln2g(int ffn) { return 7 * DM + ffn; }
__host__ __device__ constexpr int v_ln2b(int ffn) { return 8 * DM + ffn; }

// Orders a wave's LDS writes before its later LDS reads of rows other lanes wrote
// (the wave's own token rows: no workgroup barrier is needed for them).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Copy a row-major [rows][cols] bf16 matrix into LDS rows of stride ld.
__device__ __forceinline__ void copy_matrix(bf16_t* dst, int ld, const bf16_t* src, int rows,
                                            int cols, int src_ld) {
  const int per = cols / 8;
  for (int e = threadIdx.x; e < rows * per; e += NT) {
    const int r = e / per, c = e % per;
    *reinterpret_cast<uint4*>(dst + r * ld + c * 8) =
        *reinterpret_cast<const uint4*>(src + int64_t(r) * src_ld + c * 8);
  }
}
__device__ __forceinline__ void copy_floats(float* dst, const float* src, int n) {
  for (int e = threadIdx.x; e < n; e += NT) dst[e] = src[e];
}

// Waits for the wave's vector memory loads, LDS-DMA included.
__device__ __forceinline__ void wait_vm_all() {
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0); expcnt and lgkmcnt unconstrained
}

// The layer weights and W_in's token half into LDS.  The packed image (wbytes, a
// multiple of 16) goes by LDS-DMA, asynchronously: 1 KB pieces, piece i issued by
// wave i mod 4, lane l moving bytes 16 l .. 16 l + 15 of it (lanes past the image
// re-read its last 16 bytes and drop them past wbytes, at the start of the
// activation area, which is written before it is read); the caller waits
// (wait_vm_all in every wave, then a workgroup barrier) before the first LDS read
// of a weight, so the loads of the first candidate's operands are in flight with
// it.  Without the image: matrix by matrix from the caller's layout, synchronously.
__device__ __forceinline__ void load_weights(const Args& A, uint8_t* smem) {
  if (A.packed) {
    const int lane = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
    const int npiece = (A.wbytes + 1023) / 1024;
    for (int i = w; i < npiece; i += NT / WAVE) {
      const int off = min(i * 1024 + 16 * lane, A.wbytes - 16);
      __builtin_amdgcn_global_load_lds(A.packed + off, smem + i * 1024, 16, 0, 0);
    }
    return;
  }
  const int ffn = A.ffn;
  for (int l = 0; l < A.n_layers; ++l) {
    const tav2_layer& L = A.layers[l];
    copy_matrix(reinterpret_cast<bf16_t*>(smem + A.lw[l].qkv), RLD,
                static_cast<const bf16_t*>(L.W_qkv), 3 * DM, DM, DM);
    copy_matrix(reinterpret_cast<bf16_t*>(smem + A.lw[l].o), RLD, static_cast<const bf16_t*>(L.W_o),
                DM, DM, DM);
    copy_matrix(reinterpret_cast<bf16_t*>(smem + A.lw[l].w1), RLD,
                static_cast<const bf16_t*>(L.W_1), ffn, DM, DM);
    copy_matrix(reinterpret_cast<bf16_t*>(smem + A.lw[l].w2), ffn + 8,
                static_cast<const bf16_t*>(L.W_2), DM, ffn, ffn);
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
  // token half of W_in: columns 0 .. d - 1 of [DM][2 d]
  copy_matrix(reinterpret_cast<bf16_t*>(smem + A.win), A.d + 8, A.W_in, DM, A.d, 2 * A.d);
}

// ---------------------------------------------------------------- LayerNorm
// x[f] holds X^T of the lane's token: features 16 f + 4 g + i.  Normalises over
// the 64 features (two passes: mean, then the centred squares).
__device__ __forceinline__ void layer_norm(f32x4 (&x)[4], const float* g, const float* b) {
  const int lane = threadIdx.x % WAVE, grp = lane / 16;
  float s = 0.f;
#pragma unroll
  for (int f = 0; f < 4; ++f) s += (x[f][0] + x[f][1]) + (x[f][2] + x[f][3]);
  s = xsum32(xsum16(s));
  const float mean = s * (1.f / DM);
  float v = 0.f;
#pragma unroll
  for (int f = 0; f < 4; ++f)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float c = x[f][i] - mean;
      v = fmaf(c, c, v);
    }
  v = xsum32(xsum16(v));
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
// The 4 bf16 of r added to v.
__device__ __forceinline__ void add4(float (&v)[4], uint2 r) {
  v[0] += __uint_as_float(r.x << 16);
  v[1] += __uint_as_float(r.x & 0xFFFF0000u);
  v[2] += __uint_as_float(r.y << 16);
  v[3] += __uint_as_float(r.y & 0xFFFF0000u);
}
// Operand fragments of the wave's own 16 token rows of a [BT][RLD] buffer over
// 64 features (identical for the A and the B operand: row / column l % 16, k = 8 (l / 16)).
__device__ __forceinline__ void own_rows(bf16x8 (&xf)[2], const bf16_t* buf) {
  const int lane = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
  const bf16_t* row = buf + (16 * w + lane % 16) * RLD + 8 * (lane / 16);
  xf[0] = frag(row);
  xf[1] = frag(row + 32);
}

// ------------------------------------------------------------ token inputs
// One lane's token for Eq. 4: its embedding fragments (k-steps of 32) and the 4
// side-table values of each feature tile; zeros for a padding position.
template <int NK>
struct TokLoad {
  bf16x8 e[NK];
  uint2 ea[4], ep[4], et[4];
};
__device__ __forceinline__ TokenRef lane_token(const Args& A, int64_t n, int p, int Tv) {
  TokenRef t{nullptr, 0, 0};
  if (p < Tv) t = resolve_token(A.s, n, p, A.s.codes ? A.d : A.d * 2);
  return t;
}
// 8 int8 codes as bf16 (exact: |q| <= 127).
__device__ __forceinline__ bf16x8 codes8(uint2 raw) {
  bf16x8 v;
#pragma unroll
  for (int j = 0; j < 8; ++j)
    v[j] = static_cast<__bf16>(float(int8_t(((j < 4 ? raw.x : raw.y) >> (8 * (j & 3))) & 0xFF)));
  return v;
}
template <int NK>
__device__ __forceinline__ void load_token(TokLoad<NK>& L, const TokenRef& t, int p, bool valid,
                                           const Args& A, int nk) {
  const int g = (threadIdx.x % WAVE) / 16;
  const bool have = valid && t.emb != nullptr;
#pragma unroll
  for (int k = 0; k < NK; ++k) {
    L.e[k] = bf16x8{};
    if (have && k < nk) {
      if (A.s.codes)   // int8 codes: dequantised after the product (Eq. 4 in the kernel)
        L.e[k] = codes8(*reinterpret_cast<const uint2*>(t.emb + 32 * k + 8 * g));
      else
        L.e[k] = frag(reinterpret_cast<const bf16_t*>(t.emb) + 32 * k + 8 * g);
    }
  }
#pragma unroll
  for (int f = 0; f < 4; ++f) {
    const int feat = 16 * f + 4 * g;
    L.ea[f] = L.ep[f] = L.et[f] = make_uint2(0u, 0u);
    if (valid) {
      L.ea[f] = *reinterpret_cast<const uint2*>(A.E_act + t.act * DM + feat);
      L.ep[f] = *reinterpret_cast<const uint2*>(A.E_pos + int64_t(p) * DM + feat);
      if (A.E_time) L.et[f] = *reinterpret_cast<const uint2*>(A.E_time + t.time * DM + feat);
    }
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
// Operands of one 32-key pair: K rows (A operand of S^T = K Q^T: rows keys,
// k = dims) and V^T rows (A operand of O^T += V^T P^T: rows dims, k = keys in
// vpos order).
template <int DH>
struct Pair {
  bf16x8 k[2][DH / 32];
  bf16x8 v[DH / 16];
};
template <int DH>
__device__ __forceinline__ void load_pair(Pair<DH>& f, const bf16_t* K, int kld, const bf16_t* Vt,
                                          int vld, int col0) {
  const int lane = threadIdx.x % WAVE;
  const int c16 = lane % 16, g = lane / 16;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int kb = 0; kb < DH / 32; ++kb)
      f.k[t][kb] = frag(K + (16 * t + c16) * kld + col0 + 32 * kb + 8 * g);
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) f.v[dt] = frag(Vt + (col0 + 16 * dt + c16) * vld + 8 * g);
}

// One 32-key pair.  Key j of the pair is visible to the lane's query iff j < lim
// (32: all).  Before the first visible key the running max is -inf: the
// exponents then use 0 as reference, which gives zero weights and a zero rescale
// of the (zero) sums.  exp2 is the hardware instruction (results below 2^-126
// flush to zero, far under the bf16 resolution of P).
template <int DH>
__device__ __forceinline__ void att_pair(Att<DH>& st, const Pair<DH>& f, int lim, float scale_l2) {
  const int g = (threadIdx.x % WAVE) / 16;
  f32x4 s[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < DH / 32; ++kb) a = mma(f.k[t][kb], st.qf[kb], a);
    s[t] = a;
  }
  // key 16 t + 4 g + i of the pair
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (4 * g + i >= lim) s[0][i] = -__builtin_inff();
    if (16 + 4 * g + i >= lim) s[1][i] = -__builtin_inff();
  }
  float mx = vmax(vmax(vmax(s[0][0], s[0][1]), vmax(s[0][2], s[0][3])),
                  vmax(vmax(s[1][0], s[1][1]), vmax(s[1][2], s[1][3])));
  mx = xmax32(xmax16(mx));
  const float mnew = vmax(st.m, mx * scale_l2);
  const float mref = mnew == -__builtin_inff() ? 0.f : mnew;
  const float alpha = __builtin_amdgcn_exp2f(st.m - mref);
  st.l *= alpha;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) st.o[dt] *= alpha;
  st.m = mnew;
  bf16x8 pb;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = __builtin_amdgcn_exp2f(fmaf(s[t][i], scale_l2, -mref));
      st.l += p;
      pb[4 * t + i] = static_cast<__bf16>(p);
    }
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) st.o[dt] = mma(f.v[dt], pb, st.o[dt]);
}

// Attention of the wave's 16 queries (block positions 16 w ..) for every head:
// the block's own keys 0 .. 16 w + 15 (causal; unmasked: 0 .. nkv - 1) from LDS,
// then the p0 keys of earlier blocks from the cache, one 32-key pair at a time
// staged in LDS by the whole workgroup (each key is read from the cache once per
// workgroup, not once per wave); the loads of the next two pairs are in flight
// while a pair is computed.  The stage alternates between Kst / Vst and the
// block's own K / V^T rows (free once every wave is past the block's own keys,
// i.e. after the first pair's barrier), so one barrier per pair orders both the
// stage's writes before its reads and its reads two pairs earlier before its
// rewrite.  Leaves O = softmax(S) V in the Q rows.
template <int DH>
__device__ __forceinline__ void attend(bf16_t* Qs, bf16_t* Ks, bf16_t* Vts,
                                       const bf16_t* kc, const bf16_t* vc, int tpad, int p0,
                                       int nkv, bool unmasked, bf16_t* Kst, bf16_t* Vst) {
  constexpr int NH = DM / DH;
  const int tid = threadIdx.x, lane = tid % WAVE, w = tid / WAVE;
  const int c16 = lane % 16, g = lane / 16;
  constexpr float scale_l2 = (DH == 64 ? 0.125f : 0.17677669529663688f) * 1.4426950408889634f;
  const int npair = p0 / 32;
  // staging: thread t moves 16 bytes of K (key t / 8) and of V^T (dim t / 4)
  const int kkey = tid / 8, kcol = 8 * (tid % 8), vdim = tid / 4, vcol = 8 * (tid % 4);
  auto fetch = [&](uint4& kr, uint4& vr, int c) {
    if (c < npair) {
      kr = *reinterpret_cast<const uint4*>(kc + int64_t(c * 32 + kkey) * DM + kcol);
      vr = *reinterpret_cast<const uint4*>(vc + int64_t(vdim) * tpad + c * 32 + vcol);
    }
  };
  uint4 k0 = make_uint4(0u, 0u, 0u, 0u), v0 = k0, k1 = k0, v1 = k0, k2 = k0, v2 = k0;
  fetch(k0, v0, 0);
  fetch(k1, v1, 1);
  Att<DH> st[NH];
#pragma unroll
  for (int h = 0; h < NH; ++h) {
#pragma unroll
    for (int kb = 0; kb < DH / 32; ++kb)
      st[h].qf[kb] = frag(Qs + (16 * w + c16) * RLD + h * DH + 32 * kb + 8 * g);
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) st[h].o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    st[h].m = -__builtin_inff();
    st[h].l = 0.f;
  }
  // own block: query 16 w + c16 sees keys <= itself (causal) or < nkv (unmasked)
  const int q = 16 * w + c16;
  const int kend = unmasked ? nkv : 16 * (w + 1);
  for (int k0p = 0; k0p < kend; k0p += 32) {
    const int lim = unmasked ? nkv - k0p : q + 1 - k0p;
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      Pair<DH> f;
      load_pair<DH>(f, Ks + k0p * RLD, RLD, Vts + k0p, RLD, h * DH);
      att_pair<DH>(st[h], f, lim, scale_l2);
    }
  }
  // earlier blocks: every key visible
  auto step = [&](const uint4& kr, const uint4& vr, uint4& kn, uint4& vn, int c) {
    bf16_t* ks = (c & 1) ? Ks : Kst;
    bf16_t* vs = (c & 1) ? Vts : Vst;
    *reinterpret_cast<uint4*>(ks + kkey * RLD + kcol) = kr;
    *reinterpret_cast<uint4*>(vs + vdim * SLD + vcol) = vr;
    __syncthreads();
    fetch(kn, vn, c + 2);
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      Pair<DH> f;
      load_pair<DH>(f, ks, RLD, vs, SLD, h * DH);
      att_pair<DH>(st[h], f, 32, scale_l2);
    }
  };
  for (int c = 0; c < npair; c += 3) {
    step(k0, v0, k2, v2, c);
    if (c + 1 < npair) step(k1, v1, k0, v0, c + 1);
    if (c + 2 < npair) step(k2, v2, k1, v1, c + 2);
  }
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    const float inv = 1.f / xsum32(xsum16(st[h].l));
    // O^T tile dt: lane holds query c16, dims 16 dt + 4 g + i
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt)
      put4(Qs + (16 * w + c16) * RLD + h * DH + 16 * dt + 4 * g, st[h].o[dt][0] * inv,
           st[h].o[dt][1] * inv, st[h].o[dt][2] * inv, st[h].o[dt][3] * inv);
  }
  wave_lds_sync();
}

// ---------------------------------------------------------------- the kernel
// NK: k-steps of 32 token features the kernel is built for (d / 32 <= NK).
template <int NK>
__global__ __launch_bounds__(NT) void encoder_small_kernel(Args A) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int tid = threadIdx.x, lane = tid % WAVE, w = tid / WAVE;
  const int c16 = lane % 16, g = lane / 16;
  const int d = A.d, ffn = A.ffn, fld = ffn + 8, nk = d / 32;
  load_weights(A, smem);
  bf16_t* Xb = reinterpret_cast<bf16_t*>(smem + A.xb);
  bf16_t* Qs = reinterpret_cast<bf16_t*>(smem + A.q);
  bf16_t* Ks = reinterpret_cast<bf16_t*>(smem + A.k);
  bf16_t* Vts = reinterpret_cast<bf16_t*>(smem + A.vt);
  bf16_t* Hs = reinterpret_cast<bf16_t*>(smem + A.h);
  float* cvec = reinterpret_cast<float*>(smem + A.cvec);
  float* pool = reinterpret_cast<float*>(smem + A.pool);
  const bf16_t* Win = reinterpret_cast<const bf16_t*>(smem + A.win);
  bf16_t* Kst = reinterpret_cast<bf16_t*>(smem + A.kst);
  bf16_t* Vst = reinterpret_cast<bf16_t*>(smem + A.vst);
  // W_pool as B operand fragments (rows 16 f + c16, k = 32 kb + 8 g), held in
  // registers for the workgroup's lifetime
  bf16x8 wpf[2][4];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int f = 0; f < 4; ++f) wpf[kb][f] = frag(A.W_pool + (16 * f + c16) * DM + 32 * kb + 8 * g);
  bf16_t* kc_wg = A.kcache ? A.kcache + int64_t(blockIdx.x) * A.n_layers * A.tpad * DM : nullptr;
  bf16_t* vc_wg = A.vcache ? A.vcache + int64_t(blockIdx.x) * A.n_layers * DM * A.tpad : nullptr;

  for (int64_t n = blockIdx.x; n < A.total; n += gridDim.x) {
    // the previous candidate is done with the buffers (no barrier before the
    // first: a barrier waits for the weights' LDS-DMA, and the first candidate's
    // metadata and operand loads go out while it is in flight)
    if (n != blockIdx.x) __syncthreads();
    const int Tv = token_valid_len(A.s, n);
    float* out = A.out + n * 2 * DM;
    if (Tv == 0) {
      for (int c = tid; c < 2 * DM; c += NT) out[c] = 0.f;
      continue;
    }
    // this lane's token of the first block (B operand column c16 of wave w)
    TokLoad<NK> tl;
    {
      const int p = 16 * w + c16;
      load_token(tl, lane_token(A, n, p, Tv), p, p < Tv, A, nk);
    }
    if (tid < DM) {   // candidate half of the input projection: W_in[:, d:] c + b_in
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
    }
    wait_vm_all();     // this wave's share of the weights is in LDS (first candidate)
    __syncthreads();
    // running max of X W_pool^T over the wave's valid tokens: lane holds features 16 f + c16
    float pmax[4] = {-__builtin_inff(), -__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
    const int nblk = (Tv + BT - 1) / BT;
    for (int blk = 0; blk < nblk; ++blk) {
      const int p0 = blk * BT;
      const int nv = Tv - p0 < BT ? Tv - p0 : BT;   // valid positions of the block
      const int p = p0 + 16 * w + c16;              // this lane's token (B operand column)
      // ---- Eq. 4: X0^T = W_in[:, :d] E^T + cvec + E_act + E_time + E_pos
      f32x4 x[4];
#pragma unroll
      for (int f = 0; f < 4; ++f) x[f] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < NK; ++k) {
        if (k < nk) {
#pragma unroll
          for (int f = 0; f < 4; ++f)
            x[f] = mma(frag(Win + (16 * f + c16) * (d + 8) + 32 * k + 8 * g), tl.e[k], x[f]);
        }
      }
      // D of the transposed product: lane holds token c16 of the wave's tile,
      // features 16 f + 4 g + i.  int8 codes: the product of the codes times the
      // scale 0.65 / 127 of their quantisation (Sec. 3.2.1) is that of the values.
      if (A.s.codes) {
#pragma unroll
        for (int f = 0; f < 4; ++f) x[f] *= 0.65f / 127.f;
      }
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        const int feat = 16 * f + 4 * g;
        float v[4] = {cvec[feat], cvec[feat + 1], cvec[feat + 2], cvec[feat + 3]};
        add4(v, tl.ea[f]);
        add4(v, tl.ep[f]);
        add4(v, tl.et[f]);
#pragma unroll
        for (int i = 0; i < 4; ++i) x[f][i] += v[i];
      }
      store_xb(Xb, x);
      // the next block's token: its row resolved now, its operands loaded after the
      // last layer's attention
      const TokenRef next = blk + 1 < nblk ? lane_token(A, n, p + BT, Tv) : TokenRef{nullptr, 0, 0};
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
        bf16x8 xf[2];
        own_rows(xf, Xb);
        f32x4 qk[8], vv[4];
#pragma unroll
        for (int f = 0; f < 8; ++f) qk[f] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int f = 0; f < 4; ++f) vv[f] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
          for (int f = 0; f < 8; ++f)
            qk[f] = mma(frag(Wqkv + (16 * f + c16) * RLD + 32 * kb + 8 * g), xf[kb], qk[f]);
#pragma unroll
          for (int f = 0; f < 4; ++f)
            vv[f] = mma(xf[kb], frag(Wqkv + (2 * DM + 16 * f + c16) * RLD + 32 * kb + 8 * g), vv[f]);
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
        if (A.dh == 64)
          attend<64>(Qs, Ks, Vts, kc, vc, A.tpad, p0, nv, nm, Kst, Vst);
        else
          attend<32>(Qs, Ks, Vts, kc, vc, A.tpad, p0, nv, nm, Kst, Vst);
        if (li == A.n_layers - 1 && blk + 1 < nblk)
          load_token(tl, next, p + BT, p + BT < Tv, A, nk);
        // ---- x += O W_o^T + b_o; LayerNorm 1 (the wave's own O rows: no barrier)
        {
          bf16x8 of[2];
          own_rows(of, Qs);
          f32x4 o[4];
#pragma unroll
          for (int f = 0; f < 4; ++f) o[f] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int f = 0; f < 4; ++f)
              o[f] = mma(frag(Wo + (16 * f + c16) * RLD + 32 * kb + 8 * g), of[kb], o[f]);
#pragma unroll
          for (int f = 0; f < 4; ++f)
#pragma unroll
            for (int i = 0; i < 4; ++i) x[f][i] += o[f][i] + vec[V_BO + 16 * f + 4 * g + i];
          layer_norm(x, vec + V_LN1G, vec + V_LN1B);
          store_xb(Xb, x);
        }
        // ---- FFN: H = ReLU(x W_1^T + b_1); x += H W_2^T + b_2; LayerNorm 2
        {
          bf16x8 hf[2];
          own_rows(hf, Xb);
          for (int f0 = 0; f0 < ffn; f0 += 16) {
            f32x4 hh = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
              hh = mma(frag(W1 + (f0 + c16) * RLD + 32 * kb + 8 * g), hf[kb], hh);
            const float* b1 = vec + V_B1 + f0 + 4 * g;
            put4(Hs + (16 * w + c16) * fld + f0 + 4 * g, fmaxf(hh[0] + b1[0], 0.f),
                 fmaxf(hh[1] + b1[1], 0.f), fmaxf(hh[2] + b1[2], 0.f), fmaxf(hh[3] + b1[3], 0.f));
          }
          wave_lds_sync();
          f32x4 o[4];
#pragma unroll
          for (int f = 0; f < 4; ++f) o[f] = f32x4{0.f, 0.f, 0.f, 0.f};
          const bf16_t* hrow = Hs + (16 * w + c16) * fld + 8 * g;
          for (int k0 = 0; k0 < ffn; k0 += 32) {
            const bf16x8 b = frag(hrow + k0);
#pragma unroll
            for (int f = 0; f < 4; ++f) o[f] = mma(frag(W2 + (16 * f + c16) * fld + k0 + 8 * g), b, o[f]);
          }
#pragma unroll
          for (int f = 0; f < 4; ++f)
#pragma unroll
            for (int i = 0; i < 4; ++i) x[f][i] += o[f][i] + vec[v_b2(ffn) + 16 * f + 4 * g + i];
          layer_norm(x, vec + v_ln2g(ffn), vec + v_ln2b(ffn));
          store_xb(Xb, x);
        }
      }
      // ---- head: the last token's X; the running max of X W_pool^T over valid tokens
      if (p == Tv - 1) {
#pragma unroll
        for (int f = 0; f < 4; ++f)
          *reinterpret_cast<float4*>(out + DM + 16 * f + 4 * g) =
              make_float4(x[f][0], x[f][1], x[f][2], x[f][3]);
      }
      {
        bf16x8 xf[2];
        own_rows(xf, Xb);
        f32x4 y[4];
#pragma unroll
        for (int f = 0; f < 4; ++f) y[f] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int f = 0; f < 4; ++f)
            y[f] = mma(xf[kb], wpf[kb][f], y[f]);
        // D[token][feature]: lane holds feature 16 f + c16 of tokens 16 w + 4 g + i
        const int t0 = p0 + 16 * w + 4 * g;
#pragma unroll
        for (int f = 0; f < 4; ++f) {
          float m = -__builtin_inff();
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (t0 + i < Tv) m = vmax(m, y[f][i]);
          pmax[f] = vmax(pmax[f], xmax32(xmax16(m)));
        }
      }
    }
    if (g == 0) {
#pragma unroll
      for (int f = 0; f < 4; ++f) pool[w * DM + 16 * f + c16] = pmax[f];
    }
    __syncthreads();
    if (tid < DM)
      out[tid] = vmax(vmax(pool[tid], pool[DM + tid]), vmax(pool[2 * DM + tid], pool[3 * DM + tid])) +
                 A.b_pool[tid];
  }
  wait_vm_all();   // no LDS-DMA outlives the workgroup (every candidate empty)
}

// The weights' LDS image: one workgroup per piece (a matrix or a vector).
struct Seg {
  const uint8_t* src;
  int dst, rows, units, src_ld, dst_ld;   // bytes; units of 16 bytes per row
};
constexpr int MAX_SEGS = 12 * MAX_LAYERS + 1;
struct PackArgs {
  Seg seg[MAX_SEGS];
  uint8_t* blob;
};
__global__ __launch_bounds__(256) void small_pack_kernel(PackArgs P) {
  const Seg s = P.seg[blockIdx.x];
  const int n = s.rows * s.units;
  for (int e = threadIdx.x; e < n; e += 256) {
    const int r = e / s.units, c = e % s.units;
    *reinterpret_cast<uint4*>(P.blob + s.dst + int64_t(r) * s.dst_ld + c * 16) =
        *reinterpret_cast<const uint4*>(s.src + int64_t(r) * s.src_ld + c * 16);
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
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// The pieces of the weights' LDS image: every layer matrix and vector and the
// token half of W_in.
int small_segments(const tav2_weights& w, int d, const sm::Args& a, sm::Seg* seg) {
  int n = 0;
  auto add = [&](const void* src, int dst, int rows, int row_bytes, int src_ld, int dst_ld) {
    seg[n++] = sm::Seg{static_cast<const uint8_t*>(src), dst, rows, row_bytes / 16, src_ld,
                       dst_ld};
  };
  constexpr int DM = sm::DM, RB = sm::RLD * 2;
  const int ffn = w.d_ffn, fb = (ffn + 8) * 2;
  for (int l = 0; l < w.n_layers; ++l) {
    const tav2_layer& L = w.layers[l];
    const int v = a.lw[l].vec;
    add(L.W_qkv, a.lw[l].qkv, 3 * DM, DM * 2, DM * 2, RB);
    add(L.W_o, a.lw[l].o, DM, DM * 2, DM * 2, RB);
    add(L.W_1, a.lw[l].w1, ffn, DM * 2, DM * 2, RB);
    add(L.W_2, a.lw[l].w2, DM, ffn * 2, ffn * 2, fb);
    add(L.b_qkv, v + sm::V_BQKV * 4, 1, 3 * DM * 4, 0, 0);
    add(L.b_o, v + sm::V_BO * 4, 1, DM * 4, 0, 0);
    add(L.ln1_g, v + sm::V_LN1G * 4, 1, DM * 4, 0, 0);
    add(L.ln1_b, v + sm::V_LN1B * 4, 1, DM * 4, 0, 0);
    add(L.b_1, v + sm::V_B1 * 4, 1, ffn * 4, 0, 0);
    add(L.b_2, v + sm::v_b2(ffn) * 4, 1, DM * 4, 0, 0);
    add(L.ln2_g, v + sm::v_ln2g(ffn) * 4, 1, DM * 4, 0, 0);
    add(L.ln2_b, v + sm::v_ln2b(ffn) * 4, 1, DM * 4, 0, 0);
  }
  add(w.W_in, a.win, DM, d * 2, 2 * d * 2, (d + 8) * 2);
  return n;
}
}  // namespace

bool encode_small_supported(int d, const tav2_weights& w) {
  if (w.d_model != sm::DM || w.n_layers > sm::MAX_LAYERS) return false;
  const int dh = w.d_model / w.n_heads;
  if (dh != 32 && dh != 64) return false;
  if (w.d_ffn % 32 || w.d_ffn > 256 || d % 32 || d > 32 * sm::MAX_DK) return false;
  return small_args(w, d).lds_bytes <= SM_LDS_MAX;
}

bool encode_small_aligned(const tav2_weights& w) {
  if (!aligned16(w.W_in) || !aligned16(w.W_pool) || (reinterpret_cast<uintptr_t>(w.E_act) & 7) ||
      (reinterpret_cast<uintptr_t>(w.E_pos) & 7) || (reinterpret_cast<uintptr_t>(w.E_time) & 7))
    return false;
  for (int l = 0; l < w.n_layers; ++l) {
    const tav2_layer& L = w.layers[l];
    if (!aligned16(L.W_qkv) || !aligned16(L.W_o) || !aligned16(L.W_1) || !aligned16(L.W_2))
      return false;
  }
  return true;
}

size_t encode_small_packed_bytes(const tav2_weights& w) {
  return size_t(small_args(w, w.d_in).wbytes);
}

hipError_t launch_encode_small_pack(const tav2_weights& w, void* packed, hipStream_t st) {
  const sm::Args a = small_args(w, w.d_in);
  sm::PackArgs P{};
  const int n = small_segments(w, w.d_in, a, P.seg);
  P.blob = static_cast<uint8_t*>(packed);
  ProfScope prof("pack_weights", st);
  sm::small_pack_kernel<<<unsigned(n), 256, 0, st>>>(P);
  return hipGetLastError();
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
  a.packed = static_cast<const uint8_t*>(w.packed);
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
  const int nk = src.d / 32;
  const int which = nk <= 1 ? 0 : nk <= 2 ? 1 : nk <= 4 ? 2 : 3;
  void (*const kernels[4])(sm::Args) = {sm::encoder_small_kernel<1>, sm::encoder_small_kernel<2>,
                                         sm::encoder_small_kernel<4>, sm::encoder_small_kernel<8>};
  static std::atomic<bool> done[64][4] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64 && !done[dev][which].load(std::memory_order_acquire)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernels[which]),
                            hipFuncAttributeMaxDynamicSharedMemorySize, SM_LDS_MAX);
    if (e != hipSuccess) return e;
    done[dev][which].store(true, std::memory_order_release);
  }
  ProfScope prof("encoder_small", st);
  hipLaunchKernelGGL(kernels[which], dim3(unsigned(grid)), dim3(sm::NT), size_t(a.lds_bytes), st, a);
  return hipGetLastError();
}

}  // namespace tav2
