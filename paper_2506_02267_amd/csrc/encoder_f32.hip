// float32 encoder for small shapes (T <= 64, d_model <= 128, FFN <= 512, d <=
// 256): one workgroup per candidate runs Eq. 4's feature encoding, the causal
// post-LN layers and the linear + max-pool head (Sec. 3.2.2) with fp32 FMA.
// Only the valid prefix of each candidate is computed: no valid position sees
// padding (under the causal mask, or in the unmasked mode, where a position sees
// the whole valid prefix).
//
// Every product is an LDS-resident GEMM Y[r][c] = sum_k A[r][k] B[k][c] with one
// register tile per thread: rows w + 4 i of wave w (one 16-byte broadcast read of
// A per 4 k), columns lane + 64 j (consecutive LDS words of B).  Weight matrices
// stream from memory in chunks of 16 k (coalesced along k) into a transposed LDS
// chunk; Q, V, the token rows and the FFN hidden chunk share one LDS region, K is
// kept transposed (keys as columns) for the score product, and the attention
// probabilities go through their own buffer into the P V product.  Rows of a
// product belong to one wave, so LayerNorm and softmax reduce across the lanes of
// a wave (DPP) on registers.
#include "common.h"
#include "internal.h"
#include "token_source.h"

#include <atomic>

namespace tav2 {
namespace f32e {

constexpr int NT = 256;
constexpr int NW = NT / WAVE;
constexpr int MAX_LAYERS = 8;
constexpr int KC_MAX = 32;           // k per staged weight chunk at most (16 or 32)
constexpr int NB = 128;              // output columns per weight product at most
constexpr int WS_LD = NB + 4;        // chunk row stride (== 4 mod 64: conflict-free stores)
constexpr int FC = 128;              // FFN hidden units per chunk
constexpr int SPT = KC_MAX * NB / NT;   // staged weight words per thread at most
constexpr int LDS_MAX = 163840 - F32_MAX_T * int(sizeof(void*));   // dynamic LDS bytes

struct Args {
  TokenSource s;
  const float* cand;
  int d, dm, H, ffn, n_layers;
  const float *W_in, *b_in, *E_act, *E_time, *E_pos, *W_pool, *b_pool;
  tav2_layer layers[MAX_LAYERS];
  float* out;
  int unmasked;   // 1: every valid position sees every valid position
  // LDS plan (floats)
  int ldx, ldq, ldk, ldp, lde, ldh;
  int kc_shift;   // log2 of k per weight chunk: the largest chunk the LDS has room for
  int o_x, o_q, o_k, o_p, o_w, o_cv, o_red, o_meta, lds_floats;
};

__host__ __device__ inline int round4(int x) { return (x + 3) / 4 * 4; }

__host__ inline void plan(Args& a, int T) {
  a.ldx = a.dm + 4;
  a.ldq = 2 * a.dm + 4;                   // [Q | V] rows
  a.ldk = T % 2 ? T + 2 : T + 1;          // K^T rows (odd: conflict-free transposed stores)
  a.ldp = round4(T) + 4;
  a.lde = a.d + 4;
  a.ldh = FC + 4;
  int off = 0;
  auto take = [&](int floats) {
    const int at = off;
    off += round4(floats);
    return at;
  };
  const int rows = round4(T);
  a.o_x = take(rows * a.ldx);
  int region = rows * a.ldq;
  region = region > rows * a.lde ? region : rows * a.lde;
  region = region > rows * a.ldh ? region : rows * a.ldh;
  a.o_q = take(region);
  a.o_k = take(a.dm * a.ldk);
  a.o_p = take(rows * a.ldp);
  a.o_cv = take(a.dm);
  a.o_red = take(NW * a.dm);
  a.o_meta = take(2 * F32_MAX_T);         // act, time of each row
  a.kc_shift = 4;
  for (int sh = 5; sh > 4; --sh)
    if ((off + (1 << sh) * WS_LD) * 4 <= LDS_MAX) {
      a.kc_shift = sh;
      break;
    }
  a.o_w = take((1 << a.kc_shift) * WS_LD);
  a.lds_floats = off;
}

// Wave-wide float sum / max, returned to every lane (DPP row shifts and row
// broadcasts; lane 63 ends with the result).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_f(float v, float id) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(id), __float_as_int(v), CTRL,
                                                    ROW_MASK, 0xf, false));
}
#define F32E_REDUCE(OP, ID)                       \
  v = OP(v, dpp_f<0x111, 0xf>(v, ID));            \
  v = OP(v, dpp_f<0x112, 0xf>(v, ID));            \
  v = OP(v, dpp_f<0x114, 0xf>(v, ID));            \
  v = OP(v, dpp_f<0x118, 0xf>(v, ID));            \
  v = OP(v, dpp_f<0x142, 0xa>(v, ID));            \
  v = OP(v, dpp_f<0x143, 0xc>(v, ID));            \
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
__device__ __forceinline__ float f_add(float a, float b) { return a + b; }
__device__ __forceinline__ float f_max(float a, float b) { return vmax(a, b); }
__device__ __forceinline__ float wave_sum_f(float v) { F32E_REDUCE(f_add, 0.f) }
__device__ __forceinline__ float wave_max_f(float v) { F32E_REDUCE(f_max, -__builtin_inff()) }
#undef F32E_REDUCE

template <int RI, int CJ>
__device__ __forceinline__ void zero(float (&acc)[RI][CJ]) {
#pragma unroll
  for (int i = 0; i < RI; ++i)
#pragma unroll
    for (int j = 0; j < CJ; ++j) acc[i][j] = 0.f;
}

// acc[i][j] += sum_{k < K} A[r][k] B[k][c] for rows r = w + 4 i (RI of them:
// those at or past `rows` repeat the last row and are discarded by the caller)
// and columns c = lane + 64 j, with A and B in LDS (B: row stride ldb; columns
// past the product's width read whatever follows in LDS and are discarded too).
// K is a multiple of 4 and A's rows 16-byte aligned.  No branch inside: every
// load of a k step is in flight at once.
template <int RI, int CJ>
__device__ __forceinline__ void gemm_lds(float (&acc)[RI][CJ], const float* A, int lda, int rows,
                                         int K, const float* B, int ldb) {
  const int w = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  const float* ar[RI];
#pragma unroll
  for (int i = 0; i < RI; ++i) {
    const int r = w + NW * i;
    ar[i] = A + (r < rows ? r : rows - 1) * lda;
  }
  const float* bc = B + lane;
  for (int k = 0; k < K; k += 4) {
    float b[4][CJ];
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int j = 0; j < CJ; ++j) b[e][j] = bc[(k + e) * ldb + WAVE * j];
    float4 av[RI];
#pragma unroll
    for (int i = 0; i < RI; ++i) av[i] = *reinterpret_cast<const float4*>(ar[i] + k);
#pragma unroll
    for (int i = 0; i < RI; ++i)
#pragma unroll
      for (int j = 0; j < CJ; ++j) {
        float t = acc[i][j];
        t = fmaf(av[i].x, b[0][j], t);
        t = fmaf(av[i].y, b[1][j], t);
        t = fmaf(av[i].z, b[2][j], t);
        t = fmaf(av[i].w, b[3][j], t);
        acc[i][j] = t;
      }
  }
}

// One staged chunk of a weight matrix W ([N][K] with row stride ldw, N <= NB) in
// registers: the thread's 16-byte pieces (4 consecutive k of one column) e = tid +
// NT q, column e / (kc / 4), k 4 (e % (kc / 4)).  K, ldw and the column offsets are
// multiples of 4, so a piece is all inside or all past K.
struct WChunk {
  float4 v[SPT / 4];
};
__device__ __forceinline__ void w_fetch(WChunk& st, const float* __restrict__ W, int ldw, int N,
                                        int K, int k0, int ks) {
  const int tid = threadIdx.x, ks4 = ks - 2, spt = ((1 << ks) * NB) / (4 * NT);
#pragma unroll
  for (int q = 0; q < SPT / 4; ++q) {
    const int e = tid + NT * q, c = e >> ks4, kk = (e & ((1 << ks4) - 1)) * 4;
    st.v[q] = (q < spt && c < N && k0 + kk < K)
                  ? *reinterpret_cast<const float4*>(W + c * ldw + k0 + kk)
                  : make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

// acc[i][j] += sum_{k < K} A[r][k] W[c][k]: A in LDS, W staged through the LDS
// chunk Ws, 2^ks k at a time (coalesced along k, stored transposed), each chunk's
// loads in flight while the one before is multiplied.  Starts with a barrier
// (earlier readers of Ws and of anything the caller writes before calling are
// done) and ends without one.
template <int RI, int CJ>
__device__ __forceinline__ void gemm_w(float (&acc)[RI][CJ], const float* A, int lda, int rows,
                                       int K, const float* __restrict__ W, int ldw, int N,
                                       float* Ws, int ks) {
  const int tid = threadIdx.x;
  WChunk st;
  w_fetch(st, W, ldw, N, K, 0, ks);
  const int kc_full = 1 << ks, spt = (kc_full * NB) / (4 * NT), ks4 = ks - 2;
  for (int k0 = 0; k0 < K; k0 += kc_full) {
    __syncthreads();
#pragma unroll
    for (int q = 0; q < SPT / 4; ++q) {
      const int e = tid + NT * q, c = e >> ks4, kk = (e & ((1 << ks4) - 1)) * 4;
      if (q < spt && c < N) {
        Ws[kk * WS_LD + c] = st.v[q].x;
        Ws[(kk + 1) * WS_LD + c] = st.v[q].y;
        Ws[(kk + 2) * WS_LD + c] = st.v[q].z;
        Ws[(kk + 3) * WS_LD + c] = st.v[q].w;
      }
    }
    __syncthreads();
    if (k0 + kc_full < K) w_fetch(st, W, ldw, N, K, k0 + kc_full, ks);
    const int kc = K - k0 < kc_full ? K - k0 : kc_full;
    gemm_lds<RI, CJ>(acc, A + k0, lda, rows, kc, Ws, WS_LD);
  }
}

// Post-LN sublayer end on registers: X[r] <- LayerNorm(acc[r] + bias + X[r]).
// The row's dm values sit in the lanes of one wave.
template <int RI>
__device__ __forceinline__ void add_norm(float (&acc)[RI][2], float* X, int ldx, int rows, int dm,
                                         const float* __restrict__ bias,
                                         const float* __restrict__ g,
                                         const float* __restrict__ be) {
  const int w = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  float bv[2], gv[2], ev[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int c = lane + WAVE * j;
    bv[j] = c < dm ? bias[c] : 0.f;
    gv[j] = c < dm ? g[c] : 0.f;
    ev[j] = c < dm ? be[c] : 0.f;
  }
  const float inv = 1.f / float(dm);
#pragma unroll
  for (int i = 0; i < RI; ++i) {
    const int r = w + NW * i;
    if (r < rows) {
      float y[2];
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int c = lane + WAVE * j;
        y[j] = c < dm ? acc[i][j] + bv[j] + X[r * ldx + c] : 0.f;
        s += y[j];
      }
      const float mu = wave_sum_f(s) * inv;
      float q = 0.f;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int c = lane + WAVE * j;
        const float t = c < dm ? y[j] - mu : 0.f;
        q = fmaf(t, t, q);
      }
      const float rs = rsqrtf(wave_sum_f(q) * inv + 1e-5f);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int c = lane + WAVE * j;
        if (c < dm) X[r * ldx + c] = (y[j] - mu) * rs * gv[j] + ev[j];
      }
    }
  }
}

// RI = rows per wave: positions up to 4 RI.
template <int RI>
__global__ __launch_bounds__(NT) void encode_f32_kernel(Args a) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int64_t n = blockIdx.x;
  const int tid = threadIdx.x, w = tid / WAVE, lane = tid % WAVE;
  const int dm = a.dm, d = a.d;
  const int dh = dm / a.H;
  const int Tv = token_valid_len(a.s, n);
  float* out = a.out + n * 2 * dm;
  if (Tv == 0) {
    for (int c = tid; c < 2 * dm; c += NT) out[c] = 0.f;
    return;
  }
  float* X = lds + a.o_x;
  float* QV = lds + a.o_q;   // [Q | V], the token rows, the FFN hidden chunk
  float* Kt = lds + a.o_k;
  float* P = lds + a.o_p;
  float* Ws = lds + a.o_w;
  float* cvec = lds + a.o_cv;
  float* red = lds + a.o_red;
  int* meta = reinterpret_cast<int*>(lds + a.o_meta);   // act [64], time [64]
  const float** rowp = nullptr;
  __shared__ const float* rows_ptr[F32_MAX_T];
  rowp = rows_ptr;

  // ---- Eq. 4 with early fusion: [e_p ; e_c] W_in^T + b_in + side tables
  if (tid < Tv) {
    const TokenRef t = resolve_token(a.s, n, tid, d * 4);
    rowp[tid] = reinterpret_cast<const float*>(t.emb);
    meta[tid] = t.act;
    meta[F32_MAX_T + tid] = t.time;
  }
  {   // candidate half, once: cvec[c] = b_in[c] + sum_k cand[k] W_in[c][d + k]
      // (wave w: columns w + 4 q, 8 at a time; lanes over k)
    const float* cv = a.cand + n * d;
    float cq[F32_MAX_D / WAVE];
#pragma unroll
    for (int t = 0; t < F32_MAX_D / WAVE; ++t) {
      const int k = lane + WAVE * t;
      cq[t] = k < d ? cv[k] : 0.f;
    }
    for (int c0 = w; c0 < dm; c0 += NW * 8) {
      float sv[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int c = c0 + NW * q;
        const float* wr = a.W_in + int64_t(c < dm ? c : 0) * 2 * d + d;
        float s = 0.f;
#pragma unroll
        for (int t = 0; t < F32_MAX_D / WAVE; ++t) {
          const int k = lane + WAVE * t;
          if (k < d) s = fmaf(cq[t], wr[k], s);
        }
        sv[q] = s;
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int c = c0 + NW * q;
        const float s = wave_sum_f(sv[q]);
        if (lane == 0 && c < dm) cvec[c] = s + a.b_in[c];
      }
    }
  }
  __syncthreads();
  for (int e0 = 0; e0 < Tv * d; e0 += NT * 8) {   // token rows into LDS (zeros for padding)
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int e = e0 + tid + NT * q;
      const int r = e / d, k = e % d;
      v[q] = 0.f;
      if (e < Tv * d && rowp[r]) v[q] = rowp[r][k];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int e = e0 + tid + NT * q;
      if (e < Tv * d) QV[(e / d) * a.lde + e % d] = v[q];
    }
  }
  {
    float acc[RI][2];
    zero<RI, 2>(acc);
    gemm_w<RI, 2>(acc, QV, a.lde, Tv, d, a.W_in, 2 * d, dm, Ws, a.kc_shift);
#pragma unroll
    for (int i = 0; i < RI; ++i) {
      const int r = w + NW * i;
      if (r < Tv) {
        const int act = meta[r], tm = meta[F32_MAX_T + r];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int c = lane + WAVE * j;
          if (c < dm) {
            float x = acc[i][j] + cvec[c] + a.E_act[act * dm + c] + a.E_pos[r * dm + c];
            if (a.E_time) x += a.E_time[tm * dm + c];
            X[r * a.ldx + c] = x;
          }
        }
      }
    }
  }

  const float scale = 1.f / sqrtf(float(dh));
  const int Kr = round4(Tv);   // keys of the P V product, zero-padded to a multiple of 4
  for (int li = 0; li < a.n_layers; ++li) {
    const tav2_layer& L = a.layers[li];
    const float* Wqkv = static_cast<const float*>(L.W_qkv);
    // ---- Q, K (transposed), V
    for (int part = 0; part < 3; ++part) {
      float acc[RI][2];
      zero<RI, 2>(acc);
      gemm_w<RI, 2>(acc, X, a.ldx, Tv, dm, Wqkv + int64_t(part) * dm * dm, dm, dm, Ws, a.kc_shift);
#pragma unroll
      for (int i = 0; i < RI; ++i) {
        const int r = w + NW * i;
        if (r < Tv) {
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const int c = lane + WAVE * j;
            if (c < dm) {
              const float y = acc[i][j] + L.b_qkv[part * dm + c];
              if (part == 1)
                Kt[c * a.ldk + r] = y;
              else
                QV[r * a.ldq + (part == 2 ? dm : 0) + c] = y;
            }
          }
        }
      }
    }
    for (int e = tid; e < (Kr - Tv) * dm; e += NT)   // V rows past the valid keys: zero
      QV[(Tv + e / dm) * a.ldq + dm + e % dm] = 0.f;
    // ---- attention, one head at a time; O_h overwrites Q_h
    for (int h = 0; h < a.H; ++h) {
      __syncthreads();   // Q, K, V complete; P free
      {
        float s[RI][1];
        zero<RI, 1>(s);
        gemm_lds<RI, 1>(s, QV + h * dh, a.ldq, Tv, dh, Kt + h * dh * a.ldk, a.ldk);
        float x[RI], m[RI], p[RI], l[RI];
#pragma unroll
        for (int i = 0; i < RI; ++i) {
          const int r = w + NW * i;
          const bool ok = lane < Tv && (a.unmasked || lane <= r);
          x[i] = ok ? s[i][0] * scale : -__builtin_inff();
          m[i] = wave_max_f(x[i]);   // finite: key 0 is valid for every row
        }
#pragma unroll
        for (int i = 0; i < RI; ++i) {
          p[i] = x[i] == -__builtin_inff() ? 0.f : expf(x[i] - m[i]);
          l[i] = wave_sum_f(p[i]);
        }
#pragma unroll
        for (int i = 0; i < RI; ++i) {
          const int r = w + NW * i;
          if (r < Tv && lane < Kr) P[r * a.ldp + lane] = p[i] / l[i];
        }
      }
      __syncthreads();
      {
        float o[RI][2];
        zero<RI, 2>(o);
        gemm_lds<RI, 2>(o, P, a.ldp, Tv, Kr, QV + dm + h * dh, a.ldq);
#pragma unroll
        for (int i = 0; i < RI; ++i) {
          const int r = w + NW * i;
          if (r < Tv) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
              const int c = lane + WAVE * j;
              if (c < dh) QV[r * a.ldq + h * dh + c] = o[i][j];
            }
          }
        }
      }
    }
    // ---- output projection + residual + LayerNorm 1
    {
      float acc[RI][2];
      zero<RI, 2>(acc);
      gemm_w<RI, 2>(acc, QV, a.ldq, Tv, dm, static_cast<const float*>(L.W_o), dm, dm, Ws, a.kc_shift);
      add_norm<RI>(acc, X, a.ldx, Tv, dm, L.b_o, L.ln1_g, L.ln1_b);
    }
    // ---- FFN in hidden chunks of FC units + residual + LayerNorm 2
    {
      float acc2[RI][2];
      zero<RI, 2>(acc2);
      for (int c0 = 0; c0 < a.ffn; c0 += FC) {
        const int nc = a.ffn - c0 < FC ? a.ffn - c0 : FC;
        float acc1[RI][2];
        zero<RI, 2>(acc1);
        gemm_w<RI, 2>(acc1, X, a.ldx, Tv, dm, static_cast<const float*>(L.W_1) + int64_t(c0) * dm, dm,
                      nc, Ws, a.kc_shift);
#pragma unroll
        for (int i = 0; i < RI; ++i) {
          const int r = w + NW * i;
          if (r < Tv) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
              const int c = lane + WAVE * j;
              if (c < nc) QV[r * a.ldh + c] = fmaxf(acc1[i][j] + L.b_1[c0 + c], 0.f);
            }
          }
        }
        gemm_w<RI, 2>(acc2, QV, a.ldh, Tv, nc, static_cast<const float*>(L.W_2) + c0, a.ffn, dm, Ws,
                      a.kc_shift);
      }
      __syncthreads();   // every wave is past its reads of X's rows
      add_norm<RI>(acc2, X, a.ldx, Tv, dm, L.b_2, L.ln2_g, L.ln2_b);
    }
  }

  // ---- head: max over valid rows of X W_pool^T + b_pool; X of the last row
  {
    float acc[RI][2];
    zero<RI, 2>(acc);
    gemm_w<RI, 2>(acc, X, a.ldx, Tv, dm, a.W_pool, dm, dm, Ws, a.kc_shift);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = lane + WAVE * j;
      float mx = -__builtin_inff();
#pragma unroll
      for (int i = 0; i < RI; ++i)
        if (w + NW * i < Tv) mx = fmaxf(mx, acc[i][j]);
      if (c < dm) red[w * dm + c] = mx;
    }
    __syncthreads();
    for (int c = tid; c < dm; c += NT) {
      float mx = red[c];
#pragma unroll
      for (int q = 1; q < NW; ++q) mx = fmaxf(mx, red[q * dm + c]);
      out[c] = mx + a.b_pool[c];
      out[dm + c] = X[(Tv - 1) * a.ldx + c];
    }
  }
}

}  // namespace f32e

bool encode_f32_fits(int T, const tav2_weights& w) {
  if (T < 1 || T > F32_MAX_T || w.d_model > F32_MAX_DM || w.d_ffn > F32_MAX_FFN) return false;
  if (w.n_layers > f32e::MAX_LAYERS) return false;
  // every product's k and row strides in whole 16-byte groups
  if (w.d_model % 4 || (w.d_model / w.n_heads) % 4 || w.d_ffn % 4) return false;
  f32e::Args a{};
  a.d = w.d_in;
  a.dm = w.d_model;
  f32e::plan(a, T);
  return a.lds_floats * 4 <= f32e::LDS_MAX;
}

hipError_t launch_encode_f32(const TokenSource& src, const void* cand_emb, int64_t total,
                             const tav2_weights& w, float* out, bool unmasked, hipStream_t st) {
  if (total == 0) return hipSuccess;
  f32e::Args a{};
  a.s = src;
  a.cand = static_cast<const float*>(cand_emb);
  a.d = src.d;
  a.dm = w.d_model;
  a.H = w.n_heads;
  a.ffn = w.d_ffn;
  a.n_layers = w.n_layers;
  a.W_in = static_cast<const float*>(w.W_in);
  a.b_in = w.b_in;
  a.E_act = static_cast<const float*>(w.E_act);
  a.E_time = static_cast<const float*>(w.E_time);
  a.E_pos = static_cast<const float*>(w.E_pos);
  a.W_pool = static_cast<const float*>(w.W_pool);
  a.b_pool = w.b_pool;
  for (int i = 0; i < w.n_layers; ++i) a.layers[i] = w.layers[i];
  a.out = out;
  a.unmasked = unmasked ? 1 : 0;
  f32e::plan(a, src.T);
  const size_t lds = size_t(a.lds_floats) * 4;
  // rows per wave: positions up to 16, 32, 48 or 64
  const int ri = (src.T + 15) / 16 * 4;
  const void* kernels[4] = {reinterpret_cast<const void*>(f32e::encode_f32_kernel<4>),
                            reinterpret_cast<const void*>(f32e::encode_f32_kernel<8>),
                            reinterpret_cast<const void*>(f32e::encode_f32_kernel<12>),
                            reinterpret_cast<const void*>(f32e::encode_f32_kernel<16>)};
  const int which = ri / 4 - 1;
  static std::atomic<bool> done[64][4] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64 || !done[dev][which].load(std::memory_order_acquire)) {
    e = hipFuncSetAttribute(kernels[which], hipFuncAttributeMaxDynamicSharedMemorySize,
                            f32e::LDS_MAX);
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < 64) done[dev][which].store(true, std::memory_order_release);
  }
  ProfScope prof("encode_f32", st);
  switch (which) {
    case 0: f32e::encode_f32_kernel<4><<<unsigned(total), f32e::NT, lds, st>>>(a); break;
    case 1: f32e::encode_f32_kernel<8><<<unsigned(total), f32e::NT, lds, st>>>(a); break;
    case 2: f32e::encode_f32_kernel<12><<<unsigned(total), f32e::NT, lds, st>>>(a); break;
    default: f32e::encode_f32_kernel<16><<<unsigned(total), f32e::NT, lds, st>>>(a); break;
  }
  return hipGetLastError();
}

}  // namespace tav2
