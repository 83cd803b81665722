// float32 encoder for small shapes: one workgroup per candidate keeps the
// whole candidate (tokens, Q/K/V, FFN hidden state) in LDS and runs Eq. 4's
// feature encoding, the causal post-LN layers and the linear + max-pool head
// (Sec. 3.2.2) with fp32 FMA.  Only the valid prefix of each candidate is
// computed: no valid position sees padding (under the causal mask, or in the
// unmasked mode, where a position sees the whole valid prefix).
#include "common.h"
#include "internal.h"
#include "token_source.h"

namespace tav2 {

constexpr int F32_MAX_LAYERS = 8;

struct EncF32Args {
  TokenSource s;
  const float* cand;
  int d, dm, H, ffn, n_layers;
  const float *W_in, *b_in, *E_act, *E_time, *E_pos, *W_pool, *b_pool;
  tav2_layer layers[F32_MAX_LAYERS];
  float* out;
  int unmasked;   // 1: every valid position sees every valid position
};

__device__ void layer_norm_rows(float* src, float* dst, int rows, int dm, const float* g,
                                const float* b) {
  const int lane = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
  for (int p = w; p < rows; p += 256 / WAVE) {
    float s = 0.f;
    for (int c = lane; c < dm; c += WAVE) s += src[p * dm + c];
    const float mu = wave_sum(s) / dm;
    float v = 0.f;
    for (int c = lane; c < dm; c += WAVE) {
      const float t = src[p * dm + c] - mu;
      v += t * t;
    }
    const float rs = rsqrtf(wave_sum(v) / dm + 1e-5f);
    for (int c = lane; c < dm; c += WAVE) dst[p * dm + c] = (src[p * dm + c] - mu) * rs * g[c] + b[c];
  }
}

__global__ __launch_bounds__(256) void encode_f32_kernel(EncF32Args a) {
  __shared__ float lds[F32_LDS_FLOATS];
  const int64_t n = blockIdx.x;
  const int tid = threadIdx.x;
  const int dm = a.dm, d = a.d, H = a.H, ff = a.ffn;
  const int dh = dm / H;
  const int Tv = token_valid_len(a.s, n);
  float* out = a.out + n * 2 * dm;
  if (Tv == 0) {
    for (int c = tid; c < 2 * dm; c += 256) out[c] = 0.f;
    return;
  }
  const int wide = 3 * dm > ff ? 3 * dm : ff;
  float* X = lds;                 // [Tv][dm]
  float* B1 = X + Tv * dm;        // [Tv][wide]
  float* B2 = B1 + Tv * wide;     // [Tv][dm]
  const float* cv = a.cand + n * d;

  // Eq. 4 with early fusion: [e_p ; e_c] W_in^T + b_in + side tables
  for (int e = tid; e < Tv * dm; e += 256) {
    const int p = e / dm, c = e % dm;
    const TokenRef t = resolve_token(a.s, n, p, d * 4);
    const float* ep = reinterpret_cast<const float*>(t.emb);
    const float* wr = a.W_in + int64_t(c) * 2 * d;
    float acc = a.b_in[c] + a.E_act[t.act * dm + c] + a.E_pos[p * dm + c];
    if (a.E_time) acc += a.E_time[t.time * dm + c];
    if (ep)
      for (int j = 0; j < d; ++j) acc = fmaf(ep[j], wr[j], acc);
    for (int j = 0; j < d; ++j) acc = fmaf(cv[j], wr[d + j], acc);
    X[e] = acc;
  }
  __syncthreads();

  const float scale = rsqrtf(float(dh));
  for (int li = 0; li < a.n_layers; ++li) {
    const tav2_layer& L = a.layers[li];
    const float* Wqkv = static_cast<const float*>(L.W_qkv);
    const float* Wo = static_cast<const float*>(L.W_o);
    const float* W1 = static_cast<const float*>(L.W_1);
    const float* W2 = static_cast<const float*>(L.W_2);
    for (int e = tid; e < Tv * 3 * dm; e += 256) {
      const int p = e / (3 * dm), c = e % (3 * dm);
      float acc = L.b_qkv[c];
      for (int j = 0; j < dm; ++j) acc = fmaf(X[p * dm + j], Wqkv[int64_t(c) * dm + j], acc);
      B1[p * wide + c] = acc;
    }
    __syncthreads();
    // attention (causal: keys j <= p; unmasked: every valid key): element (p, head, i)
    for (int e = tid; e < Tv * dm; e += 256) {
      const int p = e / dm, c = e % dm;
      const int hh = c / dh;
      const int jend = a.unmasked ? Tv - 1 : p;
      const float* q = B1 + p * wide + hh * dh;
      float m = -__builtin_inff();
      for (int j = 0; j <= jend; ++j) {
        const float* kj = B1 + j * wide + dm + hh * dh;
        float s = 0.f;
        for (int i = 0; i < dh; ++i) s = fmaf(q[i], kj[i], s);
        m = fmaxf(m, s * scale);
      }
      float l = 0.f, o = 0.f;
      for (int j = 0; j <= jend; ++j) {
        const float* kj = B1 + j * wide + dm + hh * dh;
        float s = 0.f;
        for (int i = 0; i < dh; ++i) s = fmaf(q[i], kj[i], s);
        const float pj = expf(s * scale - m);
        l += pj;
        o = fmaf(pj, B1[j * wide + 2 * dm + c], o);
      }
      B2[p * dm + c] = o / l;
    }
    __syncthreads();
    for (int e = tid; e < Tv * dm; e += 256) {
      const int p = e / dm, c = e % dm;
      float acc = X[p * dm + c] + L.b_o[c];
      for (int j = 0; j < dm; ++j) acc = fmaf(B2[p * dm + j], Wo[int64_t(c) * dm + j], acc);
      B1[p * dm + c] = acc;   // B1 reused as a [Tv][dm] scratch
    }
    __syncthreads();
    layer_norm_rows(B1, X, Tv, dm, L.ln1_g, L.ln1_b);
    __syncthreads();
    for (int e = tid; e < Tv * ff; e += 256) {
      const int p = e / ff, f = e % ff;
      float acc = L.b_1[f];
      for (int j = 0; j < dm; ++j) acc = fmaf(X[p * dm + j], W1[int64_t(f) * dm + j], acc);
      B1[p * wide + f] = fmaxf(acc, 0.f);
    }
    __syncthreads();
    for (int e = tid; e < Tv * dm; e += 256) {
      const int p = e / dm, c = e % dm;
      float acc = X[p * dm + c] + L.b_2[c];
      for (int f = 0; f < ff; ++f) acc = fmaf(B1[p * wide + f], W2[int64_t(c) * ff + f], acc);
      B2[p * dm + c] = acc;
    }
    __syncthreads();
    layer_norm_rows(B2, X, Tv, dm, L.ln2_g, L.ln2_b);
    __syncthreads();
  }

  for (int c = tid; c < dm; c += 256) {
    float mx = -__builtin_inff();
    for (int p = 0; p < Tv; ++p) {
      float acc = a.b_pool[c];
      for (int j = 0; j < dm; ++j) acc = fmaf(X[p * dm + j], a.W_pool[int64_t(c) * dm + j], acc);
      mx = fmaxf(mx, acc);
    }
    out[c] = mx;
    out[dm + c] = X[(Tv - 1) * dm + c];
  }
}

bool encode_f32_fits(int T, const tav2_weights& w) {
  if (T > F32_MAX_T || w.d_model > F32_MAX_DM || w.d_ffn > F32_MAX_FFN) return false;
  if (w.n_layers > F32_MAX_LAYERS) return false;
  const int wide = 3 * w.d_model > w.d_ffn ? 3 * w.d_model : w.d_ffn;
  return int64_t(T) * (2 * w.d_model + wide) <= F32_LDS_FLOATS;
}

hipError_t launch_encode_f32(const TokenSource& src, const void* cand_emb, int64_t total,
                             const tav2_weights& w, float* out, bool unmasked, hipStream_t st) {
  if (total == 0) return hipSuccess;
  EncF32Args a{};
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
  ProfScope prof("encode_f32", st);
  encode_f32_kernel<<<unsigned(total), 256, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace tav2
