// bf16 encoder over the selected tokens (Eq. 4 feature encoding with early
// fusion, causal post-LN transformer layers and the linear + max-pool head of
// Sec. 3.2.2), on the 32x32x16 bf16 MFMA with fp32 accumulation.
//
// All candidates' tokens form one token matrix (M = candidates x T rows), so
// every per-token linear map is one GEMM against the shared weights:
//   X0   = gathered rows x W_in[:, :d]^T + (cand x W_in[:, d:]^T + b_in) + tables
//   QKV  = Xb W_qkv^T + b                       -> Q, K [cand][head][T][dh], V^T [cand][head][dh][Tp]
//   O    = causal softmax(Q K^T / sqrt(dh)) V   (flash-style, per candidate and head)
//   X    = LN1(X + O W_o^T + b_o)
//   H    = ReLU(Xb W_1^T + b_1)
//   X    = LN2(X + H W_2^T + b_2)
//   out  = [max_p (Xb W_pool^T + b_pool) ; X_last]
// The residual stream X stays fp32; Xb is its bf16 copy used as MFMA operand.
// Rows are processed in candidate chunks so the workspace stays bounded.
#include "common.h"
#include "internal.h"
#include "token_source.h"

namespace tav2 {

// ---------------------------------------------------------------- GEMM
// C[M, N] = A[M, K] B[N, K]^T.  Block tile 64 x 256, K step 32, 4 waves; wave w
// owns columns [64w, 64w + 64) as 2 x 2 MFMA tiles.  A and B are staged in LDS
// (double buffered); the fp32 tile is staged in LDS again for the epilogue.
constexpr int GM = 64, GN = 256, GK = 32, GPAD = 8;
constexpr int GLD = GK + GPAD;                    // bf16 elements per staged row
constexpr int CLD = GN + 4;                       // floats per epilogue row
constexpr int G_AB_BYTES = 2 * (GM + GN) * GLD * 2;
constexpr int G_C_BYTES = GM * CLD * 4;
constexpr int G_LDS = G_AB_BYTES > G_C_BYTES ? G_AB_BYTES : G_C_BYTES;

struct AMat {
  const bf16_t* p;
  int64_t lda;
  int64_t M;
  __device__ const bf16_t* row(int64_t m) const { return m < M ? p + m * lda : nullptr; }
};

// Token rows of candidates [c0, c0 + nc): row m = (c0 + m / T, m % T).
struct ATokens {
  TokenSource s;
  int64_t c0;
  int64_t M;
  __device__ const bf16_t* row(int64_t m) const {
    if (m >= M) return nullptr;
    const int64_t n = c0 + m / s.T;
    const int p = int(m % s.T);
    return reinterpret_cast<const bf16_t*>(resolve_token(s, n, p, s.d * 2).emb);
  }
};

template <class ALoad, class Epi>
__global__ __launch_bounds__(256) void gemm_kernel(ALoad al, const bf16_t* __restrict__ B,
                                                   int64_t ldb, int K, Epi epi) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[G_LDS];
  bf16_t* As = reinterpret_cast<bf16_t*>(smem);              // [2][GM][GLD]
  bf16_t* Bs = As + 2 * GM * GLD;                            // [2][GN][GLD]
  float* Cs = reinterpret_cast<float*>(smem);                // [GM][CLD] (after the loop)

  const int tid = threadIdx.x, lane = tid % WAVE, w = tid / WAVE;
  const int h = lane / 32, l32 = lane % 32;
  const int64_t m0 = int64_t(blockIdx.x) * GM;
  const int n0 = blockIdx.y * GN;

  // loader mapping: 16-byte piece (tid % 4) of A row tid / 4 and B rows tid / 4 + 64 q
  const int lr = tid / 4, lc = (tid % 4) * 8;
  const bf16_t* arow = al.row(m0 + lr);
  const bf16_t* brow[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) brow[q] = B + int64_t(n0 + lr + 64 * q) * ldb;

  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};

  const int nk = K / GK;
  uint4 ra = arow ? *reinterpret_cast<const uint4*>(arow + lc) : make_uint4(0, 0, 0, 0);
  uint4 rb0 = *reinterpret_cast<const uint4*>(brow[0] + lc);
  uint4 rb1 = *reinterpret_cast<const uint4*>(brow[1] + lc);
  uint4 rb2 = *reinterpret_cast<const uint4*>(brow[2] + lc);
  uint4 rb3 = *reinterpret_cast<const uint4*>(brow[3] + lc);
#define TAV2_SSTORE(buf)                                                        \
  do {                                                                          \
    *reinterpret_cast<uint4*>(As + ((buf) * GM + lr) * GLD + lc) = ra;          \
    *reinterpret_cast<uint4*>(Bs + ((buf) * GN + lr) * GLD + lc) = rb0;         \
    *reinterpret_cast<uint4*>(Bs + ((buf) * GN + lr + 64) * GLD + lc) = rb1;    \
    *reinterpret_cast<uint4*>(Bs + ((buf) * GN + lr + 128) * GLD + lc) = rb2;   \
    *reinterpret_cast<uint4*>(Bs + ((buf) * GN + lr + 192) * GLD + lc) = rb3;   \
  } while (0)
  TAV2_SSTORE(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) {
      const int k1 = (kt + 1) * GK + lc;
      ra = arow ? *reinterpret_cast<const uint4*>(arow + k1) : make_uint4(0, 0, 0, 0);
      rb0 = *reinterpret_cast<const uint4*>(brow[0] + k1);
      rb1 = *reinterpret_cast<const uint4*>(brow[1] + k1);
      rb2 = *reinterpret_cast<const uint4*>(brow[2] + k1);
      rb3 = *reinterpret_cast<const uint4*>(brow[3] + k1);
    }
#pragma unroll
    for (int kb = 0; kb < GK / 16; ++kb) {
      bf16x8 av[2], bv[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        av[t] = as_bf16x8(*reinterpret_cast<const uint4*>(
            As + (buf * GM + t * 32 + l32) * GLD + kb * 16 + 8 * h));
        bv[t] = as_bf16x8(*reinterpret_cast<const uint4*>(
            Bs + (buf * GN + 64 * w + t * 32 + l32) * GLD + kb * 16 + 8 * h));
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = mfma32(av[a], bv[b], acc[a][b]);
    }
    if (kt + 1 < nk) TAV2_SSTORE(buf ^ 1);
    __syncthreads();
  }
#undef TAV2_SSTORE

  // stage the fp32 tile: D register 4j + i of tile (a, b) is row a*32 + 8j + 4h + i,
  // column 64w + b*32 + l32
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int reg = 0; reg < 16; ++reg)
        Cs[(a * 32 + 8 * (reg / 4) + 4 * h + (reg % 4)) * CLD + 64 * w + b * 32 + l32] =
            acc[a][b][reg];
  __syncthreads();
  epi(Cs, m0, n0);
}

// ---------------------------------------------------------------- epilogues
// Every epilogue runs with all 256 threads over the staged 64 x 256 tile.

struct EpiBiasF32 {  // out[m, n] = C + bias[n]   (fp32)
  float* out;
  int64_t ldo;
  const float* bias;
  int64_t M;
  __device__ void operator()(const float* Cs, int64_t m0, int n0) const {
    for (int e = threadIdx.x; e < GM * GN; e += 256) {
      const int r = e / GN, c = e % GN;
      if (m0 + r < M) out[(m0 + r) * ldo + n0 + c] = Cs[r * CLD + c] + bias[n0 + c];
    }
  }
};

struct EpiReluBf16 {  // out[m, n] = bf16(ReLU(C + bias[n]))
  bf16_t* out;
  int64_t ldo;
  const float* bias;
  int64_t M;
  __device__ void operator()(const float* Cs, int64_t m0, int n0) const {
    for (int e = threadIdx.x; e < GM * GN / 2; e += 256) {
      const int r = e / (GN / 2), c = 2 * (e % (GN / 2));
      if (m0 + r >= M) continue;
      const float v0 = fmaxf(Cs[r * CLD + c] + bias[n0 + c], 0.f);
      const float v1 = fmaxf(Cs[r * CLD + c + 1] + bias[n0 + c + 1], 0.f);
      *reinterpret_cast<uint32_t*>(out + (m0 + r) * ldo + n0 + c) = pack2(v0, v1);
    }
  }
};

// Columns [0, dm) -> Q, [dm, 2dm) -> K, [2dm, 3dm) -> V^T; with dm == GN each
// column tile is exactly one of the three.
struct EpiQKV {
  bf16_t *Q, *K, *Vt;
  const float* bias;
  int T, Tp, H, dh;
  int64_t M;
  __device__ void operator()(const float* Cs, int64_t m0, int n0) const {
    const int part = n0 / GN;
    if (part < 2) {
      bf16_t* dst = part == 0 ? Q : K;
      for (int e = threadIdx.x; e < GM * GN / 2; e += 256) {
        const int r = e / (GN / 2), c = 2 * (e % (GN / 2));
        const int64_t m = m0 + r;
        if (m >= M) continue;
        const int64_t n = m / T;
        const int p = int(m % T);
        const int hh = c / dh, dim = c % dh;
        const float v0 = Cs[r * CLD + c] + bias[n0 + c];
        const float v1 = Cs[r * CLD + c + 1] + bias[n0 + c + 1];
        *reinterpret_cast<uint32_t*>(dst + ((n * H + hh) * int64_t(T) + p) * dh + dim) =
            pack2(v0, v1);
      }
    } else {
      for (int e = threadIdx.x; e < GM * GN; e += 256) {
        const int c = e / GM, r = e % GM;   // rows fastest: contiguous along p in V^T
        const int64_t m = m0 + r;
        if (m >= M) continue;
        const int64_t n = m / T;
        const int p = int(m % T);
        const int hh = c / dh, dim = c % dh;
        Vt[((n * H + hh) * int64_t(dh) + dim) * Tp + p] = f2bf(Cs[r * CLD + c] + bias[n0 + c]);
      }
    }
  }
};

// X[m, :] = LN(C + bias + X[m, :]) over the GN (= dm) columns; one wave per row.
// SITE distinguishes the attention sublayer (1) from the FFN sublayer (2) so the
// two instantiations are separate kernels in traces.
template <int SITE>
struct EpiResLN {
  float* X;
  bf16_t* Xb;
  const float* bias;
  const float* g;
  const float* b;
  int64_t M;
  __device__ void operator()(const float* Cs, int64_t m0, int) const {
    const int lane = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
    const int c = 4 * lane;
    const float4 bi = *reinterpret_cast<const float4*>(bias + c);
    const float4 gg = *reinterpret_cast<const float4*>(g + c);
    const float4 bb = *reinterpret_cast<const float4*>(b + c);
    for (int r = w; r < GM; r += 4) {
      const int64_t m = m0 + r;
      if (m >= M) break;
      float4 x = *reinterpret_cast<const float4*>(X + m * GN + c);
      const float4 cv = *reinterpret_cast<const float4*>(Cs + r * CLD + c);
      x.x += cv.x + bi.x;
      x.y += cv.y + bi.y;
      x.z += cv.z + bi.z;
      x.w += cv.w + bi.w;
      const float mu = wave_sum(x.x + x.y + x.z + x.w) * (1.f / GN);
      const float dx = x.x - mu, dy = x.y - mu, dz = x.z - mu, dw = x.w - mu;
      const float var = wave_sum(dx * dx + dy * dy + dz * dz + dw * dw) * (1.f / GN);
      const float rs = rsqrtf(var + 1e-5f);
      float4 y;
      y.x = dx * rs * gg.x + bb.x;
      y.y = dy * rs * gg.y + bb.y;
      y.z = dz * rs * gg.z + bb.z;
      y.w = dw * rs * gg.w + bb.w;
      *reinterpret_cast<float4*>(X + m * GN + c) = y;
      *reinterpret_cast<uint2*>(Xb + m * GN + c) = make_uint2(pack2(y.x, y.y), pack2(y.z, y.w));
    }
  }
};

// X0 = C + cvec[n] + E_act[a] + E_time[t] + E_pos[p]  (dm == GN)
struct EpiEmbed {
  float* X;
  bf16_t* Xb;
  const float* cvec;      // [nc, dm] for candidates c0 ..
  const bf16_t* E_act;
  const bf16_t* E_time;   // may be null
  const bf16_t* E_pos;
  TokenSource s;
  int64_t c0;
  int64_t M;
  __device__ void operator()(const float* Cs, int64_t m0, int) const {
    const int lane = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
    const int c = 4 * lane;
    for (int r = w; r < GM; r += 4) {
      const int64_t m = m0 + r;
      if (m >= M) break;
      const int64_t nl = m / s.T;
      const int p = int(m % s.T);
      const TokenRef t = resolve_token(s, c0 + nl, p, s.d * 2);
      const float4 cv = *reinterpret_cast<const float4*>(Cs + r * CLD + c);
      const float4 ce = *reinterpret_cast<const float4*>(cvec + nl * GN + c);
      float v[4] = {cv.x + ce.x, cv.y + ce.y, cv.z + ce.z, cv.w + ce.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        v[u] += bf2f(E_act[t.act * GN + c + u]) + bf2f(E_pos[p * GN + c + u]);
        if (E_time) v[u] += bf2f(E_time[t.time * GN + c + u]);
      }
      *reinterpret_cast<float4*>(X + m * GN + c) = make_float4(v[0], v[1], v[2], v[3]);
      *reinterpret_cast<uint2*>(Xb + m * GN + c) =
          make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
    }
  }
};

// running max of (C + b_pool) over each candidate's valid positions, as keys
struct EpiPool {
  uint32_t* keys;   // [nc, dm]
  const float* bias;
  TokenSource s;
  int64_t c0;
  int64_t M;
  __device__ void operator()(const float* Cs, int64_t m0, int) const {
    for (int e = threadIdx.x; e < GM * GN; e += 256) {
      const int r = e / GN, c = e % GN;
      const int64_t m = m0 + r;
      if (m >= M) continue;
      const int64_t nl = m / s.T;
      const int p = int(m % s.T);
      if (p >= token_valid_len(s, c0 + nl)) continue;
      atomicMax(keys + nl * GN + c, score_key(Cs[r * CLD + c] + bias[c]));
    }
  }
};

// ---------------------------------------------------------------- attention
// grid (ceil(T / 128), heads, candidates); wave w handles queries q0 .. q0 + 31.
// S^T = K Q^T puts keys on the MFMA rows and queries on lanes, so each lane owns
// one query's softmax state.  P^T is fed back as the B operand of O^T = V^T P^T
// directly from its accumulator registers; V^T is read with the matching key
// order (keys 4h..4h+3 then 8+4h..8+4h+3 of each 16-key block).
template <int DH>
__global__ __launch_bounds__(256) void attention_kernel(const bf16_t* __restrict__ Q,
                                                        const bf16_t* __restrict__ K,
                                                        const bf16_t* __restrict__ Vt,
                                                        bf16_t* __restrict__ O, int T, int Tp,
                                                        int H) {
  const int lane = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
  const int h = lane / 32, l32 = lane % 32;
  const int64_t n = blockIdx.z;
  const int head = blockIdx.y;
  const int q0 = blockIdx.x * 128 + w * 32;
  if (q0 >= T) return;
  const bf16_t* Qh = Q + (n * H + head) * int64_t(T) * DH;
  const bf16_t* Kh = K + (n * H + head) * int64_t(T) * DH;
  const bf16_t* Vh = Vt + (n * H + head) * int64_t(DH) * Tp;
  const int q = q0 + l32;
  const int qc = q < T ? q : T - 1;

  bf16x8 qf[DH / 16];
#pragma unroll
  for (int kb = 0; kb < DH / 16; ++kb)
    qf[kb] = as_bf16x8(*reinterpret_cast<const uint4*>(Qh + int64_t(qc) * DH + kb * 16 + 8 * h));

  f32x16 o[DH / 32];
#pragma unroll
  for (int t = 0; t < DH / 32; ++t) o[t] = f32x16{};
  float mrun = -__builtin_inff(), lrun = 0.f;
  const float sc = rsqrtf(float(DH)) * 1.4426950408889634f;
  const int qlast = (q0 + 31 < T ? q0 + 31 : T - 1);
  const int nkt = qlast / 32 + 1;

  for (int kt = 0; kt < nkt; ++kt) {
    int kr = kt * 32 + l32;
    kr = kr < T ? kr : T - 1;
    f32x16 s = f32x16{};
#pragma unroll
    for (int kb = 0; kb < DH / 16; ++kb) {
      const bf16x8 kf =
          as_bf16x8(*reinterpret_cast<const uint4*>(Kh + int64_t(kr) * DH + kb * 16 + 8 * h));
      s = mfma32(kf, qf[kb], s);
    }
    float mx = -__builtin_inff();
#pragma unroll
    for (int reg = 0; reg < 16; ++reg) {
      const int key = kt * 32 + 8 * (reg / 4) + 4 * h + (reg % 4);
      const float v = (key > q || key >= T) ? -__builtin_inff() : s[reg] * sc;
      s[reg] = v;
      mx = fmaxf(mx, v);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, WAVE));
    const float mnew = fmaxf(mrun, mx);
    const float alpha = exp2f(mrun - mnew);
    float psum = 0.f;
#pragma unroll
    for (int reg = 0; reg < 16; ++reg) {
      s[reg] = exp2f(s[reg] - mnew);
      psum += s[reg];
    }
    lrun = lrun * alpha + psum;
    mrun = mnew;
#pragma unroll
    for (int t = 0; t < DH / 32; ++t) o[t] *= alpha;
    const bool tail = kt * 32 + 32 > T;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      bf16x8 pb;
#pragma unroll
      for (int u = 0; u < 8; ++u) pb[u] = static_cast<__bf16>(s[8 * kb + u]);
      const int kbase = kt * 32 + kb * 16 + 4 * h;
#pragma unroll
      for (int t = 0; t < DH / 32; ++t) {
        const bf16_t* vr = Vh + int64_t(t * 32 + l32) * Tp + kbase;
        uint2 lo = *reinterpret_cast<const uint2*>(vr);
        uint2 hi = *reinterpret_cast<const uint2*>(vr + 8);
        if (tail) {
          // keys >= T hold no value: zero them so 0 * garbage cannot appear
          uint16_t e[8];
          __builtin_memcpy(e, &lo, 8);
          __builtin_memcpy(e + 4, &hi, 8);
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int key = kbase + (u < 4 ? u : 4 + u);
            if (key >= T) e[u] = 0;
          }
          __builtin_memcpy(&lo, e, 8);
          __builtin_memcpy(&hi, e + 4, 8);
        }
        o[t] = mfma32(as_bf16x8(lo, hi), pb, o[t]);
      }
    }
  }
  const float l = lrun + __shfl_xor(lrun, 32, WAVE);
  const float inv = 1.f / l;
  if (q >= T) return;
  const int dm = H * DH;
  bf16_t* orow = O + (n * T + q) * int64_t(dm) + head * DH;
#pragma unroll
  for (int t = 0; t < DH / 32; ++t)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int dim = t * 32 + 8 * j + 4 * h;
      *reinterpret_cast<uint2*>(orow + dim) =
          make_uint2(pack2(o[t][4 * j] * inv, o[t][4 * j + 1] * inv),
                     pack2(o[t][4 * j + 2] * inv, o[t][4 * j + 3] * inv));
    }
}

// ---------------------------------------------------------------- pool finalize
__global__ __launch_bounds__(256) void fill_u32_kernel(uint32_t* p, int64_t n, uint32_t v) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ __launch_bounds__(256) void pool_finalize_kernel(const uint32_t* __restrict__ keys,
                                                            const float* __restrict__ X,
                                                            TokenSource s, int64_t c0, int dm,
                                                            float* __restrict__ out) {
  const int64_t nl = blockIdx.x;
  const int64_t n = c0 + nl;
  const int valid = token_valid_len(s, n);
  for (int c = threadIdx.x; c < dm; c += 256) {
    float mx = 0.f, last = 0.f;
    if (valid > 0) {
      mx = key_score(keys[nl * dm + c]);
      last = X[(nl * s.T + valid - 1) * dm + c];
    }
    out[n * 2 * dm + c] = mx;
    out[n * 2 * dm + dm + c] = last;
  }
}

// ---------------------------------------------------------------- host side
namespace {

struct Layout {
  int64_t chunk;   // candidates per pass
  size_t cvec, X, Xb, Q, K, Vt, O, H, keys, total;
};

Layout make_layout(int64_t total, int T, const tav2_weights& w) {
  Layout L{};
  const int dm = w.d_model, ff = w.d_ffn;
  const int Tp = int(align_up(size_t(T), 32));
  int64_t chunk = (int64_t(1) << 20) / T;
  if (chunk < 1) chunk = 1;
  if (chunk > total) chunk = total > 0 ? total : 1;
  L.chunk = chunk;
  const size_t rows = size_t(chunk) * T;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  L.cvec = take(size_t(chunk) * dm * 4);
  L.X = take(rows * dm * 4);
  L.Xb = take(rows * dm * 2);
  L.Q = take(rows * dm * 2);
  L.K = take(rows * dm * 2);
  L.Vt = take(size_t(chunk) * dm * Tp * 2);
  L.O = take(rows * dm * 2);
  L.H = take(rows * ff * 2);
  L.keys = take(size_t(chunk) * dm * 4);
  L.total = off;
  return L;
}

template <class ALoad, class Epi>
hipError_t gemm(const char* site, ALoad al, int64_t M, const void* B, int64_t ldb, int N, int K,
                Epi epi, hipStream_t st) {
  if (M == 0) return hipSuccess;
  dim3 grid(unsigned(cdiv(M, GM)), unsigned(N / GN));
  ProfScope prof(site, st);
  gemm_kernel<ALoad, Epi><<<grid, 256, 0, st>>>(al, static_cast<const bf16_t*>(B), ldb, K, epi);
  return hipGetLastError();
}

}  // namespace

size_t encode_bf16_workspace(int64_t total, int T, const tav2_weights& w) {
  return make_layout(total, T, w).total;
}

hipError_t launch_encode_bf16(const TokenSource& src, const void* cand_emb, int64_t total,
                              const tav2_weights& w, float* out, void* ws, size_t,
                              hipStream_t st) {
  if (total == 0) return hipSuccess;
  const int T = src.T, d = src.d, dm = w.d_model, ff = w.d_ffn, H = w.n_heads;
  const int dh = dm / H;
  const int Tp = int(align_up(size_t(T), 32));
  const Layout Lo = make_layout(total, T, w);
  uint8_t* base = static_cast<uint8_t*>(ws);
  float* cvec = reinterpret_cast<float*>(base + Lo.cvec);
  float* X = reinterpret_cast<float*>(base + Lo.X);
  bf16_t* Xb = reinterpret_cast<bf16_t*>(base + Lo.Xb);
  bf16_t* Q = reinterpret_cast<bf16_t*>(base + Lo.Q);
  bf16_t* Kb = reinterpret_cast<bf16_t*>(base + Lo.K);
  bf16_t* Vt = reinterpret_cast<bf16_t*>(base + Lo.Vt);
  bf16_t* O = reinterpret_cast<bf16_t*>(base + Lo.O);
  bf16_t* Hb = reinterpret_cast<bf16_t*>(base + Lo.H);
  uint32_t* keys = reinterpret_cast<uint32_t*>(base + Lo.keys);
  const bf16_t* W_in = static_cast<const bf16_t*>(w.W_in);
  hipError_t e = hipSuccess;
#define TAV2_TRY(x)          \
  do {                       \
    e = (x);                 \
    if (e != hipSuccess) return e; \
  } while (0)

  for (int64_t c0 = 0; c0 < total; c0 += Lo.chunk) {
    const int64_t nc = (total - c0 < Lo.chunk) ? total - c0 : Lo.chunk;
    const int64_t M = nc * T;
    // candidate half of the fused input projection, once per candidate
    TAV2_TRY(gemm("gemm_cand", AMat{static_cast<const bf16_t*>(cand_emb) + c0 * d, d, nc}, nc, W_in + d,
                  2 * d, dm, d, EpiBiasF32{cvec, dm, w.b_in, nc}, st));
    // token half + side tables, with the gather fused into the A loads
    TAV2_TRY(gemm("gemm_embed", ATokens{src, c0, M}, M, W_in, 2 * d, dm, d,
                  EpiEmbed{X, Xb, cvec, static_cast<const bf16_t*>(w.E_act),
                           static_cast<const bf16_t*>(w.E_time),
                           static_cast<const bf16_t*>(w.E_pos), src, c0, M},
                  st));
    for (int li = 0; li < w.n_layers; ++li) {
      const tav2_layer& Lw = w.layers[li];
      TAV2_TRY(gemm("gemm_qkv", AMat{Xb, dm, M}, M, Lw.W_qkv, dm, 3 * dm, dm,
                    EpiQKV{Q, Kb, Vt, Lw.b_qkv, T, Tp, H, dh, M}, st));
      dim3 ag(unsigned(cdiv(T, 128)), unsigned(H), unsigned(nc));
      {
        ProfScope prof("attention", st);
        if (dh == 64)
          attention_kernel<64><<<ag, 256, 0, st>>>(Q, Kb, Vt, O, T, Tp, H);
        else
          attention_kernel<32><<<ag, 256, 0, st>>>(Q, Kb, Vt, O, T, Tp, H);
      }
      TAV2_TRY(hipGetLastError());
      TAV2_TRY(gemm("gemm_oproj_ln1", AMat{O, dm, M}, M, Lw.W_o, dm, dm, dm,
                    EpiResLN<1>{X, Xb, Lw.b_o, Lw.ln1_g, Lw.ln1_b, M}, st));
      TAV2_TRY(gemm("gemm_ffn1", AMat{Xb, dm, M}, M, Lw.W_1, dm, ff, dm, EpiReluBf16{Hb, ff, Lw.b_1, M}, st));
      TAV2_TRY(gemm("gemm_ffn2_ln2", AMat{Hb, ff, M}, M, Lw.W_2, ff, dm, ff,
                    EpiResLN<2>{X, Xb, Lw.b_2, Lw.ln2_g, Lw.ln2_b, M}, st));
    }
    {
      ProfScope prof("fill", st);
      fill_u32_kernel<<<unsigned(cdiv(nc * dm, 256)), 256, 0, st>>>(keys, nc * dm, 0u);
    }
    TAV2_TRY(hipGetLastError());
    TAV2_TRY(gemm("gemm_pool", AMat{Xb, dm, M}, M, w.W_pool, dm, dm, dm,
                  EpiPool{keys, w.b_pool, src, c0, M}, st));
    {
      ProfScope prof("pool_finalize", st);
      pool_finalize_kernel<<<unsigned(nc), 256, 0, st>>>(keys, X, src, c0, dm, out);
    }
    TAV2_TRY(hipGetLastError());
  }
#undef TAV2_TRY
  return hipSuccess;
}

}  // namespace tav2
