// Fused bf16 encoder, host side and small kernels: the candidate half of the
// input projection (cand_proj_kernel), the weight packing (pack_weights_kernel),
// and the launches of the per-candidate encoder kernel (encoder_fused_device.h).
#include "encoder_fused_device.h"

namespace tav2 {
namespace fz {

// ---------------------------------------------------------------- candidate half
// cvec[i] = c W_in[:, d:]^T + b_in for candidates c0 + i (the candidate's part of
// the Eq. 4 input projection, the same for every position of the candidate): one
// 32 x 32 MFMA tile (32 candidates x 32 features) per single-wave workgroup, every
// k-block's operands loaded up front (A: candidate rows, B: W_in rows, both 16
// bytes per lane straight from global memory).
constexpr int CP_KB = KIN / 16;   // k-blocks at most (d <= KIN)
__global__ __launch_bounds__(WAVE) void cand_proj_kernel(const bf16_t* __restrict__ cand,
                                                         const bf16_t* __restrict__ W_in,
                                                         const float* __restrict__ b_in, int d,
                                                         int64_t c0, int64_t nc,
                                                         float* __restrict__ cvec) {
  const int lane = threadIdx.x;
  const int hf = lane / 32, l32 = lane % 32;
  const int64_t nb = int64_t(blockIdx.x) * 32;    // first candidate of the tile
  const int f0 = blockIdx.y * 32;                 // first feature
  int64_t ci = nb + l32;
  ci = ci < nc ? ci : nc - 1;                     // rows past the chunk: clamped, not stored
  const bf16_t* arow = cand + (c0 + ci) * d + 8 * hf;
  const bf16_t* brow = W_in + int64_t(f0 + l32) * 2 * d + d + 8 * hf;
  const int nkb = (d + 15) / 16;
  bf16x8 a[CP_KB], b[CP_KB];
#pragma unroll
  for (int kb = 0; kb < CP_KB; ++kb) {
    const bool ok = kb < nkb && 16 * kb + 8 * hf < d;   // d is a multiple of 8
    a[kb] = ok ? as_bf16x8(*reinterpret_cast<const uint4*>(arow + 16 * kb)) : bf16x8{};
    b[kb] = ok ? as_bf16x8(*reinterpret_cast<const uint4*>(brow + 16 * kb)) : bf16x8{};
  }
  f32x16 acc = f32x16{};
#pragma unroll
  for (int kb = 0; kb < CP_KB; ++kb)
    if (kb < nkb) acc = mfma32(a[kb], b[kb], acc);
  const float bias = b_in[f0 + l32];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int64_t n = nb + 8 * (r / 4) + 4 * hf + (r % 4);
    if (n < nc) cvec[n * DM + f0 + l32] = acc[r] + bias;
  }
}

// ---------------------------------------------------------------- weight packing
// Rewrites a row-major [rows x K] bf16 matrix (row stride ld, columns >= kvalid
// read as zero) into MFMA-fragment order: fragment (rt, kb) is 1 KB at
// ((rt * nkb) + kb) * 512 elements, lane l holding row 32 rt + l % 32, columns
// 16 kb + 8 (l / 32) .. +7.  A bias job writes the bias k-block of a matrix
// instead: columns 0 and 1 of row r hold the bf16 value nearest to bias[r] and
// the bf16 value nearest to the remainder, the other columns zero.
struct PackJob {
  const bf16_t* src;
  bf16_t* dst;       // first fragment of the destination matrix
  int rows;          // destination rows (multiple of 32)
  int nkb;           // k-blocks per destination row
  int kb0, nkbj;     // k-blocks [kb0, kb0 + nkbj) of the destination written by this job
  int ld;            // source row stride (elements)
  int kvalid;        // job columns >= kvalid are zero
  int trans;         // destination (row r, job column k) = src[k * ld + r] instead of src[r * ld + k]
  const float* bias; // non-null: a bias job (one k-block)
};
constexpr int MAX_JOBS = 4 + 8 * MAX_LAYERS;
struct PackArgs {
  PackJob job[MAX_JOBS];
  int njobs;
};

// Grid: (workgroups of the largest job) x (jobs); blockIdx.y names the job, so its
// fields are scalar loads, and the workgroups past a smaller job's end return.
__global__ __launch_bounds__(256) void pack_weights_kernel(PackArgs P) {
  const PackJob& J = P.job[blockIdx.y];
  const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;   // piece within the job
  if (e >= int64_t(J.rows) * J.nkbj * 2) return;
  const int lane = int(e % 64);
  const int64_t frag = e / 64;
  const int rt = int(frag / J.nkbj), kbj = int(frag % J.nkbj);
  const int row = rt * 32 + lane % 32, col = kbj * 16 + 8 * (lane / 32);   // job column
  uint4 v = make_uint4(0, 0, 0, 0);
  if (J.bias) {
    if (lane < 32) {
      const float b = J.bias[row];
      const __bf16 hi = static_cast<__bf16>(b);
      const __bf16 lo = static_cast<__bf16>(b - static_cast<float>(hi));
      v.x = uint32_t(__builtin_bit_cast(uint16_t, hi)) | (uint32_t(__builtin_bit_cast(uint16_t, lo)) << 16);
    }
  } else if (!J.trans) {
    if (col < J.kvalid) v = *reinterpret_cast<const uint4*>(J.src + int64_t(row) * J.ld + col);
  } else {
    bf16_t x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = col + u < J.kvalid ? J.src[int64_t(col + u) * J.ld + row] : bf16_t(0);
    v = *reinterpret_cast<const uint4*>(x);
  }
  *reinterpret_cast<uint4*>(J.dst + ((int64_t(rt) * J.nkb + J.kb0 + kbj) * 64 + lane) * 8) = v;
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

// packed E_pos^T columns: every position of any 128-position block below max_pos
int pos_cols(const tav2_weights& w) { return (w.max_pos + fz::BT - 1) / fz::BT * fz::BT; }

size_t packed_bytes(const tav2_weights& w) {
  const size_t dm = fz::DM, ff = size_t(w.d_ffn);
  // W_qkv, W_o, W_1 with a bias k-block after their dm columns, W_2 after its ff
  const size_t per_layer = (3 * dm + dm + ff) * (dm + 16) + dm * (ff + 16);
  const size_t tables = dm * (fz::AT_COLS + size_t(pos_cols(w)));
  return align_up((dm * fz::KIN + dm * dm + size_t(w.n_layers) * per_layer + tables) * 2, 256);
}
}  // namespace

bool encode_fused_supported(int d, const tav2_weights& w) {
  const int dh = w.d_model / w.n_heads;
  return w.d_model == fz::DM && (dh == 32 || dh == 64) && w.d_ffn % fz::FC == 0 &&
         d % 32 == 0 && d <= fz::KIN && w.n_layers <= fz::MAX_LAYERS;
}

// Pack plan: fragment offsets of every packed matrix (into a) and the packing
// jobs (into P, with pk the destination), in one fixed layout that depends only
// on the weights' shape.
static void plan_pack(const tav2_weights& w, bf16_t* pk, fz::PackArgs& P, fz::Args& a,
                      int64_t& maxwg) {
  const int d = w.d_in, dm = fz::DM, ff = w.d_ffn;
  P = fz::PackArgs{};
  maxwg = 0;   // workgroups of the largest job
  size_t off = 0;
  // matrix m of rows x (16 nkb) columns at fragment `off`; add_cols fills k-blocks
  // [kb0, kb0 + nkbj) from a row-major (or transposed) source
  auto add_cols = [&](size_t mat, int rows, int nkb, int kb0, int nkbj, const void* srcm, int ld,
                      int kvalid, int trans) {
    fz::PackJob& J = P.job[P.njobs++];
    J.src = static_cast<const bf16_t*>(srcm);
    J.dst = pk + mat;
    J.rows = rows;
    J.nkb = nkb;
    J.kb0 = kb0;
    J.nkbj = nkbj;
    J.ld = ld;
    J.kvalid = kvalid;
    J.trans = trans;
    J.bias = nullptr;
    // 16-byte pieces: 2 per row per k-block, one per thread
    maxwg = std::max(maxwg, (int64_t(rows) * nkbj * 2 + 255) / 256);
  };
  // matrix of rows x K (row-major source), followed by a bias k-block if bias
  auto add = [&](const void* srcm, int rows, int K, int ld, int kvalid,
                 const float* bias = nullptr) {
    const size_t mat = off;
    const int nkb = K / 16 + (bias ? 1 : 0);
    add_cols(mat, rows, nkb, 0, K / 16, srcm, ld, kvalid, 0);
    if (bias) {
      add_cols(mat, rows, nkb, K / 16, 1, nullptr, 0, 0, 0);
      P.job[P.njobs - 1].bias = bias;
    }
    off += size_t(rows) * nkb * 16;
    return int(mat / 512);   // 512 bf16 per fragment; every matrix is whole fragments
  };
  a.pk_bytes = unsigned(packed_bytes(w));
  a.pk_in = add(w.W_in, dm, fz::KIN, 2 * d, d);
  a.pk_pool = add(w.W_pool, dm, dm, dm, dm);
  for (int i = 0; i < w.n_layers; ++i) {
    const tav2_layer& L = w.layers[i];
    a.pk[i].qkv = add(L.W_qkv, 3 * dm, dm, dm, dm, L.b_qkv);
    a.pk[i].o = add(L.W_o, dm, dm, dm, dm, L.b_o);
    a.pk[i].w1 = add(L.W_1, ff, dm, dm, dm, L.b_1);
    a.pk[i].w2 = add(L.W_2, dm, ff, ff, ff, L.b_2);
  }
  // side tables as [feature][row] matrices for the one-hot products of the input
  // encoding: E_act^T in columns 0..7, E_time^T in columns 16..79 (zero without
  // a time table); E_pos^T in its own matrix of pos_cols(w) columns
  a.pk_at = int(off / 512);
  add_cols(off, dm, fz::AT_COLS / 16, 0, 1, w.E_act, dm, fz::N_ACT, 1);
  add_cols(off, dm, fz::AT_COLS / 16, 1, 4, w.E_time ? w.E_time : w.E_act, dm,
           w.E_time ? fz::N_TIME : 0, 1);
  off += size_t(dm) * fz::AT_COLS;
  a.pk_pos = int(off / 512);
  a.pos_nkb = pos_cols(w) / 16;
  add_cols(off, dm, pos_cols(w) / 16, 0, pos_cols(w) / 16, w.E_pos, dm, w.max_pos, 1);
}

static hipError_t launch_pack(const tav2_weights& w, bf16_t* pk, hipStream_t st) {
  fz::PackArgs P;
  fz::Args a{};
  int64_t maxwg = 0;
  plan_pack(w, pk, P, a, maxwg);
  ProfScope prof("pack_weights", st);
  fz::pack_weights_kernel<<<dim3(unsigned(maxwg), unsigned(P.njobs)), 256, 0, st>>>(P);
  return hipGetLastError();
}

size_t encode_fused_packed_bytes(const tav2_weights& w) { return packed_bytes(w); }

hipError_t launch_encode_fused_pack(const tav2_weights& w, void* dst, hipStream_t st) {
  return launch_pack(w, static_cast<bf16_t*>(dst), st);
}

// Workspace: the packed weights (unless the weights bring them), the candidate
// half of the input projection per chunk, and the K / V cache per chunk.
size_t encode_fused_workspace(int64_t total, int T, const tav2_weights& w) {
  const size_t per = per_candidate_cache(T, w);
  const size_t chunk = size_t(fused_chunk(total, T, w));
  return (w.packed ? 0 : packed_bytes(w)) + align_up(chunk * fz::DM * 4, 256) + per * chunk;
}

hipError_t launch_encode_fused(const TokenSource& src, const void* cand_emb, int64_t total,
                               const tav2_weights& w, float* out, void* ws, bool unmasked,
                               hipStream_t st) {
  if (total == 0) return hipSuccess;
  const int d = src.d, ff = w.d_ffn;
  fz::Args a{};
  uint8_t* wsb = static_cast<uint8_t*>(ws);
  if (w.packed) {   // packed once by the caller (tav2_pack_weights)
    fz::PackArgs P;
    int64_t maxwg = 0;
    plan_pack(w, const_cast<bf16_t*>(static_cast<const bf16_t*>(w.packed)), P, a, maxwg);
    a.pkw = static_cast<const bf16_t*>(w.packed);
  } else {          // packed into the head of the workspace, every call
    bf16_t* pk = reinterpret_cast<bf16_t*>(wsb);
    fz::PackArgs P;
    int64_t maxwg = 0;
    plan_pack(w, pk, P, a, maxwg);
    a.pkw = pk;
    hipError_t e = launch_pack(w, pk, st);
    if (e != hipSuccess) return e;
    wsb += packed_bytes(w);
  }
  const size_t per = per_candidate_cache(src.T, w);
  const int64_t chunk = fused_chunk(total, src.T, w);
  float* cvec = reinterpret_cast<float*>(wsb);
  uint8_t* cache = reinterpret_cast<uint8_t*>(cvec) + align_up(size_t(chunk) * fz::DM * 4, 256);

  a.s = src;
  a.cand = static_cast<const bf16_t*>(cand_emb);
  a.W_in = static_cast<const bf16_t*>(w.W_in);
  a.b_in = w.b_in;
  a.E_act = static_cast<const bf16_t*>(w.E_act);
  a.E_time = static_cast<const bf16_t*>(w.E_time);
  a.E_pos = static_cast<const bf16_t*>(w.E_pos);
  a.b_pool = w.b_pool;
  for (int i = 0; i < w.n_layers; ++i) a.layers[i] = w.layers[i];
  a.n_layers = w.n_layers;
  a.d = d;
  a.dh = w.d_model / w.n_heads;
  a.ffn = ff;
  a.tpad = int(fused_tpad(src.T));
  a.out = out;
  a.cvec = cvec;
  for (int64_t c0 = 0; c0 < total; c0 += chunk) {
    const int64_t nc = total - c0 < chunk ? total - c0 : chunk;
    a.c0 = c0;
    {
      ProfScope prof("cand_proj", st);
      fz::cand_proj_kernel<<<dim3(unsigned(cdiv(nc, 32)), unsigned(fz::DM / 32)), WAVE, 0,
                             st>>>(a.cand, a.W_in, a.b_in, d, c0, nc, cvec);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    if (per) {
      a.kcache = reinterpret_cast<bf16_t*>(cache);
      a.vcache = reinterpret_cast<bf16_t*>(cache + per / 2 * size_t(chunk));
    }
    ProfScope prof("encoder_fused", st);
    hipError_t e;
    if (unmasked) {
      e = launch_encoder_fused_unmasked(a, unsigned(nc), st);
    } else {
      fz::encoder_fused_kernel<false><<<unsigned(nc), fz::NT, 0, st>>>(a);
      e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace tav2
