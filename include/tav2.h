/*
 * tav2.h - C ABI of the lifelong-sequence NN-select + encode library (gfx950).
 *
 * The library computes, for every candidate item of a ranking request, the
 * serving hot path of TransAct V2's lifelong user-sequence module
 * (Xia et al., "TransAct V2: Lifelong User Action Sequence Modeling on
 * Pinterest Recommendation"):
 *   1. candidate-anchored nearest-neighbour search over the user's lifelong
 *      action sequence (Eq. 3, Sec. 3.2.2): dot-product scores of every action
 *      row against the candidate embedding and the top-k rows;
 *   2. the selected rows (plus, optionally, the kept most-recent real-time
 *      actions of Eq. 2) gathered into a token sequence;
 *   3. feature encoding with early fusion of the candidate embedding
 *      (Eq. 4), a causal transformer encoder, and a linear + max-pool head
 *      (Sec. 3.2.2, 'Transformer Encoder').
 * The request-level sequence is stored once per request and shared by all of
 * its candidates (the de-duplicated request-level format of Sec. 3.4.2,
 * 'Request Level De-duplication').
 *
 * Conventions shared by every entry point:
 *   - Pointers documented as "device" are HIP device pointers (or managed /
 *     host-pinned memory the GPU can read).  Pointers documented as "host" are
 *     read by the CPU during the call.  The caller owns every buffer, including
 *     outputs and the workspace; the library never allocates, frees or
 *     synchronises.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *     work is enqueued on it; the call returns before the GPU finishes.
 *   - Argument errors are detected on the host before anything is enqueued and
 *     return a negative status; nothing is launched in that case.  A launch
 *     failure returns TAV2_ERR_HIP.  Faults during execution surface at the
 *     caller's next synchronisation.
 *   - Calls are stateless; concurrent calls are safe when they use distinct
 *     outputs and workspaces.
 *   - Sequences are stored most-recent-first: row 0 of a request is its newest
 *     action.  Among equal scores, the more recent row (lower index) ranks
 *     first, so the selection order is the total order
 *     (score descending, row index ascending).  -0.0 and +0.0 are one score;
 *     reported zero scores are +0.0.
 *   - Matrices use the [out_features, in_features] row-major layout
 *     (y = x W^T + b).
 */
#ifndef TAV2_H
#define TAV2_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t tav2_status;
#define TAV2_OK               0
#define TAV2_ERR_NULL        -1   /* a required pointer is NULL */
#define TAV2_ERR_SHAPE       -2   /* a size is out of range or inconsistent */
#define TAV2_ERR_DTYPE       -3   /* unknown dtype, or dtypes that do not match */
#define TAV2_ERR_UNSUPPORTED -4   /* a valid request this build does not implement */
#define TAV2_ERR_WORKSPACE   -5   /* workspace NULL or smaller than the query says */
#define TAV2_ERR_HIP         -6   /* a HIP launch failed */
#define TAV2_ERR_TOO_LARGE   -7   /* the request needs more than the static scratch holds */

#define TAV2_F32  0   /* float32 storage and arithmetic */
#define TAV2_BF16 1   /* bfloat16 storage, fp32 accumulation */
#define TAV2_I8   2   /* int8 codes of the quantised sequence storage (Sec. 3.2.1): a
                         sequence dtype for the NN search (with bf16 candidates) and for
                         the d_model-64 encoder, which takes the dequantised values */

/* Attention mask of the encoder: the flags argument of tav2_encode and
 * tav2_select_encode. */
#define TAV2_MASK_CAUSAL 0u  /* position p attends to positions 0..p, the causal mask the
                                encoder applies (Sec. 3.2.2, 'Transformer Encoder'); default */
#define TAV2_MASK_NONE   1u  /* every valid position attends to every valid position: the
                                unmasked setting of the paper's comparison of its fused
                                transformer with FlashAttention-2 (Appendix B).  For tests and
                                comparisons; bf16 encoders take it only when T <= 128 */

#define TAV2_K_MAX     1024  /* largest k of the NN search */
#define TAV2_T_MAX     2048  /* largest encoder sequence (all token parts) */
#define TAV2_N_ACT        8  /* action types: values in [0, 8) */
#define TAV2_N_TIME      64  /* time buckets: values in [0, 64) */

/*
 * A de-duplicated request-level action sequence batch (Sec. 3.4.2, 'Request
 * Level De-duplication'): the rows of all R requests are stored once; request r
 * owns rows [offset[r], offset[r] + len[r]).  Packed (offset = prefix sum of
 * len) and fixed-stride padded layouts are both valid.
 */
typedef struct tav2_seq {
  const void*    emb;          /* device [rows, d], dtype; values finite */
  const uint8_t* action_type;  /* device [rows], values in [0, 8) */
  const uint8_t* time_bucket;  /* device [rows], values in [0, 64), or NULL (no time feature) */
  const int64_t* offset;       /* device [R]: first row of each request */
  const int32_t* len;          /* device [R]: rows of each request, 0 <= len[r] <= max_len */
  int32_t num_requests;        /* R >= 0 */
  int32_t d;                   /* embedding width, multiple of 16, 16..512 */
  int32_t dtype;               /* TAV2_F32, TAV2_BF16, or TAV2_I8 (tav2_nn_select only) */
  int32_t max_len;             /* host-side bound: len[r] <= max_len for every r */
} tav2_seq;

/* The candidate items of the same R requests, stored contiguously by request. */
typedef struct tav2_cands {
  const void*    emb;          /* device [total, d], same dtype and d as the sequence
                                  (bf16 when the sequence is TAV2_I8) */
  const int64_t* offset;       /* device [R + 1]: candidates of request r are
                                  [offset[r], offset[r+1]); offset[0] = 0, offset[R] = total */
  int64_t total;               /* host: number of candidates (>= 0) */
  int32_t max_count;           /* host-side bound: offset[r+1]-offset[r] <= max_count */
  int32_t reserved;            /* set to 0 */
} tav2_cands;

/* Explicit gathered tokens in encoder order (what tav2_gather writes). */
typedef struct tav2_tokens {
  const void*    emb;          /* device [total, T, d], dtype */
  const uint8_t* action_type;  /* device [total, T] */
  const uint8_t* time_bucket;  /* device [total, T], or NULL when the weights have no time table */
  const int32_t* valid_len;    /* device [total]: tokens [0, valid_len) are real, 0 <= valid_len <= T */
  int64_t total;               /* host: number of candidates */
  int32_t T;                   /* positions per candidate, 1..TAV2_T_MAX */
  int32_t d;                   /* token embedding width */
  int32_t dtype;               /* TAV2_F32 or TAV2_BF16 */
  int32_t reserved;            /* set to 0 */
} tav2_tokens;

/* One post-LayerNorm encoder layer.  Matrices in the weights' dtype,
 * vectors (biases, LayerNorm gain/offset) always float32.  Device pointers. */
typedef struct tav2_layer {
  const void*  W_qkv;  const float* b_qkv;   /* [3 dm, dm]: rows q | k | v; [3 dm] */
  const void*  W_o;    const float* b_o;     /* [dm, dm]; [dm] */
  const float* ln1_g;  const float* ln1_b;   /* [dm] */
  const void*  W_1;    const float* b_1;     /* [d_ffn, dm]; [d_ffn] */
  const void*  W_2;    const float* b_2;     /* [dm, d_ffn]; [dm] */
  const float* ln2_g;  const float* ln2_b;   /* [dm] */
} tav2_layer;

/*
 * Encoder weights.  Feature encoding (Eq. 4 with early fusion): the token's
 * embedding e_p and the candidate's e_c are concatenated and projected,
 *   x_p = [e_p ; e_c] W_in^T + b_in + E_act[a_p] + E_time[t_p] + E_pos[p],
 * which is Eq. 4 exactly when dm = 2 d and W_in = I.  Each layer:
 *   X <- LN1(X + MHA_causal(X) W_o^T + b_o);  X <- LN2(X + ReLU(X W_1^T + b_1) W_2^T + b_2)
 * with per-head scale 1/sqrt(dm / n_heads) and LayerNorm eps 1e-5.
 */
typedef struct tav2_weights {
  int32_t d_in;                /* token / candidate embedding width d */
  int32_t d_model;             /* dm */
  int32_t n_heads;             /* dm % n_heads == 0 */
  int32_t d_ffn;
  int32_t n_layers;            /* >= 1 */
  int32_t max_pos;             /* rows of E_pos, >= the encoder sequence length T */
  int32_t dtype;               /* TAV2_F32 or TAV2_BF16 */
  int32_t reserved;            /* set to 0 */
  const void*  W_in;  const float* b_in;     /* device [dm, 2 d] (token columns first); [dm] */
  const void*  E_act;                        /* device [8, dm] */
  const void*  E_time;                       /* device [64, dm], or NULL (no time feature) */
  const void*  E_pos;                        /* device [max_pos, dm] */
  const tav2_layer* layers;                  /* HOST array of n_layers layer records */
  const void*  W_pool; const float* b_pool;  /* device [dm, dm]; [dm] */
  const void*  packed;         /* device: these weights as tav2_pack_weights wrote them, or
                                  NULL (then every call packs them into its workspace;
                                  dm 64: every call reads them as given) */
  uint64_t     packed_bytes;   /* size of `packed` (ignored when it is NULL) */
} tav2_weights;

/* Human-readable text of a status code (static storage). */
const char* tav2_status_string(tav2_status s);

/* Version of the library's ABI (monotonically increasing). */
int32_t tav2_abi_version(void);

/*
 * NN search (Eq. 3): for every candidate n of request r, the k rows i of
 * request r with the largest score s[n, i] = <emb[offset[r] + i], cand[n]>,
 * in the order (score desc, row asc).
 *   out_idx   device [total, k] int32: row index within the request; -1 when
 *             k > len[r] (positions >= len[r]).
 *   out_score device [total, k] float32: the scores (fp32 accumulation; exact
 *             whenever the fp32 sum is exact), -inf in padded positions.
 * A TAV2_I8 sequence holds int8 codes q (Sec. 3.2.1); each row is dequantised and
 * L2-normalised before the dot product (Sec. 3.4.2, fused sequence
 * dequantisation), all inside the score kernel: the dequantisation scale cancels
 * and s[n, i] = <q_i, cand[n]> / |q_i| (0 for an all-zero row), from the fp32 dot
 * product and the exact sum of squares with one correctly rounded square root
 * and one correctly rounded division.  tav2_gather, tav2_encode and
 * tav2_select_encode return TAV2_ERR_UNSUPPORTED for TAV2_I8.
 *   ws        device workspace of at least tav2_nn_select_workspace() bytes,
 *             256-byte aligned.
 * Errors: TAV2_ERR_NULL, TAV2_ERR_SHAPE (k < 1 or k > TAV2_K_MAX, d, counts),
 * TAV2_ERR_DTYPE, TAV2_ERR_WORKSPACE, TAV2_ERR_HIP.
 */
size_t tav2_nn_select_workspace(const tav2_seq* seq, const tav2_cands* cands, int32_t k);
tav2_status tav2_nn_select(const tav2_seq* seq, const tav2_cands* cands, int32_t k,
                           int32_t* out_idx, float* out_score,
                           void* ws, size_t ws_bytes, void* stream);

/*
 * tav2_nn_select without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP-graph capture, serving loops and
 * harnesses that forbid allocation).  The search's working memory is a static
 * device buffer of TAV2_SCRATCH_BYTES inside the library (one per GPU, held from
 * the first call on that GPU until the process ends; no allocation on any
 * call).  Requests whose workspace (tav2_nn_select_workspace) exceeds it return
 * TAV2_ERR_TOO_LARGE before anything is launched.  Every call on one GPU shares
 * that GPU's buffer, so calls that overlap in time on one GPU (concurrent
 * streams or host threads) race and must be serialised by the caller; the
 * kernels initialise what they read, so no clearing is needed between calls.
 * Arguments, outputs and the other errors as for tav2_nn_select.
 */
#define TAV2_SCRATCH_BYTES ((size_t)64 << 20)
size_t tav2_scratch_bytes(void);
tav2_status tav2_nn_select_noalloc(const tav2_seq* seq, const tav2_cands* cands, int32_t k,
                                   int32_t* out_idx, float* out_score, void* stream);

/*
 * Token assembly for the encoder (Eq. 2 restricted to NN(S_LL, c) and the kept
 * most-recent real-time actions S_RT[:r]).  For candidate n with T_LL valid
 * entries in idx[n] (entries >= 0, rank order as tav2_nn_select writes them),
 * position p < T_LL holds sequence row idx[n][T_LL - 1 - p] (ascending score,
 * best match last, as Eq. 3's ascending argsort returns them); positions
 * T_LL .. T_LL + len_rt[r] - 1 hold the request's real-time rows oldest first;
 * later positions are zero.
 *   rt        NULL, or a real-time sequence batch with the same R, d and dtype.
 *   tok_*     device outputs [total, T, d], [total, T], [total, T]
 *             (tok_time may be NULL), with T = k + (rt ? rt->max_len : 0).
 *   valid_len device [total] int32 output.
 * Errors: TAV2_ERR_NULL, TAV2_ERR_SHAPE, TAV2_ERR_DTYPE, TAV2_ERR_HIP.
 */
tav2_status tav2_gather(const tav2_seq* seq, const tav2_seq* rt, const tav2_cands* cands,
                        const int32_t* idx, int32_t k,
                        void* tok_emb, uint8_t* tok_act, uint8_t* tok_time,
                        int32_t* valid_len, void* stream);

/*
 * Packed encoder weights: the bf16 encoder reads its matrices and side tables in
 * its own fragment order (dm 64: the image of every layer weight, W_in's token
 * half and W_pool as the kernel holds them in LDS, which it then loads with one
 * contiguous copy).  tav2_pack_weights writes that form once into a
 * caller-owned device buffer of tav2_pack_weights_bytes(w) bytes (256-byte
 * aligned); a tav2_weights whose `packed` points at it skips the packing step
 * of every later call (the paper's serving engine likewise keeps its model in
 * pre-allocated device memory, Sec. 3.4.2).  The buffer stays valid while the
 * weights it was packed from are unchanged; it is read-only to the library.
 * float32 weights are used as given: 0 bytes, and packing them is a no-op.
 * Errors: TAV2_ERR_NULL, TAV2_ERR_SHAPE, TAV2_ERR_DTYPE, TAV2_ERR_UNSUPPORTED,
 * TAV2_ERR_WORKSPACE (buffer NULL, misaligned or too small), TAV2_ERR_HIP.
 */
size_t tav2_pack_weights_bytes(const tav2_weights* w);
tav2_status tav2_pack_weights(const tav2_weights* w, void* packed, size_t bytes, void* stream);

/*
 * Encoder + head over explicit tokens (Eq. 4, Sec. 3.2.2):
 *   out device [total, 2 dm] float32:
 *     out[n, 0:dm]    = max over p < valid_len[n] of (X_p W_pool^T + b_pool)
 *     out[n, dm:2dm]  = X_{valid_len[n]-1}
 *   where X is the last layer's output under the mask `flags` selects
 *   (TAV2_MASK_CAUSAL or TAV2_MASK_NONE); rows with valid_len = 0 are zero.
 *   cand_emb device [total, d] (the tokens' dtype).
 * Supported shapes: bf16 with dm == 256, dm / n_heads in {32, 64},
 * d_ffn a multiple of 256 up to 4096, d a multiple of 32 up to 256, at most 8
 * layers; bf16 with dm == 64 (the paper's production encoder, Sec. 3.2.2),
 * dm / n_heads in {32, 64}, d_ffn a multiple of 32 up to 256, d a multiple of
 * 32 up to 256, at most 4 layers, all layer weights fitting the 160 KiB of LDS
 * next to the activations (2 layers of FFN 32 with d <= 64 do), its matrices
 * 16-byte and its tables 8-byte aligned (else TAV2_ERR_SHAPE); float32 with dm <= 128,
 * d_ffn <= 512, T <= 64 and d <= 256, dm, dm / n_heads and d_ffn multiples of 4.  Other valid shapes return
 * TAV2_ERR_UNSUPPORTED.  TAV2_MASK_NONE: T <= 128 for dm 256, T <= 64 for dm 64.
 * Errors: TAV2_ERR_NULL, TAV2_ERR_SHAPE, TAV2_ERR_DTYPE, TAV2_ERR_UNSUPPORTED,
 * TAV2_ERR_WORKSPACE, TAV2_ERR_HIP.
 */
size_t tav2_encode_workspace(const tav2_tokens* tok, const tav2_weights* w);
tav2_status tav2_encode(const tav2_tokens* tok, const void* cand_emb, const tav2_weights* w,
                        uint32_t flags, float* out, void* ws, size_t ws_bytes, void* stream);

/*
 * The whole path for a request batch, as the lifelong-sequence module computes
 * it at serving time: the candidate-anchored NN search of Eq. 3 over each
 * request's de-duplicated sequence (Sec. 3.4.2, 'Request Level
 * De-duplication'), the selected rows followed by the kept most-recent
 * real-time actions (Eq. 2, NN(S_LL, c) + S_RT[:r]), the feature encoding of
 * Eq. 4 and the encoder and head of Sec. 3.2.2, in one call.  out_idx /
 * out_score / out as in the calls above (out_idx and out_score may not be NULL:
 * the encoder reads the selection from them); flags as for tav2_encode.
 * T = k + (rt ? rt->max_len : 0) must not exceed w->max_pos.
 * Errors: those of tav2_nn_select and tav2_encode.
 */
size_t tav2_select_encode_workspace(const tav2_seq* seq, const tav2_seq* rt,
                                    const tav2_cands* cands, int32_t k,
                                    const tav2_weights* w);
tav2_status tav2_select_encode(const tav2_seq* seq, const tav2_seq* rt,
                               const tav2_cands* cands, int32_t k, const tav2_weights* w,
                               uint32_t flags, int32_t* out_idx, float* out_score, float* out,
                               void* ws, size_t ws_bytes, void* stream);

/*
 * The whole of Eq. 2 (Sec. 3.2.2): S_all = NN(S_LL, c) + S_RT[:r] +
 * NN(S_RT[r:], c) + NN(S_imp, c).  Besides the lifelong search of `seq` (k rows,
 * Eq. 3), the real-time sequence's most recent r rows are kept as they are, its
 * remaining rows are searched for k_rt rows, and the impression sequence is
 * searched for k_imp rows; the tokens of each search enter the encoder by
 * ascending score, the kept real-time rows oldest first, all valid tokens
 * packed from position 0.  Real-time and impression batches have the same
 * requests, width, dtype and time feature as `seq` (requests may be shorter
 * than r, k_rt or k_imp: their tokens are fewer).
 *   out_idx, out_score: device [total, k + k_rt + k_imp]: the lifelong rows, the
 *     real-time rest's rows (counted from S_RT[r]) and the impression rows, each
 *     in rank order and padded as tav2_nn_select pads.
 *   T = k + min(r, rt->max_len) + k_rt + k_imp positions; T <= w->max_pos.
 * tav2_select_encode(seq, rt, ...) is the case r = rt->max_len, k_rt = k_imp = 0.
 * Errors: those of tav2_select_encode; TAV2_ERR_NULL when a search or r > 0
 * names a missing sequence.
 */
typedef struct tav2_eq2 {
  const tav2_seq* rt;          /* real-time sequence S_RT (row 0 newest), or NULL */
  int32_t r;                   /* rows of S_RT kept unconditionally, >= 0 */
  int32_t k_rt;                /* NN top-k over S_RT[r:], 0..TAV2_K_MAX (0: no search) */
  const tav2_seq* imp;         /* impression sequence S_imp, or NULL */
  int32_t k_imp;               /* NN top-k over S_imp, 0..TAV2_K_MAX (0: no search) */
  int32_t reserved;            /* set to 0 */
} tav2_eq2;
size_t tav2_select_encode_eq2_workspace(const tav2_seq* seq, const tav2_eq2* eq2,
                                        const tav2_cands* cands, int32_t k,
                                        const tav2_weights* w);
tav2_status tav2_select_encode_eq2(const tav2_seq* seq, const tav2_eq2* eq2,
                                   const tav2_cands* cands, int32_t k, const tav2_weights* w,
                                   uint32_t flags, int32_t* out_idx, float* out_score, float* out,
                                   void* ws, size_t ws_bytes, void* stream);

/*
 * Measurement hook for benchmarks and profilers (not needed for serving).
 * tav2_profile_enable(1, site) makes every later kernel launch of the library
 * whose site name equals `site` (NULL: every site) record a HIP event before
 * and after itself on its stream (timing-only events, without a system-scope
 * fence); tav2_profile_enable(0, NULL) stops it.
 * After the caller has synchronised, tav2_profile_report() writes one line
 * "<site> <launches> <total_ms>" per site into buf (NUL-terminated, truncated
 * to buf_bytes), forgets the recorded launches and returns the untruncated
 * text length.  Site names: seq_view, nn_sample, nn_threshold, nn_filter, nn_select,
 * nn_fallback (the NN search with on-chip scores, for bf16 and int8 sequences of
 * more than 4096 rows), score_bf16, score_i8, score_f32, topk (the NN search over
 * materialised score rows), gather, pack_weights, cand_proj, encoder_fused (the
 * bf16 encoder of d_model 256), encoder_small (d_model 64), encode_f32.
 */
int32_t tav2_profile_enable(int32_t on, const char* only_site);
int64_t tav2_profile_report(char* buf, size_t buf_bytes);

/*
 * Serving-side batching (Sec. 3.4.2, 'Pinned Memory Arena' and 'Request Level
 * De-duplication').  A batcher owns a pinned host arena and a device mirror of
 * one mini-batch in the de-duplicated layout of tav2_seq / tav2_cands, both
 * allocated once by tav2_batcher_create and freed by tav2_batcher_destroy (the
 * only calls of this library that allocate; the arena is reset, never freed,
 * between mini-batches).  Requests are collated straight into the pinned arena
 * (no pageable staging copy), each request's sequences once whatever its number
 * of candidates; tav2_batcher_upload moves the whole mini-batch to the device
 * with one host-to-device copy on the caller's stream; tav2_batcher_views gives
 * the tav2_seq / tav2_cands that tav2_select_encode then takes.
 *
 * Dynamic batching: tav2_batcher_add returns TAV2_ERR_TOO_LARGE when the request
 * does not fit the capacities; the caller uploads and runs the mini-batch and
 * starts the next one with tav2_batcher_reset.  After an upload the mini-batch
 * is sealed: add returns TAV2_ERR_SHAPE until reset, and a second upload copies
 * the same bytes again.  The copy is asynchronous: the caller synchronises the
 * stream before it resets the batcher or reuses the views' memory for the next
 * mini-batch.  A batcher is not thread-safe; use one per serving thread (the
 * paper's arena is thread-local).
 */
typedef struct tav2_batcher tav2_batcher;
typedef struct tav2_batcher_config {
  int32_t dtype;          /* sequence dtype: TAV2_F32, TAV2_BF16 or TAV2_I8 (candidates: fp32
                             with fp32 sequences, else bf16) */
  int32_t d;              /* embedding width, multiple of 16, 16..512 */
  int32_t has_time;       /* 1: time buckets present, 0: absent */
  int32_t max_requests;   /* requests of one mini-batch, 1..65535 */
  int64_t max_rows;       /* lifelong rows of one mini-batch, summed over its requests */
  int64_t max_rt_rows;    /* real-time rows of one mini-batch (0: none) */
  int64_t max_cands;      /* candidates of one mini-batch, >= 1 */
} tav2_batcher_config;
typedef struct tav2_request {   /* HOST pointers, read during tav2_batcher_add only */
  const void*    emb;             /* [len, d]: the lifelong sequence, most recent first */
  const uint8_t* action_type;     /* [len] */
  const uint8_t* time_bucket;     /* [len], or NULL without the time feature */
  int32_t        len;
  int32_t        rt_len;          /* real-time rows (0: none) */
  const void*    rt_emb;          /* [rt_len, d], most recent first */
  const uint8_t* rt_action_type;  /* [rt_len] */
  const uint8_t* rt_time_bucket;  /* [rt_len], or NULL */
  const void*    cand_emb;        /* [n_cands, d] */
  int32_t        n_cands;
  int32_t        reserved;        /* set to 0 */
} tav2_request;
/* Errors: TAV2_ERR_NULL, TAV2_ERR_SHAPE, TAV2_ERR_DTYPE (bad configuration, checked
 * before anything is allocated), TAV2_ERR_HIP (allocation failed). */
tav2_status tav2_batcher_create(const tav2_batcher_config* cfg, tav2_batcher** out);
void tav2_batcher_destroy(tav2_batcher* b);
size_t tav2_batcher_arena_bytes(const tav2_batcher* b);   /* pinned bytes (= device bytes) */
tav2_status tav2_batcher_reset(tav2_batcher* b);
/* Errors: TAV2_ERR_NULL, TAV2_ERR_SHAPE, TAV2_ERR_TOO_LARGE (does not fit: nothing added). */
tav2_status tav2_batcher_add(tav2_batcher* b, const tav2_request* r);
/* Errors: TAV2_ERR_NULL, TAV2_ERR_HIP. */
tav2_status tav2_batcher_upload(tav2_batcher* b, void* stream);
/* Device views of the uploaded mini-batch (rt may be NULL; its num_requests is the
 * batch's, with rt_len 0 for requests without real-time rows).  Errors:
 * TAV2_ERR_NULL, TAV2_ERR_SHAPE (nothing uploaded since the last reset). */
tav2_status tav2_batcher_views(const tav2_batcher* b, tav2_seq* seq, tav2_seq* rt,
                               tav2_cands* cands);

#ifdef __cplusplus
}
#endif

#endif /* TAV2_H */
