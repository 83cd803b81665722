// Serving-side batching (Sec. 3.4.2, 'Pinned Memory Arena' and 'Request Level
// De-duplication'): a mini-batch of requests is collated straight into a pinned
// host arena in the de-duplicated layout of tav2_seq / tav2_cands (each request's
// sequences once, however many candidates it has), then moved to static device
// memory with one host-to-device copy.  Every buffer is allocated at creation;
// between mini-batches the arena is reset, never freed.
//
// Arena layout (host, pinned): [lifelong rows | staging areas | metadata].
// add() writes a request's lifelong embedding rows at the running row cursor of
// the first region and everything else (action types, time buckets, real-time
// rows, candidate rows) into per-array staging areas.  upload() packs the used
// part of every staged array, then the offsets and lengths, right after the used
// lifelong rows (host moves of the small arrays only), so that the whole
// mini-batch is one contiguous range, and copies that range to the device mirror
// in one call.
#include <string.h>

#include <algorithm>
#include <vector>

#include "common.h"
#include "internal.h"

namespace {

constexpr size_t ALIGN = 256;

size_t up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

size_t elem_bytes(int32_t dtype) { return dtype == TAV2_I8 ? 1 : dtype == TAV2_BF16 ? 2 : 4; }
size_t cand_elem_bytes(int32_t dtype) { return dtype == TAV2_F32 ? 4 : 2; }

}  // namespace

struct tav2_batcher {
  tav2_batcher_config cfg;
  size_t row_bytes, cand_row_bytes;
  // staging areas inside the arena (byte offsets) and their capacities
  size_t st_act, st_time, st_rt_emb, st_rt_act, st_rt_time, st_cand;
  size_t tail;            // end of the staging areas
  size_t arena_bytes;
  uint8_t* host = nullptr;   // pinned arena
  uint8_t* dev = nullptr;    // device mirror of the arena
  // the mini-batch being collated
  int32_t requests = 0;
  int64_t rows = 0, rt_rows = 0, cands = 0;
  int32_t max_len = 0, rt_max_len = 0, max_count = 0;
  std::vector<int64_t> off, rt_off, cand_off;
  std::vector<int32_t> len, rt_len;
  // the packed layout of the last upload (byte offsets into the arena / mirror)
  bool packed = false;     // upload() has packed the mini-batch (sealed until reset)
  size_t p_act, p_time, p_off, p_len, p_rt_emb, p_rt_act, p_rt_time, p_rt_off, p_rt_len,
      p_cand, p_cand_off, used;
};

namespace {

tav2_status check_config(const tav2_batcher_config* c) {
  if (!c) return TAV2_ERR_NULL;
  if (c->dtype != TAV2_F32 && c->dtype != TAV2_BF16 && c->dtype != TAV2_I8) return TAV2_ERR_DTYPE;
  if (c->d < 16 || c->d > 512 || c->d % 16) return TAV2_ERR_SHAPE;
  if (c->max_requests < 1 || c->max_requests > 65535) return TAV2_ERR_SHAPE;
  if (c->max_rows < 0 || c->max_rt_rows < 0 || c->max_cands < 1) return TAV2_ERR_SHAPE;
  if (c->max_cands > (int64_t(1) << 31) - 1 || c->max_rows > (int64_t(1) << 40) ||
      c->max_rt_rows > (int64_t(1) << 40))
    return TAV2_ERR_SHAPE;
  if (c->has_time != 0 && c->has_time != 1) return TAV2_ERR_SHAPE;
  return TAV2_OK;
}

}  // namespace

extern "C" {

tav2_status tav2_batcher_create(const tav2_batcher_config* cfg, tav2_batcher** out) {
  if (!out) return TAV2_ERR_NULL;
  *out = nullptr;
  tav2_status st = check_config(cfg);
  if (st) return st;
  tav2_batcher* b = new tav2_batcher();
  b->cfg = *cfg;
  const tav2_batcher_config& c = *cfg;
  const size_t R = size_t(c.max_requests);
  b->row_bytes = size_t(c.d) * elem_bytes(c.dtype);
  b->cand_row_bytes = size_t(c.d) * cand_elem_bytes(c.dtype);
  const size_t rows = size_t(c.max_rows), rt = size_t(c.max_rt_rows), nc = size_t(c.max_cands);
  // staging (after the lifelong rows)
  size_t o = up(rows * b->row_bytes);
  b->st_act = o;     o += up(rows);
  b->st_time = o;    o += up(c.has_time ? rows : 0);
  b->st_rt_emb = o;  o += up(rt * b->row_bytes);
  b->st_rt_act = o;  o += up(rt);
  b->st_rt_time = o; o += up(c.has_time ? rt : 0);
  b->st_cand = o;    o += up(nc * b->cand_row_bytes);
  // upload() packs the staged arrays down over the staging areas and appends the
  // offsets and lengths: at most the staging areas plus the metadata
  b->tail = o;
  const size_t meta = up(R * 8) + up(R * 4) + up(R * 8) + up(R * 4) + up((R + 1) * 8);
  b->arena_bytes = o + meta;
  if (hipHostMalloc(reinterpret_cast<void**>(&b->host), b->arena_bytes, hipHostMallocDefault) !=
      hipSuccess) {
    delete b;
    return TAV2_ERR_HIP;
  }
  if (hipMalloc(reinterpret_cast<void**>(&b->dev), b->arena_bytes) != hipSuccess) {
    (void)hipHostFree(b->host);
    delete b;
    return TAV2_ERR_HIP;
  }
  b->off.reserve(R);
  b->rt_off.reserve(R);
  b->cand_off.reserve(R + 1);
  b->len.reserve(R);
  b->rt_len.reserve(R);
  *out = b;
  return tav2_batcher_reset(b);
}

void tav2_batcher_destroy(tav2_batcher* b) {
  if (!b) return;
  (void)hipFree(b->dev);
  (void)hipHostFree(b->host);
  delete b;
}

tav2_status tav2_batcher_reset(tav2_batcher* b) {
  if (!b) return TAV2_ERR_NULL;
  b->requests = 0;
  b->rows = b->rt_rows = b->cands = 0;
  b->max_len = b->rt_max_len = b->max_count = 0;
  b->off.clear();
  b->rt_off.clear();
  b->len.clear();
  b->rt_len.clear();
  b->cand_off.assign(1, 0);
  b->packed = false;
  return TAV2_OK;
}

size_t tav2_batcher_arena_bytes(const tav2_batcher* b) { return b ? b->arena_bytes : 0; }

tav2_status tav2_batcher_add(tav2_batcher* b, const tav2_request* q) {
  if (!b || !q) return TAV2_ERR_NULL;
  if (b->packed) return TAV2_ERR_SHAPE;   // uploaded: reset before the next mini-batch
  const tav2_batcher_config& c = b->cfg;
  if (q->len < 0 || q->rt_len < 0 || q->n_cands < 0) return TAV2_ERR_SHAPE;
  if ((q->len > 0 && (!q->emb || !q->action_type)) ||
      (q->rt_len > 0 && (!q->rt_emb || !q->rt_action_type)) || (q->n_cands > 0 && !q->cand_emb))
    return TAV2_ERR_NULL;
  if (c.has_time && ((q->len > 0 && !q->time_bucket) || (q->rt_len > 0 && !q->rt_time_bucket)))
    return TAV2_ERR_NULL;
  if (b->requests + 1 > c.max_requests || b->rows + q->len > c.max_rows ||
      b->rt_rows + q->rt_len > c.max_rt_rows || b->cands + q->n_cands > c.max_cands)
    return TAV2_ERR_TOO_LARGE;   // the mini-batch is full: upload it and start the next
  uint8_t* h = b->host;
  const size_t n = size_t(q->len), m = size_t(q->rt_len), k = size_t(q->n_cands);
  if (n) {
    memcpy(h + size_t(b->rows) * b->row_bytes, q->emb, n * b->row_bytes);
    memcpy(h + b->st_act + size_t(b->rows), q->action_type, n);
    if (c.has_time) memcpy(h + b->st_time + size_t(b->rows), q->time_bucket, n);
  }
  if (m) {
    memcpy(h + b->st_rt_emb + size_t(b->rt_rows) * b->row_bytes, q->rt_emb, m * b->row_bytes);
    memcpy(h + b->st_rt_act + size_t(b->rt_rows), q->rt_action_type, m);
    if (c.has_time) memcpy(h + b->st_rt_time + size_t(b->rt_rows), q->rt_time_bucket, m);
  }
  if (k) memcpy(h + b->st_cand + size_t(b->cands) * b->cand_row_bytes, q->cand_emb, k * b->cand_row_bytes);
  b->off.push_back(b->rows);
  b->len.push_back(q->len);
  b->rt_off.push_back(b->rt_rows);
  b->rt_len.push_back(q->rt_len);
  b->rows += q->len;
  b->rt_rows += q->rt_len;
  b->cands += q->n_cands;
  b->cand_off.push_back(b->cands);
  b->max_len = std::max(b->max_len, q->len);
  b->rt_max_len = std::max(b->rt_max_len, q->rt_len);
  b->max_count = std::max(b->max_count, q->n_cands);
  b->requests += 1;
  return TAV2_OK;
}

tav2_status tav2_batcher_upload(tav2_batcher* b, void* stream) {
  if (!b) return TAV2_ERR_NULL;
  if (b->packed) {   // already packed: copy the same range again
    return hipMemcpyAsync(b->dev, b->host, b->used, hipMemcpyHostToDevice,
                          static_cast<hipStream_t>(stream)) == hipSuccess ? TAV2_OK : TAV2_ERR_HIP;
  }
  const tav2_batcher_config& c = b->cfg;
  uint8_t* h = b->host;
  const size_t R = size_t(b->requests), rows = size_t(b->rows), rt = size_t(b->rt_rows),
               nc = size_t(b->cands);
  // pack: the used lifelong rows stay where they are; the rest follows them
  size_t o = up(rows * b->row_bytes);
  auto put = [&](size_t& at, const void* src, size_t bytes) {
    at = o;
    if (bytes) memmove(h + o, src, bytes);
    o += up(bytes);
  };
  // The staged arrays move in staging order, each to an offset at or below its
  // own staging offset and ending before the next array's (the used part of
  // every region is at most its capacity), so no move overwrites data still to
  // be moved; the offsets and lengths, from host vectors, follow them.
  put(b->p_act, h + b->st_act, rows);
  put(b->p_time, h + b->st_time, c.has_time ? rows : 0);
  put(b->p_rt_emb, h + b->st_rt_emb, rt * b->row_bytes);
  put(b->p_rt_act, h + b->st_rt_act, rt);
  put(b->p_rt_time, h + b->st_rt_time, c.has_time ? rt : 0);
  put(b->p_cand, h + b->st_cand, nc * b->cand_row_bytes);
  put(b->p_off, b->off.data(), R * 8);
  put(b->p_len, b->len.data(), R * 4);
  put(b->p_rt_off, b->rt_off.data(), R * 8);
  put(b->p_rt_len, b->rt_len.data(), R * 4);
  put(b->p_cand_off, b->cand_off.data(), (R + 1) * 8);
  b->used = o;
  b->packed = true;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (hipMemcpyAsync(b->dev, b->host, b->used, hipMemcpyHostToDevice, st) != hipSuccess)
    return TAV2_ERR_HIP;
  return TAV2_OK;
}

tav2_status tav2_batcher_views(const tav2_batcher* b, tav2_seq* seq, tav2_seq* rt,
                               tav2_cands* cands) {
  if (!b || !seq || !cands) return TAV2_ERR_NULL;
  if (!b->packed) return TAV2_ERR_SHAPE;
  const tav2_batcher_config& c = b->cfg;
  uint8_t* d = b->dev;
  seq->emb = d;
  seq->action_type = d + b->p_act;
  seq->time_bucket = c.has_time ? d + b->p_time : nullptr;
  seq->offset = reinterpret_cast<const int64_t*>(d + b->p_off);
  seq->len = reinterpret_cast<const int32_t*>(d + b->p_len);
  seq->num_requests = b->requests;
  seq->d = c.d;
  seq->dtype = c.dtype;
  seq->max_len = b->max_len;
  if (rt) {
    rt->emb = d + b->p_rt_emb;
    rt->action_type = d + b->p_rt_act;
    rt->time_bucket = c.has_time ? d + b->p_rt_time : nullptr;
    rt->offset = reinterpret_cast<const int64_t*>(d + b->p_rt_off);
    rt->len = reinterpret_cast<const int32_t*>(d + b->p_rt_len);
    rt->num_requests = b->requests;
    rt->d = c.d;
    rt->dtype = c.dtype;
    rt->max_len = b->rt_max_len;
  }
  cands->emb = d + b->p_cand;
  cands->offset = reinterpret_cast<const int64_t*>(d + b->p_cand_off);
  cands->total = b->cands;
  cands->max_count = b->max_count;
  cands->reserved = 0;
  return TAV2_OK;
}

}  // extern "C"
