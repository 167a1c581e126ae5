// C ABI of the Minima-KV gfx950 library: argument validation, pool set-up and
// kernel launches on the caller's stream.  See include/minima_kv.h.
#include <hip/hip_runtime.h>

#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/minima_kv.h"
#include "mkv_internal.h"

using namespace mkv;

namespace {

mkv_status check_geometry(const mkv_pool_desc* d) {
  if (!d) return MKV_EINVAL;
  if (d->n_layers < 1 || d->n_q_heads < 1 || d->n_kv_heads < 1 || d->n_fp8_pages < 1 ||
      d->n_tq3_pages < 0 || d->recent_tokens < 1)
    return MKV_EINVAL;
  if (d->page_size != PAGE) return MKV_EUNSUP;
  if (d->head_dim != 128 && d->head_dim != 256) return MKV_EUNSUP;
  if (d->n_q_heads % d->n_kv_heads != 0) return MKV_EINVAL;
  if (d->n_q_heads / d->n_kv_heads > 16) return MKV_EUNSUP;
  return MKV_OK;
}

struct Sizes {
  size_t fp8, scales, tq3, ctrl;
};

Sizes sizes_of(const mkv_pool_desc* d) {
  Sizes s;
  const size_t ph8 = (size_t)d->n_layers * d->n_fp8_pages * d->n_kv_heads;
  const size_t ph3 = (size_t)d->n_layers * d->n_tq3_pages * d->n_kv_heads;
  s.fp8 = ph8 * (size_t)fp8_region_bytes(d->head_dim);
  s.scales = ph8 * 2 * sizeof(float);
  s.tq3 = ph3 * (size_t)tq3_region_bytes(d->head_dim);
  s.ctrl = (size_t)ctrl_layout(d->n_fp8_pages, d->n_tq3_pages, d->head_dim).total_words * 4;
  return s;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

bool is_permutation(const int32_t* o, int n) {
  if (!o) return true;
  std::vector<char> seen((size_t)n, 0);
  for (int i = 0; i < n; ++i) {
    if (o[i] < 0 || o[i] >= n || seen[(size_t)o[i]]) return false;
    seen[(size_t)o[i]] = 1;
  }
  return true;
}

mkv_status hip_status(hipError_t e) { return e == hipSuccess ? MKV_OK : MKV_EHIP; }

}  // namespace

extern "C" {

const char* mkv_status_string(mkv_status s) {
  switch (s) {
    case MKV_OK: return "ok";
    case MKV_EINVAL: return "invalid argument";
    case MKV_EUNSUP: return "unsupported geometry";
    case MKV_ENOMEM: return "buffer too small";
    case MKV_ERANGE: return "index or length out of range";
    case MKV_ESTATE: return "invalid pool state";
    case MKV_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

mkv_status kv_pool_bytes(const mkv_pool_desc* desc, size_t* fp8_data_bytes, size_t* fp8_scales_bytes,
                         size_t* tq3_data_bytes, size_t* ctrl_bytes) {
  mkv_status st = check_geometry(desc);
  if (st != MKV_OK) return st;
  Sizes s = sizes_of(desc);
  if (fp8_data_bytes) *fp8_data_bytes = s.fp8;
  if (fp8_scales_bytes) *fp8_scales_bytes = s.scales;
  if (tq3_data_bytes) *tq3_data_bytes = s.tq3;
  if (ctrl_bytes) *ctrl_bytes = s.ctrl;
  return MKV_OK;
}

mkv_status kv_pool_create(const mkv_pool_desc* desc, mkv_pool** out) {
  if (!out) return MKV_EINVAL;
  *out = nullptr;
  mkv_status st = check_geometry(desc);
  if (st != MKV_OK) return st;
  if (!desc->rot_signs || !desc->fp8_data || !desc->fp8_scales || !desc->ctrl ||
      (desc->n_tq3_pages > 0 && !desc->tq3_data))
    return MKV_EINVAL;
  for (int i = 0; i < desc->head_dim; ++i)
    if (desc->rot_signs[i] != 1 && desc->rot_signs[i] != -1) return MKV_EINVAL;
  if (!is_permutation(desc->fp8_order, desc->n_fp8_pages) ||
      !is_permutation(desc->tq3_order, desc->n_tq3_pages))
    return MKV_EINVAL;
  Sizes s = sizes_of(desc);
  if (desc->fp8_data_bytes < s.fp8 || desc->fp8_scales_bytes < s.scales ||
      desc->tq3_data_bytes < s.tq3 || desc->ctrl_bytes < s.ctrl)
    return MKV_ENOMEM;
  if (!aligned16(desc->fp8_data) || !aligned16(desc->fp8_scales) || !aligned16(desc->ctrl) ||
      (desc->tq3_data && !aligned16(desc->tq3_data)))
    return MKV_EINVAL;
  mkv_pool* p = new (std::nothrow) mkv_pool;
  if (!p) return MKV_ENOMEM;
  p->n_layers = desc->n_layers;
  p->n_q_heads = desc->n_q_heads;
  p->n_kv_heads = desc->n_kv_heads;
  p->d = desc->head_dim;
  p->group = desc->n_q_heads / desc->n_kv_heads;
  p->n_fp8 = desc->n_fp8_pages;
  p->n_tq3 = desc->n_tq3_pages;
  p->recent = desc->recent_tokens;
  p->fp8 = static_cast<uint8_t*>(desc->fp8_data);
  p->fp8_scales = static_cast<float*>(desc->fp8_scales);
  p->tq3 = static_cast<uint8_t*>(desc->tq3_data);
  p->ctrl = static_cast<int32_t*>(desc->ctrl);
  p->cl = ctrl_layout(p->n_fp8, p->n_tq3, p->d);
  p->decode_routes = p->chunk_routes = 0;
  p->timing = p->timed = 0;
  p->deterministic = 0;
  // host image of ctrl: header, stacks (next id handed out = last element)
  std::vector<int32_t> img((size_t)p->cl.total_words, 0);
  img[CTRL_FP8_TOP] = p->n_fp8;
  img[CTRL_TQ3_TOP] = p->n_tq3;
  for (int i = 0; i < p->n_fp8; ++i)
    img[(size_t)p->cl.fp8_stack + i] = desc->fp8_order ? desc->fp8_order[p->n_fp8 - 1 - i] : p->n_fp8 - 1 - i;
  for (int i = 0; i < p->n_tq3; ++i)
    img[(size_t)p->cl.tq3_stack + i] = desc->tq3_order ? desc->tq3_order[p->n_tq3 - 1 - i] : p->n_tq3 - 1 - i;
  std::memcpy(reinterpret_cast<uint8_t*>(img.data()) + p->cl.sigma_bytes, desc->rot_signs,
              (size_t)p->d);
  for (int i = 0; i < p->n_fp8; ++i) img[(size_t)p->cl.last8 + i] = -1;
  for (int i = 0; i < p->n_tq3; ++i) img[(size_t)p->cl.last3 + i] = -1;
  hipError_t e = hipMemcpy(p->ctrl, img.data(), img.size() * 4, hipMemcpyHostToDevice);
  int dev = -1;
  if (e == hipSuccess) e = hipGetDevice(&dev);
  // set-up of the allocation-free decode: the device address of its scratch
  if (e == hipSuccess) e = decode_scratch_init(dev);
  if (e != hipSuccess) {
    delete p;
    return MKV_EHIP;
  }
  *out = p;
  return MKV_OK;
}

mkv_status kv_pool_destroy(mkv_pool* pool) {
  if (!pool) return MKV_EINVAL;
  (void)paged_attn_set_timing(pool, 0);
  delete pool;
  return MKV_OK;
}

mkv_status kv_append_fp8(mkv_pool* pool, int32_t layer, int32_t n_req, int32_t* block_table,
                         uint8_t* tags, int32_t max_pages, const int32_t* seq_lens_before,
                         const int32_t* cu_new_tokens, int32_t n_new_total, const uint16_t* k,
                         const uint16_t* v, hipStream_t stream) {
  if (!pool || !block_table || !tags || !seq_lens_before || !cu_new_tokens) return MKV_EINVAL;
  if (n_req < 1 || max_pages < 1 || n_new_total < 0) return MKV_EINVAL;
  if (n_new_total > 0 && (!k || !v)) return MKV_EINVAL;
  if (layer != MKV_ALL_LAYERS && (layer < 0 || layer >= pool->n_layers)) return MKV_ERANGE;
  return hip_status(launch_append(view_of(pool), layer, n_req, block_table, tags, max_pages,
                                  seq_lens_before, cu_new_tokens, n_new_total, k, v, stream));
}

mkv_status kv_migrate_to_tq3(mkv_pool* pool, int32_t n_req, int32_t* block_table, uint8_t* tags,
                             int32_t max_pages, const uint8_t* anchor_mask, const int32_t* seq_lens,
                             hipStream_t stream) {
  if (!pool || !block_table || !tags || !seq_lens) return MKV_EINVAL;
  if (n_req < 1 || max_pages < 1) return MKV_EINVAL;
  return hip_status(launch_migrate(view_of(pool), n_req, block_table, tags, max_pages, anchor_mask,
                                   seq_lens, stream));
}

mkv_status kv_promote_to_fp8(mkv_pool* pool, int32_t n_req, int32_t* block_table, uint8_t* tags,
                             int32_t max_pages, const uint8_t* promote_mask,
                             const int32_t* seq_lens, hipStream_t stream) {
  if (!pool || !block_table || !tags || !promote_mask || !seq_lens) return MKV_EINVAL;
  if (n_req < 1 || max_pages < 1) return MKV_EINVAL;
  return hip_status(launch_promote(view_of(pool), n_req, block_table, tags, max_pages, promote_mask,
                                   seq_lens, stream));
}

mkv_status kv_pages_acquire(mkv_pool* pool, int32_t n, const int32_t* ids, const uint8_t* tags,
                            hipStream_t stream) {
  if (!pool || n < 0 || (n > 0 && (!ids || !tags))) return MKV_EINVAL;
  return hip_status(launch_pages_acquire(view_of(pool), n, ids, tags, stream));
}

mkv_status kv_pages_release(mkv_pool* pool, int32_t n, const int32_t* ids, const uint8_t* tags,
                            hipStream_t stream) {
  if (!pool || n < 0 || (n > 0 && (!ids || !tags))) return MKV_EINVAL;
  return hip_status(launch_pages_release(view_of(pool), n, ids, tags, 0, nullptr, 0, nullptr,
                                         nullptr, 1, stream));
}

mkv_status kv_request_finish(mkv_pool* pool, int32_t n_fin, const int32_t* reqs, int32_t n_req,
                             int32_t* block_table, uint8_t* tags, int32_t max_pages,
                             hipStream_t stream) {
  if (!pool || !reqs || !block_table || !tags || n_fin < 0 || n_req < 1 || max_pages < 1)
    return MKV_EINVAL;
  if ((int64_t)n_fin * max_pages > ((int64_t)1 << 31) - 1) return MKV_ERANGE;
  return hip_status(launch_pages_release(view_of(pool), 0, nullptr, nullptr, n_fin, reqs, n_req,
                                         block_table, tags, max_pages, stream));
}

mkv_status kv_pool_read_refcounts(mkv_pool* pool, int32_t* rc_fp8, int32_t* rc_tq3) {
  if (!pool) return MKV_EINVAL;
  if (hipDeviceSynchronize() != hipSuccess) return MKV_EHIP;
  if (rc_fp8 && hipMemcpy(rc_fp8, pool->ctrl + pool->cl.rc8, (size_t)pool->n_fp8 * 4,
                          hipMemcpyDeviceToHost) != hipSuccess)
    return MKV_EHIP;
  if (rc_tq3 && pool->n_tq3 > 0 &&
      hipMemcpy(rc_tq3, pool->ctrl + pool->cl.rc3, (size_t)pool->n_tq3 * 4, hipMemcpyDeviceToHost) !=
          hipSuccess)
    return MKV_EHIP;
  return MKV_OK;
}

mkv_status paged_attn_workspace_bytes(const mkv_pool* pool, int32_t n_req, int32_t max_pages,
                                      int32_t n_q_total, size_t* bytes) {
  if (!pool || !bytes || n_req < 1 || max_pages < 1 || n_q_total < 0) return MKV_EINVAL;
  if (n_q_total == 0)
    *bytes = decode_ws_bytes(n_req, max_pages, pool->n_kv_heads, pool->group, pool->d, pool->recent);
  else
    *bytes = chunk_ws_bytes(n_req, max_pages, n_q_total, pool->n_kv_heads, pool->group, pool->d);
  return MKV_OK;
}

mkv_status paged_attn_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!ws) return MKV_EINVAL;
  return hip_status(launch_fill_zero(ws, ws_bytes, stream));
}

mkv_status paged_attn_decode(mkv_pool* pool, int32_t layer, int32_t n_req, const uint16_t* q,
                             const int32_t* block_table, const uint8_t* tags, int32_t max_pages,
                             const int32_t* seq_lens, float* out, float* lse, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  if (!pool || !q || !block_table || !tags || !seq_lens || !out || !ws) return MKV_EINVAL;
  if (n_req < 1 || max_pages < 1) return MKV_EINVAL;
  if (!aligned16(q) || !aligned16(out) || !aligned16(ws)) return MKV_EINVAL;
  if (layer < 0 || layer >= pool->n_layers) return MKV_ERANGE;
  if (n_req > 65535 || max_pages > 1024 * 256) return MKV_ERANGE;
  if (ws_bytes < decode_ws_bytes(n_req, max_pages, pool->n_kv_heads, pool->group, pool->d, pool->recent))
    return MKV_ENOMEM;
  mkv_status st = hip_status(launch_decode(view_of(pool), layer, n_req, q, block_table, tags,
                                           max_pages, seq_lens, out, lse, ws, stream,
                                           pool->timing ? pool->timing_ev : nullptr));
  if (st == MKV_OK) {
    pool->decode_routes++;
    if (pool->timing) pool->timed = 1;
  }
  return st;
}

mkv_status paged_attn_decode_scores(mkv_pool* pool, int32_t layer, int32_t n_req,
                                    const uint16_t* q, const int32_t* block_table,
                                    const uint8_t* tags, int32_t max_pages,
                                    const int32_t* seq_lens, float* out, float* lse, void* ws,
                                    size_t ws_bytes, float* page_mass, hipStream_t stream) {
  if (!pool || !q || !block_table || !tags || !seq_lens || !out || !lse || !ws || !page_mass)
    return MKV_EINVAL;
  if (n_req < 1 || max_pages < 1) return MKV_EINVAL;
  if (!aligned16(q) || !aligned16(out) || !aligned16(ws) || (reinterpret_cast<uintptr_t>(page_mass) & 7))
    return MKV_EINVAL;
  if (layer < 0 || layer >= pool->n_layers) return MKV_ERANGE;
  if (n_req > 65535 || max_pages > 1024 * 256) return MKV_ERANGE;
  if (ws_bytes < decode_ws_bytes(n_req, max_pages, pool->n_kv_heads, pool->group, pool->d, pool->recent))
    return MKV_ENOMEM;
  mkv_status st = hip_status(launch_decode(view_of(pool), layer, n_req, q, block_table, tags,
                                           max_pages, seq_lens, out, lse, ws, stream,
                                           pool->timing ? pool->timing_ev : nullptr, nullptr,
                                           nullptr, nullptr, nullptr,
                                           reinterpret_cast<float2*>(page_mass)));
  if (st == MKV_OK) {
    pool->decode_routes++;
    if (pool->timing) pool->timed = 1;
  }
  return st;
}

mkv_status kv_page_scores_update(const mkv_pool* pool, int32_t n_req, int32_t max_pages,
                                 const int32_t* seq_lens, const float* lse,
                                 const float* page_mass, const uint8_t* head_mask, float beta,
                                 float* scores, float* r_out, float* qn_out, hipStream_t stream) {
  if (!pool || !seq_lens || !lse || !page_mass || !head_mask || !scores) return MKV_EINVAL;
  if (n_req < 1 || max_pages < 1 || !(beta >= 0.0f && beta <= 1.0f)) return MKV_EINVAL;
  if (reinterpret_cast<uintptr_t>(page_mass) & 7) return MKV_EINVAL;
  if (pool->n_q_heads > 256) return MKV_EUNSUP;
  if (n_req > 65535 || max_pages > 1024 * 256) return MKV_ERANGE;
  return hip_status(launch_score_collect(n_req, pool->n_q_heads, max_pages, seq_lens, lse,
                                         reinterpret_cast<const float2*>(page_mass), head_mask,
                                         beta, scores, r_out, qn_out, stream));
}

mkv_status paged_attn_decode_noalloc(mkv_pool* pool, int32_t layer, int32_t n_req,
                                     const uint16_t* q, const int32_t* block_table,
                                     const uint8_t* tags, int32_t max_pages,
                                     const int32_t* seq_lens, float* out, float* lse,
                                     hipStream_t stream) {
  if (!pool || !q || !block_table || !tags || !seq_lens || !out) return MKV_EINVAL;
  if (n_req < 1 || max_pages < 1) return MKV_EINVAL;
  if (!aligned16(q) || !aligned16(out)) return MKV_EINVAL;
  if (layer < 0 || layer >= pool->n_layers) return MKV_ERANGE;
  if (n_req > 65535 || max_pages > 1024 * 256) return MKV_ERANGE;
  if (decode_ws_bytes(n_req, max_pages, pool->n_kv_heads, pool->group, pool->d, pool->recent) >
      (size_t)MKV_DECODE_SCRATCH_BYTES)
    return MKV_ENOMEM;
  int dev = -1;
  void* ws = nullptr;
  if (hipGetDevice(&dev) != hipSuccess || decode_scratch(dev, &ws) != hipSuccess) return MKV_EHIP;
  mkv_status st = hip_status(launch_decode(view_of(pool), layer, n_req, q, block_table, tags,
                                           max_pages, seq_lens, out, lse, ws, stream,
                                           pool->timing ? pool->timing_ev : nullptr));
  if (st == MKV_OK) {
    pool->decode_routes++;
    if (pool->timing) pool->timed = 1;
  }
  return st;
}

mkv_status paged_attn_decode_append(mkv_pool* pool, int32_t layer, int32_t n_req,
                                    const uint16_t* q, const uint16_t* k_new,
                                    const uint16_t* v_new, int32_t* block_table, uint8_t* tags,
                                    int32_t max_pages, const int32_t* seq_lens_before,
                                    float* out, float* lse, void* ws, size_t ws_bytes,
                                    hipStream_t stream) {
  if (!pool || !q || !k_new || !v_new || !block_table || !tags || !seq_lens_before || !out || !ws)
    return MKV_EINVAL;
  if (n_req < 1 || max_pages < 1) return MKV_EINVAL;
  if (!aligned16(q) || !aligned16(out) || !aligned16(ws)) return MKV_EINVAL;
  if ((reinterpret_cast<uintptr_t>(k_new) | reinterpret_cast<uintptr_t>(v_new)) & 7) return MKV_EINVAL;
  if (layer < 0 || layer >= pool->n_layers) return MKV_ERANGE;
  if (n_req > 65535 || max_pages > 1024 * 256) return MKV_ERANGE;
  if (ws_bytes < decode_ws_bytes(n_req, max_pages, pool->n_kv_heads, pool->group, pool->d, pool->recent))
    return MKV_ENOMEM;
  mkv_status st = hip_status(launch_decode(view_of(pool), layer, n_req, q, block_table, tags,
                                           max_pages, seq_lens_before, out, lse, ws, stream,
                                           pool->timing ? pool->timing_ev : nullptr, k_new, v_new,
                                           block_table, tags));
  if (st == MKV_OK) {
    pool->decode_routes++;
    if (pool->timing) pool->timed = 1;
  }
  return st;
}

mkv_status paged_attn_set_deterministic(mkv_pool* pool, int32_t enable) {
  if (!pool) return MKV_EINVAL;
  pool->deterministic = enable != 0;
  return MKV_OK;
}

mkv_status paged_attn_set_timing(mkv_pool* pool, int32_t enable) {
  if (!pool) return MKV_EINVAL;
  if (enable && !pool->timing) {
    for (int i = 0; i < 4; ++i) {
      if (hipEventCreate(&pool->timing_ev[i]) != hipSuccess) {
        for (int k = 0; k < i; ++k) (void)hipEventDestroy(pool->timing_ev[k]);
        return MKV_EHIP;
      }
    }
    pool->timing = 1;
    pool->timed = 0;
  } else if (!enable && pool->timing) {
    for (int i = 0; i < 4; ++i) (void)hipEventDestroy(pool->timing_ev[i]);
    pool->timing = pool->timed = 0;
  }
  return MKV_OK;
}

mkv_status paged_attn_last_times(mkv_pool* pool, float* scan_us, float* merge_us) {
  if (!pool || !scan_us || !merge_us) return MKV_EINVAL;
  if (!pool->timing || !pool->timed) return MKV_ESTATE;
  float a = 0.0f, b = 0.0f;
  if (hipEventSynchronize(pool->timing_ev[3]) != hipSuccess ||
      hipEventElapsedTime(&a, pool->timing_ev[0], pool->timing_ev[1]) != hipSuccess ||
      hipEventElapsedTime(&b, pool->timing_ev[2], pool->timing_ev[3]) != hipSuccess)
    return MKV_EHIP;
  *scan_us = a * 1000.0f;
  *merge_us = b * 1000.0f;
  return MKV_OK;
}

mkv_status paged_attn_chunk(mkv_pool* pool, int32_t layer, int32_t n_req, const uint16_t* q,
                            const int32_t* cu_q, int32_t n_q_total, const int32_t* block_table,
                            const uint8_t* tags, int32_t max_pages, const int32_t* seq_lens,
                            float* out, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!pool || !q || !cu_q || !block_table || !tags || !seq_lens || !out || !ws) return MKV_EINVAL;
  if (n_req < 1 || max_pages < 1 || n_q_total < 1) return MKV_EINVAL;
  if (!aligned16(q) || !aligned16(out) || !aligned16(ws)) return MKV_EINVAL;
  if (layer < 0 || layer >= pool->n_layers) return MKV_ERANGE;
  if (n_req > 65535 || max_pages > 1024 * 256) return MKV_ERANGE;
  if ((int64_t)n_q_total * pool->group > ((int64_t)1 << 31) / 2) return MKV_ERANGE;
  if (ws_bytes < chunk_ws_bytes(n_req, max_pages, n_q_total, pool->n_kv_heads, pool->group, pool->d))
    return MKV_ENOMEM;
  hipError_t e = launch_chunk(view_of(pool), layer, n_req, q, cu_q, n_q_total, block_table, tags,
                              max_pages, seq_lens, out, ws, stream);
  if (e == hipErrorNotSupported) return MKV_EUNSUP;
  mkv_status st = hip_status(e);
  if (st == MKV_OK) pool->chunk_routes++;
  return st;
}

mkv_status paged_attn_decode_cohort_key(const mkv_pool* pool, int32_t n_req, int32_t max_pages,
                                        int32_t fused_append, int32_t scoring, uint64_t* key) {
  if (!pool || !key || n_req < 1 || max_pages < 1) return MKV_EINVAL;
  if (n_req > 65535 || max_pages > 1024 * 256) return MKV_ERANGE;
  if (pool->n_tq3 < 1 || pool->timing) return MKV_ESTATE;
  const DecodeShape sh = decode_shape(n_req, max_pages, pool->n_kv_heads, pool->recent);
  const uint64_t fields[] = {(uint64_t)(uintptr_t)pool, (uint64_t)(uintptr_t)pool->ctrl,
                             (uint64_t)pool->n_layers, (uint64_t)pool->n_q_heads,
                             (uint64_t)pool->n_kv_heads, (uint64_t)pool->d, (uint64_t)PAGE,
                             (uint64_t)pool->n_fp8, (uint64_t)pool->n_tq3, (uint64_t)pool->recent,
                             (uint64_t)n_req, (uint64_t)max_pages, (uint64_t)sh.cunits,
                             (uint64_t)sh.max_chunks, (uint64_t)(fused_append != 0),
                             (uint64_t)(scoring != 0), (uint64_t)pool->deterministic,
                             0x4d4b5632ull /* key format */};
  uint64_t h = 1469598103934665603ull;  // FNV-1a over the fields' bytes
  for (uint64_t f : fields)
    for (int b = 0; b < 8; ++b) {
      h ^= (f >> (8 * b)) & 0xFFu;
      h *= 1099511628211ull;
    }
  *key = h;
  return MKV_OK;
}

mkv_status kv_partition_pages(int32_t n_req, const int32_t* block_table, const uint8_t* tags,
                              int32_t max_pages, const int32_t* seq_lens, int32_t* list8,
                              int32_t* list3, int32_t* counts, hipStream_t stream) {
  if (!block_table || !tags || !seq_lens || !list8 || !list3 || !counts) return MKV_EINVAL;
  if (n_req < 1 || max_pages < 1) return MKV_EINVAL;
  return hip_status(launch_partition(n_req, block_table, tags, max_pages, seq_lens, list8, list3,
                                     counts, nullptr, stream));
}

mkv_status kv_pool_free_counts(mkv_pool* pool, int32_t* n_fp8_free, int32_t* n_tq3_free) {
  if (!pool) return MKV_EINVAL;
  int32_t hdr[2];
  if (hipDeviceSynchronize() != hipSuccess) return MKV_EHIP;
  if (hipMemcpy(hdr, pool->ctrl, sizeof(hdr), hipMemcpyDeviceToHost) != hipSuccess) return MKV_EHIP;
  if (n_fp8_free) *n_fp8_free = hdr[CTRL_FP8_TOP];
  if (n_tq3_free) *n_tq3_free = hdr[CTRL_TQ3_TOP];
  return MKV_OK;
}

mkv_status kv_pool_read_free_lists(mkv_pool* pool, int32_t* fp8_ids, int32_t* n_fp8,
                                   int32_t* tq3_ids, int32_t* n_tq3) {
  if (!pool) return MKV_EINVAL;
  int32_t t8, t3;
  mkv_status st = kv_pool_free_counts(pool, &t8, &t3);
  if (st != MKV_OK) return st;
  if (n_fp8) *n_fp8 = t8;
  if (n_tq3) *n_tq3 = t3;
  if (fp8_ids && t8 > 0 &&
      hipMemcpy(fp8_ids, pool->ctrl + pool->cl.fp8_stack, (size_t)t8 * 4, hipMemcpyDeviceToHost) !=
          hipSuccess)
    return MKV_EHIP;
  if (tq3_ids && t3 > 0 &&
      hipMemcpy(tq3_ids, pool->ctrl + pool->cl.tq3_stack, (size_t)t3 * 4, hipMemcpyDeviceToHost) !=
          hipSuccess)
    return MKV_EHIP;
  return MKV_OK;
}

mkv_status kv_pool_counters(mkv_pool* pool, mkv_counters* out) {
  if (!pool || !out) return MKV_EINVAL;
  int32_t f8, f3;
  mkv_status st = kv_pool_free_counts(pool, &f8, &f3);
  if (st != MKV_OK) return st;
  std::memset(out, 0, sizeof(*out));
  out->decode_routes = pool->decode_routes;
  out->chunk_routes = pool->chunk_routes;
  out->fallbacks = 0;
  out->dense_shadow_bytes = 0;
  out->fp8_pages_live = (uint64_t)(pool->n_fp8 - f8);
  out->tq3_pages_live = (uint64_t)(pool->n_tq3 - f3);
  const uint64_t per = (uint64_t)pool->n_layers * pool->n_kv_heads;
  out->fp8_bytes_live = out->fp8_pages_live * per * (uint64_t)(fp8_region_bytes(pool->d) + 8);
  out->tq3_bytes_live = out->tq3_pages_live * per * (uint64_t)tq3_region_bytes(pool->d);
  return MKV_OK;
}

mkv_status mkv_stream_read(const void* buf, size_t bytes, uint32_t* sink, hipStream_t stream) {
  if (!buf || !sink || !aligned16(buf) || bytes % 16 != 0) return MKV_EINVAL;
  if (bytes == 0) return MKV_OK;
  return hip_status(launch_stream_read(buf, bytes, sink, MKV_STREAM_PROBE_WORKGROUPS, stream));
}

static mkv_status control_geometry(int32_t n_kv_heads, int32_t n_q_heads, int32_t head_dim) {
  if (n_kv_heads < 1 || n_q_heads < 1 || n_q_heads % n_kv_heads) return MKV_EINVAL;
  if (head_dim != 128 && head_dim != 256) return MKV_EUNSUP;
  if (n_q_heads / n_kv_heads > 16) return MKV_EUNSUP;
  return MKV_OK;
}

mkv_status mkv_control_bf16_write(uint16_t* pages, int32_t n_pages, int32_t n_layers,
                                  int32_t n_kv_heads, int32_t head_dim, int32_t layer,
                                  int32_t n_req, const int32_t* block_table, int32_t max_pages,
                                  const int32_t* seq_lens_before, const int32_t* cu_new_tokens,
                                  int32_t n_new_total, const uint16_t* k, const uint16_t* v,
                                  hipStream_t stream) {
  if (!pages || !block_table || !seq_lens_before || !cu_new_tokens) return MKV_EINVAL;
  if (n_pages < 1 || n_layers < 1 || n_req < 1 || max_pages < 1 || n_new_total < 0) return MKV_EINVAL;
  if (n_new_total > 0 && (!k || !v)) return MKV_EINVAL;
  mkv_status st = control_geometry(n_kv_heads, n_kv_heads, head_dim);
  if (st != MKV_OK) return st;
  if (layer < 0 || layer >= n_layers || n_new_total > (1 << 30)) return MKV_ERANGE;
  if (!aligned16(pages)) return MKV_EINVAL;
  return hip_status(launch_control_bf16_write(pages, n_pages, n_kv_heads, head_dim, layer, n_req,
                                              block_table, max_pages, seq_lens_before,
                                              cu_new_tokens, n_new_total, k, v, stream));
}

mkv_status mkv_control_bf16_workspace_bytes(int32_t n_req, int32_t max_pages, int32_t n_kv_heads,
                                            int32_t n_q_heads, int32_t head_dim, size_t* bytes) {
  if (!bytes || n_req < 1 || max_pages < 1) return MKV_EINVAL;
  mkv_status st = control_geometry(n_kv_heads, n_q_heads, head_dim);
  if (st != MKV_OK) return st;
  *bytes = control_bf16_ws_bytes(n_req, max_pages, n_kv_heads, n_q_heads / n_kv_heads, head_dim);
  return MKV_OK;
}

mkv_status mkv_control_bf16_decode(const uint16_t* pages, int32_t n_pages, int32_t n_layers,
                                   int32_t n_kv_heads, int32_t n_q_heads, int32_t head_dim,
                                   int32_t layer, int32_t n_req, const uint16_t* q,
                                   const int32_t* block_table, int32_t max_pages,
                                   const int32_t* seq_lens, float* out, float* lse, void* ws,
                                   size_t ws_bytes, hipStream_t stream) {
  if (!pages || !q || !block_table || !seq_lens || !out || !ws) return MKV_EINVAL;
  if (n_pages < 1 || n_layers < 1 || n_req < 1 || max_pages < 1) return MKV_EINVAL;
  mkv_status st = control_geometry(n_kv_heads, n_q_heads, head_dim);
  if (st != MKV_OK) return st;
  if (layer < 0 || layer >= n_layers) return MKV_ERANGE;
  if (n_req > 65535 || max_pages > 1024 * 256) return MKV_ERANGE;
  if (!aligned16(pages) || !aligned16(q) || !aligned16(out) || !aligned16(ws)) return MKV_EINVAL;
  if (ws_bytes < control_bf16_ws_bytes(n_req, max_pages, n_kv_heads, n_q_heads / n_kv_heads, head_dim))
    return MKV_ENOMEM;
  return hip_status(launch_control_bf16_decode(pages, n_pages, n_kv_heads, n_q_heads / n_kv_heads,
                                               head_dim, layer, n_req, q, block_table, max_pages,
                                               seq_lens, out, lse, ws, stream));
}

mkv_status mkv_fp64_probe(const double* a, const double* b, int64_t n, double* quot, double* root,
                          uint16_t* half, hipStream_t stream) {
  if (!a || !b || !quot || !root || !half || n < 0) return MKV_EINVAL;
  if (n == 0) return MKV_OK;
  return hip_status(launch_fp64_probe(a, b, n, quot, root, half, stream));
}

mkv_status kv_pool_check_errors(mkv_pool* pool, uint32_t* err_word, int32_t clear) {
  if (!pool) return MKV_EINVAL;
  if (hipDeviceSynchronize() != hipSuccess) return MKV_EHIP;
  int32_t e;
  if (hipMemcpy(&e, pool->ctrl + CTRL_ERR, 4, hipMemcpyDeviceToHost) != hipSuccess) return MKV_EHIP;
  if (err_word) *err_word = (uint32_t)e;
  if (clear) {
    int32_t z = 0;
    if (hipMemcpy(pool->ctrl + CTRL_ERR, &z, 4, hipMemcpyHostToDevice) != hipSuccess) return MKV_EHIP;
  }
  return MKV_OK;
}

}  // extern "C"
