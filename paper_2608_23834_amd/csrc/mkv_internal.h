// Host-side pool handle and the launchers each kernel translation unit
// exports to the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mkv_device.h"

struct mkv_pool {
  int n_layers, n_q_heads, n_kv_heads, d, group, n_fp8, n_tq3, recent;
  uint8_t* fp8;       // device
  float* fp8_scales;  // device
  uint8_t* tq3;       // device
  int32_t* ctrl;      // device
  mkv::CtrlLayout cl;
  uint64_t decode_routes, chunk_routes;
  hipEvent_t timing_ev[4];  // scan start and end, merge start and end (timing on)
  int timing, timed;
  int deterministic;  // decode with a fixed stage schedule
};

namespace mkv {

struct PoolView {
  uint8_t* fp8;
  float* fp8_scales;
  uint8_t* tq3;
  int32_t* ctrl;
  const int8_t* sigma;
  int32_t* fp8_stack;
  int32_t* tq3_stack;
  int32_t* list;
  int32_t* rc8;  // references per FP8 page
  int32_t* rc3;  // references per TQ3 page
  int32_t* occ8;
  int32_t* occ3;
  int32_t* last8;
  int32_t* last3;
  int n_layers, n_kv_heads, d, group, n_fp8, n_tq3, recent;
  int deterministic;  // decode: fixed stage schedule instead of run-time claiming
};

inline PoolView view_of(const mkv_pool* p) {
  PoolView v;
  v.fp8 = p->fp8;
  v.fp8_scales = p->fp8_scales;
  v.tq3 = p->tq3;
  v.ctrl = p->ctrl;
  v.sigma = reinterpret_cast<const int8_t*>(reinterpret_cast<const uint8_t*>(p->ctrl) + p->cl.sigma_bytes);
  v.fp8_stack = p->ctrl + p->cl.fp8_stack;
  v.tq3_stack = p->ctrl + p->cl.tq3_stack;
  v.list = p->ctrl + p->cl.list;
  v.rc8 = p->ctrl + p->cl.rc8;
  v.rc3 = p->ctrl + p->cl.rc3;
  v.occ8 = p->ctrl + p->cl.occ8;
  v.occ3 = p->ctrl + p->cl.occ3;
  v.last8 = p->ctrl + p->cl.last8;
  v.last3 = p->ctrl + p->cl.last3;
  v.n_layers = p->n_layers;
  v.n_kv_heads = p->n_kv_heads;
  v.d = p->d;
  v.group = p->group;
  v.n_fp8 = p->n_fp8;
  v.n_tq3 = p->n_tq3;
  v.recent = p->recent;
  v.deterministic = p->deterministic;
  return v;
}

// mkv_pool_kernels.hip
hipError_t launch_append(const PoolView& P, int layer, int n_req, int32_t* bt, uint8_t* tags,
                         int max_pages, const int32_t* seq_before, const int32_t* cu_new,
                         int n_new_total, const uint16_t* k, const uint16_t* v, hipStream_t s);
hipError_t launch_migrate(const PoolView& P, int n_req, int32_t* bt, uint8_t* tags, int max_pages,
                          const uint8_t* anchor, const int32_t* seq_lens, hipStream_t s);
hipError_t launch_promote(const PoolView& P, int n_req, int32_t* bt, uint8_t* tags, int max_pages,
                          const uint8_t* mask, const int32_t* seq_lens, hipStream_t s);
hipError_t launch_partition(int n_req, const int32_t* bt, const uint8_t* tags, int max_pages,
                            const int32_t* seq_lens, int32_t* list8, int32_t* list3,
                            int32_t* counts, int32_t* err, hipStream_t s);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);
hipError_t launch_fp64_probe(const double* a, const double* b, int64_t n, double* quot,
                             double* root, uint16_t* half, hipStream_t s);

hipError_t launch_pages_acquire(const PoolView& P, int n, const int32_t* ids, const uint8_t* tags,
                                hipStream_t s);
hipError_t launch_pages_release(const PoolView& P, int n, const int32_t* ids, const uint8_t* tags,
                                int n_fin, const int32_t* reqs, int n_req, int32_t* bt,
                                uint8_t* bt_tags, int max_pages, hipStream_t s);

// mkv_decode.hip
struct DecodeShape {
  int cunits, max_chunks;
};
DecodeShape decode_shape(int n_req, int max_pages, int n_kv_heads, int recent);
size_t decode_ws_bytes(int n_req, int max_pages, int n_kv_heads, int group, int d, int recent);
// the fixed device scratch of paged_attn_decode_noalloc: resolve its address on
// device dev (dev must be current; once per device), and look it up
hipError_t decode_scratch_init(int dev);
hipError_t decode_scratch(int dev, void** ptr);
hipError_t launch_decode(const PoolView& P, int layer, int n_req, const uint16_t* q,
                         const int32_t* bt, const uint8_t* tags, int max_pages,
                         const int32_t* seq_lens, float* out, float* lse, void* ws,
                         hipStream_t s, hipEvent_t* ev, const uint16_t* k_new = nullptr,
                         const uint16_t* v_new = nullptr, int32_t* bt_w = nullptr,
                         uint8_t* tags_w = nullptr, float2* page_mass = nullptr);
hipError_t launch_score_collect(int n_req, int n_q_heads, int max_pages, const int32_t* seq_lens,
                                const float* lse, const float2* page_mass,
                                const uint8_t* head_mask, float beta, float* a_io, float* r_out,
                                float* qn_out, hipStream_t s);

// mkv_control.hip (dense bf16 control, measurement only)
size_t control_bf16_ws_bytes(int n_req, int max_pages, int n_kv_heads, int group, int d);
hipError_t launch_control_bf16_write(uint16_t* pages, int n_pages, int H, int d, int layer, int n_req,
                                     const int32_t* bt, int max_pages, const int32_t* sb,
                                     const int32_t* cu, int n_new, const uint16_t* k,
                                     const uint16_t* v, hipStream_t s);
hipError_t launch_control_bf16_decode(const uint16_t* pages, int n_pages, int H, int G, int d,
                                      int layer, int n_req, const uint16_t* q, const int32_t* bt,
                                      int max_pages, const int32_t* seq_lens, float* out,
                                      float* lse, void* ws, hipStream_t s);

// mkv_probe.hip
hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, int n_wg, hipStream_t s);

// mkv_chunk.hip
size_t chunk_ws_bytes(int n_req, int max_pages, int n_q_total, int n_kv_heads, int group, int d);
hipError_t launch_chunk(const PoolView& P, int layer, int n_req, const uint16_t* q,
                        const int32_t* cu_q, int n_q_total, const int32_t* bt,
                        const uint8_t* tags, int max_pages, const int32_t* seq_lens, float* out,
                        void* ws, hipStream_t s);

}  // namespace mkv
