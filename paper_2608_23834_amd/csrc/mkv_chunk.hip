// Causal chunked-prefill attention over mixed FP8/TQ3 pages (MFMA).
#include <hip/hip_runtime.h>

#include "mkv_internal.h"
#include "../../include/minima_kv.h"

namespace mkv {

size_t chunk_ws_bytes(int n_req, int max_pages, int n_q_total, int n_kv_heads, int group, int d) {
  (void)n_req; (void)max_pages; (void)n_q_total; (void)n_kv_heads; (void)group; (void)d;
  return 256;
}

hipError_t launch_chunk(const PoolView&, int, int, const uint16_t*, const int32_t*, int,
                        const int32_t*, const uint8_t*, int, const int32_t*, float*, void*,
                        hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace mkv
