// Dense bf16 control for the decode benchmark (the dense control of the
// paper's fused-decode canary, Sec. 6.3): the same logical KV held as bf16
// pages, attended by a plain paged decode kernel, so the mixed FP8/TQ3 path
// can be timed against an uncompressed cache of the same shape.  Not part of
// the method: measurement only.
//
// Page-head layout (bf16 bits, 2*16*d values): K token-major [16][d], then V
// in 4-token groups per channel -- V(t, c) at 16 d + ((t/4) d + c) 4 + t%4 --
// so that each lane's MFMA operands are one contiguous load.
//
// Decode: grid (chunk, KV head, request), 256 threads; each wave walks every
// fourth page of its chunk with the next page's loads in flight while the
// current one is computed:
//   S = K Q^T on v_mfma_f32_16x16x32_bf16 (M = 16 tokens, N = query heads,
//       K = 32 channels), scores scaled by log2(e)/sqrt(d) in fp32;
//   online softmax per head in base 2 (one head per lane column, so the
//       rescale is a per-lane factor);
//   O^T += V^T P on v_mfma_f32_16x16x16bf16_1k (M = 16 channels, N = heads,
//       K = the page's 16 tokens): the score tile's lane layout is exactly
//       the weight operand's, and the weights go in as a bf16 hi + lo pair.
// Each wave writes its own normalized partial (O, m, l); a merge kernel folds
// them (Eq. softmax-merge).
#include <hip/hip_runtime.h>

#include "mkv_internal.h"
#include "../../include/minima_kv.h"

namespace mkv {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

constexpr int CW_WAVES = 4;

struct CtlShape {
  int ppc, max_chunks;  // pages per chunk, chunks per (request, KV head)
};

CtlShape ctl_shape(int n_req, int max_pages, int n_kv_heads) {
  CtlShape s;
  const int64_t pairs = (int64_t)n_req * n_kv_heads;
  int64_t ppc = ((int64_t)max_pages * pairs + 511) / 512;  // ~512 workgroups in all
  if (ppc < 4 * CW_WAVES) ppc = 4 * CW_WAVES;
  s.ppc = (int)ppc;
  s.max_chunks = (int)((max_pages + ppc - 1) / ppc);
  return s;
}

template <int G>
constexpr int ctl_part_floats(int D) {
  return G * D + 2 * G;
}

__device__ __forceinline__ uint32_t bf16_hi_lo(float p, uint32_t* lo_bits) {
  // hi = bf16(p) round to nearest even, lo = bf16(p - hi)
  const uint32_t u = __float_as_uint(p);
  const uint32_t hi = (u + 0x7FFFu + ((u >> 16) & 1u)) & 0xFFFF0000u;
  const float r = p - __uint_as_float(hi);
  const uint32_t ur = __float_as_uint(r);
  *lo_bits = ((ur + 0x7FFFu + ((ur >> 16) & 1u)) >> 16) & 0xFFFFu;
  return hi >> 16;
}

struct CtlArgs {
  const uint16_t* pages;
  int n_pages, H, G, layer, n_req, max_pages;
  const uint16_t* q;
  const int32_t* bt;
  const int32_t* seq_lens;
  float* part;
  int ppc, max_chunks;
  float sm_log2;
};

// One wave's page loads: K operands (NS x 16 bytes), V operands (D/16 x 8 bytes).
template <int D>
struct PageRegs {
  uint4 k[D / 32];
  uint2 v[D / 16];
};

template <int D>
__device__ __forceinline__ void load_page(PageRegs<D>& pr, const uint16_t* base, int lane) {
  const uint8_t* b = reinterpret_cast<const uint8_t*>(base);
  const int row = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int s = 0; s < D / 32; ++s)
    pr.k[s] = *reinterpret_cast<const uint4*>(b + row * D * 2 + 64 * s + 16 * grp);
  const uint8_t* vb = b + 16 * D * 2;
#pragma unroll
  for (int m = 0; m < D / 16; ++m)
    pr.v[m] = *reinterpret_cast<const uint2*>(vb + ((size_t)grp * D + 16 * m + row) * 8);
}

// One page of a wave: scores, online softmax, PV.  acc/m_run/l_run as below.
template <int D>
__device__ __forceinline__ void page_step(const PageRegs<D>& pg, const uint8_t* qlds, int lane,
                                          int tok0, int S, bool bad, float sm_log2, float4* acc,
                                          float& m_run, float& l_run) {
  constexpr int NS = D / 32, NT = D / 16;
  typedef float f4v __attribute__((ext_vector_type(4)));
  const int col = lane & 15, grp = lane >> 4;
  f4v c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const uint4 qv = *reinterpret_cast<const uint4*>(qlds + (col * D + 32 * s + 8 * grp) * 2);
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pg.k[s]),
                                                __builtin_bit_cast(bf16x8, qv), c, 0, 0, 0);
  }
  float sv[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) sv[e] = (tok0 + 4 * grp + e < S && !bad) ? c[e] * sm_log2 : -INFINITY;
  float mx = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  if (mx > m_run) {  // per lane: every accumulator entry of lane l belongs to head l % 16
    const float alpha = exp2f(m_run - mx);
    l_run *= alpha;
#pragma unroll
    for (int m = 0; m < NT; ++m) {
      acc[m].x *= alpha;
      acc[m].y *= alpha;
      acc[m].z *= alpha;
      acc[m].w *= alpha;
    }
    m_run = mx;
  }
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float w = exp2f(sv[e] - m_run);
    l_run += w;
    hi[e] = bf16_hi_lo(w, &lo[e]);
  }
  const s16x4 ph = {(short)hi[0], (short)hi[1], (short)hi[2], (short)hi[3]};
  const s16x4 pl = {(short)lo[0], (short)lo[1], (short)lo[2], (short)lo[3]};
#pragma unroll
  for (int m = 0; m < NT; ++m) {
    const s16x4 vv = __builtin_bit_cast(s16x4, pg.v[m]);
    f4v o = {acc[m].x, acc[m].y, acc[m].z, acc[m].w};
    o = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vv, ph, o, 0, 0, 0);
    o = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vv, pl, o, 0, 0, 0);
    acc[m] = make_float4(o[0], o[1], o[2], o[3]);
  }
}

// Two workgroups per CU (<= 256 registers a wave); each wave keeps two pages
// in flight: the loads of its next page are issued, unconditionally (the
// last page is re-read from cache rather than branched around, so the wait
// for the current page counts exactly the newer loads), before the current
// page is computed.
template <int D, int GMAX>
__global__ __launch_bounds__(64 * CW_WAVES, 2) void bf16_decode_kernel(CtlArgs a) {
  const int chunk = blockIdx.x, h = blockIdx.y, r = blockIdx.z;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int G = a.G, H = a.H, mp = a.max_pages;
  const int col = lane & 15, grp = lane >> 4;
  __shared__ __align__(16) uint8_t qlds[16 * D * 2];  // query heads (rows >= G zero), bf16
  for (int i = threadIdx.x; i < 16 * D / 8; i += 64 * CW_WAVES) {
    const int hd = i / (D / 8), c8 = i % (D / 8);
    const uint4 x = hd < G ? *reinterpret_cast<const uint4*>(a.q + ((int64_t)r * H * G + h * G + hd) * D + 8 * c8)
                           : make_uint4(0, 0, 0, 0);
    *reinterpret_cast<uint4*>(qlds + (hd * D + 8 * c8) * 2) = x;
  }
  __syncthreads();
  const int slot = chunk * CW_WAVES + wid;
  float* part = a.part + (((int64_t)r * H + h) * a.max_chunks * CW_WAVES + slot) *
                             ctl_part_floats<GMAX>(D);
  const int S = a.seq_lens[r];
  const int np = (S + PAGE - 1) / PAGE;
  const int p0 = chunk * a.ppc, p1 = min(np, p0 + a.ppc);
  if (S < 1 || np > mp || p0 + wid >= p1) {
    if (lane < G) part[GMAX * D + GMAX + lane] = 0.0f;  // empty partial
    return;
  }
  const int64_t ph_stride = (int64_t)2 * PAGE * D;  // uint16 values per page-head
  const uint16_t* layer_base = a.pages + (int64_t)a.layer * a.n_pages * H * ph_stride;
  const int32_t* btr = a.bt + (int64_t)r * mp;
  auto page_id = [&](int p) { return btr[p]; };
  auto page_base = [&](int id) {
    id = (id < 0 || id >= a.n_pages) ? 0 : id;  // out-of-range ids read page 0, masked
    return layer_base + ((int64_t)id * H + h) * ph_stride;
  };
  float4 acc[D / 16];
#pragma unroll
  for (int m = 0; m < D / 16; ++m) acc[m] = make_float4(0.f, 0.f, 0.f, 0.f);
  float m_run = -1.0e30f, l_run = 0.0f;
  const int last = p0 + wid + (p1 - 1 - p0 - wid) / CW_WAVES * CW_WAVES;  // this wave's last page
  PageRegs<D> A, B;
  int p = p0 + wid;
  int idA = page_id(p);
  load_page<D>(A, page_base(idA), lane);
  for (;;) {
    const int pb = min(p + CW_WAVES, last);
    const int idB = page_id(pb);
    load_page<D>(B, page_base(idB), lane);
    page_step<D>(A, qlds, lane, p * PAGE, S, idA < 0 || idA >= a.n_pages, a.sm_log2, acc, m_run, l_run);
    p += CW_WAVES;
    if (p > last) break;
    const int pa = min(p + CW_WAVES, last);
    idA = page_id(pa);
    load_page<D>(A, page_base(idA), lane);
    page_step<D>(B, qlds, lane, p * PAGE, S, idB < 0 || idB >= a.n_pages, a.sm_log2, acc, m_run, l_run);
    p += CW_WAVES;
    if (p > last) break;
  }
  // lane l holds channels 16 m + 4 grp + e of head col; l_run over its tokens
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  if (col < G) {
    const float inv = l_run > 0.0f ? 1.0f / l_run : 0.0f;
#pragma unroll
    for (int m = 0; m < D / 16; ++m)
      *reinterpret_cast<float4*>(part + col * D + 16 * m + 4 * grp) =
          make_float4(acc[m].x * inv, acc[m].y * inv, acc[m].z * inv, acc[m].w * inv);
    if (grp == 0) {
      part[GMAX * D + col] = m_run;
      part[GMAX * D + GMAX + col] = l_run;
    }
  }
}

// Eq. softmax-merge over every wave partial of a (request, KV head): one
// 4-wave workgroup per (query head of the group, KV head, request); each wave
// merges a quarter of the slots and the four results are merged in LDS.  Per
// batch of 64 slots the (m_j, l_j) are read at once (one per lane), the batch
// maximum and weights 2^(m_j - M) l_j come from wave reductions, and each
// thread folds its channels of the weighted O rows of 16 slots at a time with
// independent loads; empty slots (l_j = 0) are skipped, their O rows never
// read.
template <int D, int GMAX>
__global__ __launch_bounds__(256) void bf16_merge_kernel(int G, int H, int n_slots, const float* part,
                                                        float* out, float* lse) {
  constexpr int CPT = D / 64;  // channels per thread
  constexpr int GRP = 16;      // slots whose O rows one lane loads at once
  __shared__ float s_m[4], s_l[4], s_o[4][D];
  const int n = blockIdx.x, h = blockIdx.y, r = blockIdx.z;
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float* base = part + ((int64_t)r * H + h) * n_slots * ctl_part_floats<GMAX>(D);
  // wave wv merges the slots [k_lo, k_hi), 64 at a time
  const int quarter = (n_slots + 3) / 4;
  const int k_lo = wv * quarter, k_hi = min(n_slots, k_lo + quarter);
  float M = -INFINITY, L = 0.0f;
  float o[CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) o[i] = 0.0f;
  for (int k0 = k_lo; k0 < k_hi; k0 += 64) {
    const int k = k0 + lane;
    const float* pk = base + (int64_t)min(k, n_slots - 1) * ctl_part_floats<GMAX>(D);
    const float lj = k < k_hi ? pk[GMAX * D + GMAX + n] : 0.0f;
    const float mj = lj > 0.0f ? pk[GMAX * D + n] : -INFINITY;
    float mb = mj;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mb = fmaxf(mb, __shfl_xor(mb, off, 64));
    if (mb == -INFINITY) continue;  // nothing in this batch (wave-uniform)
    const float Mn = fmaxf(M, mb);
    const float f = M == -INFINITY ? 0.0f : exp2f(M - Mn);
    const float wj = lj > 0.0f ? exp2f(mj - Mn) * lj : 0.0f;
    float ws = wj;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) ws += __shfl_xor(ws, off, 64);
    L = L * f + ws;
#pragma unroll
    for (int i = 0; i < CPT; ++i) o[i] *= f;
    const int nb = min(64, k_hi - k0);
    for (int j0 = 0; j0 < nb; j0 += GRP) {
      float w8[GRP], x8[GRP][CPT];
#pragma unroll
      for (int j = 0; j < GRP; ++j) {
        w8[j] = __shfl(wj, min(j0 + j, 63), 64);
        const float* pj = base + (int64_t)(k0 + min(j0 + j, nb - 1)) * ctl_part_floats<GMAX>(D) + n * D;
#pragma unroll
        for (int i = 0; i < CPT; ++i) x8[j][i] = w8[j] != 0.0f && j0 + j < nb ? pj[lane + 64 * i] : 0.0f;
      }
#pragma unroll
      for (int j = 0; j < GRP; ++j)
#pragma unroll
        for (int i = 0; i < CPT; ++i) o[i] = fmaf(w8[j], x8[j][i], o[i]);
    }
    M = Mn;
  }
  // the four waves' (M, L, O) into one
  if (lane == 0) {
    s_m[wv] = M;
    s_l[wv] = L;
  }
#pragma unroll
  for (int i = 0; i < CPT; ++i) s_o[wv][lane + 64 * i] = o[i];
  __syncthreads();
  if (wv != 0) return;
  float Mt = -INFINITY;
#pragma unroll
  for (int w = 0; w < 4; ++w) Mt = fmaxf(Mt, s_l[w] > 0.0f ? s_m[w] : -INFINITY);
  float Lt = 0.0f, ot[CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) ot[i] = 0.0f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (!(s_l[w] > 0.0f)) continue;  // an empty wave's O is zero, but skip it anyway
    const float f = exp2f(s_m[w] - Mt);
    Lt = fmaf(s_l[w], f, Lt);
#pragma unroll
    for (int i = 0; i < CPT; ++i) ot[i] = fmaf(f, s_o[w][lane + 64 * i], ot[i]);
  }
  const int64_t row = (int64_t)r * H * G + h * G + n;
  const float inv = Lt > 0.0f ? 1.0f / Lt : 0.0f;
#pragma unroll
  for (int i = 0; i < CPT; ++i) out[row * D + lane + 64 * i] = Lt > 0.0f ? ot[i] * inv : 0.0f;
  if (lse && lane == 0) lse[row] = Lt > 0.0f ? (Mt + log2f(Lt)) * 0.69314718055994531f : -INFINITY;
}

// Scatter new bf16 K/V rows into their pages: one workgroup of d threads per
// (new token, KV head).
template <int D>
__global__ __launch_bounds__(D) void bf16_write_kernel(uint16_t* pages, int n_pages, int H, int layer,
                                                       int n_req, const int32_t* bt, int max_pages,
                                                       const int32_t* sb, const int32_t* cu,
                                                       const uint16_t* k, const uint16_t* v) {
  const int row = blockIdx.x, h = blockIdx.y, c = threadIdx.x;
  int lo = 0, hi = n_req - 1;  // request of this row: cu[req] <= row < cu[req + 1]
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= row) lo = mid; else hi = mid - 1;
  }
  const int req = lo;
  const int pos = sb[req] + (row - cu[req]);
  const int p = pos / PAGE, u = pos % PAGE;
  if (pos < 0 || p >= max_pages) return;
  const int id = bt[(int64_t)req * max_pages + p];
  if (id < 0 || id >= n_pages) return;
  uint16_t* ph = pages + (((int64_t)layer * n_pages + id) * H + h) * 2 * PAGE * D;
  const int64_t src = ((int64_t)row * H + h) * D + c;
  ph[u * D + c] = k[src];
  ph[PAGE * D + ((u / 4) * D + c) * 4 + (u % 4)] = v[src];
}

}  // namespace

size_t control_bf16_ws_bytes(int n_req, int max_pages, int n_kv_heads, int group, int d) {
  const CtlShape s = ctl_shape(n_req, max_pages, n_kv_heads);
  const int gmax = group <= 8 ? 8 : 16;
  return (size_t)n_req * n_kv_heads * s.max_chunks * CW_WAVES * (gmax * d + 2 * gmax) * sizeof(float);
}

hipError_t launch_control_bf16_write(uint16_t* pages, int n_pages, int H, int d, int layer, int n_req,
                                     const int32_t* bt, int max_pages, const int32_t* sb,
                                     const int32_t* cu, int n_new, const uint16_t* k,
                                     const uint16_t* v, hipStream_t s) {
  if (n_new == 0) return hipSuccess;
  dim3 grid(n_new, H);
  if (d == 256)
    hipLaunchKernelGGL(bf16_write_kernel<256>, grid, dim3(256), 0, s, pages, n_pages, H, layer, n_req,
                       bt, max_pages, sb, cu, k, v);
  else
    hipLaunchKernelGGL(bf16_write_kernel<128>, grid, dim3(128), 0, s, pages, n_pages, H, layer, n_req,
                       bt, max_pages, sb, cu, k, v);
  return hipGetLastError();
}

hipError_t launch_control_bf16_decode(const uint16_t* pages, int n_pages, int H, int G, int d,
                                      int layer, int n_req, const uint16_t* q, const int32_t* bt,
                                      int max_pages, const int32_t* seq_lens, float* out,
                                      float* lse, void* ws, hipStream_t s) {
  const CtlShape sh = ctl_shape(n_req, max_pages, H);
  CtlArgs a;
  a.pages = pages;
  a.n_pages = n_pages;
  a.H = H;
  a.G = G;
  a.layer = layer;
  a.n_req = n_req;
  a.max_pages = max_pages;
  a.q = q;
  a.bt = bt;
  a.seq_lens = seq_lens;
  a.part = reinterpret_cast<float*>(ws);
  a.ppc = sh.ppc;
  a.max_chunks = sh.max_chunks;
  a.sm_log2 = 1.4426950408889634f / sqrtf((float)d);
  const dim3 grid(sh.max_chunks, H, n_req), block(64 * CW_WAVES);
  const dim3 mgrid(G, H, n_req);
  const int n_slots = sh.max_chunks * CW_WAVES;
  const float* part = a.part;
  if (d == 256 && G <= 8) {
    hipLaunchKernelGGL((bf16_decode_kernel<256, 8>), grid, block, 0, s, a);
    hipLaunchKernelGGL((bf16_merge_kernel<256, 8>), mgrid, dim3(256), 0, s, G, H, n_slots, part, out, lse);
  } else if (d == 256) {
    hipLaunchKernelGGL((bf16_decode_kernel<256, 16>), grid, block, 0, s, a);
    hipLaunchKernelGGL((bf16_merge_kernel<256, 16>), mgrid, dim3(256), 0, s, G, H, n_slots, part, out, lse);
  } else if (G <= 8) {
    hipLaunchKernelGGL((bf16_decode_kernel<128, 8>), grid, block, 0, s, a);
    hipLaunchKernelGGL((bf16_merge_kernel<128, 8>), mgrid, dim3(256), 0, s, G, H, n_slots, part, out, lse);
  } else {
    hipLaunchKernelGGL((bf16_decode_kernel<128, 16>), grid, block, 0, s, a);
    hipLaunchKernelGGL((bf16_merge_kernel<128, 16>), mgrid, dim3(256), 0, s, G, H, n_slots, part, out, lse);
  }
  return hipGetLastError();
}

}  // namespace mkv
