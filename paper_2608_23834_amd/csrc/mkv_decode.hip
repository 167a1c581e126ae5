// Mixed-format paged decode attention (Sec. 3.3, Eq. softmax-merge; Sec. 4.1
// direct fused decode) for gfx950.
//
// One launch per layer.  Grid (chunk, KV head, request); 256 threads = 4
// wave64s.  Each workgroup
//  1. partitions the request's logical pages by format (Sec. 4.1 compact
//     per-format lists, stable, logical order kept) and takes one chunk of
//     either the FP8 list (Recent/Anchor) or the TQ3 list (Stale): format is
//     uniform per workgroup, so both scans are branch-free;
//  2. loads the GQA group's queries once; for TQ3 it rotates them (q_rot =
//     R q, exact algebra since k_hat = gamma R^T mu_c) so keys are never
//     de-rotated;
//  3. each wave walks page pairs: QK^T on MFMA 16x16x32 f16 (M = 16 tokens of
//     a page, N = the group's query heads, K = 32 channels), the 3-bit codes
//     turned into E4M3 codebook bytes by one v_perm per 4 codes and into fp16
//     by the hardware converter; online softmax in base 2; PV on MFMA with
//     M = 16 channels, N = heads, K = 32 tokens (two pages), values
//     dequantized in registers (TQ3: zero + scale * code per channel);
//  4. the four waves merge in LDS into one (m_j, l_j, O_j) partial per chunk.
// A second kernel merges all partials of both formats per (request, query
// head) (Eq. softmax-merge).  The workspace holds O(chunks x heads x d)
// partials, never anything the size of the cache.
#include <hip/hip_runtime.h>

#include "mkv_internal.h"
#include "../../include/minima_kv.h"

namespace mkv {

// tag slices of 1024 pages: max_pages <= 1024 * MAX_SLICES (4M tokens)
constexpr int MAX_SLICES = 256;

struct DecodeArgs {
  PoolView P;
  int layer, n_req, max_pages;
  const uint16_t* q;
  const int32_t* bt;
  const uint8_t* tags;
  const int32_t* seq_lens;
  float* out;
  float* lse;
  int32_t* totals;
  float* partials;
  int c3, c8, max_chunks;
  float sm_log2;  // log2(e) / sqrt(d)
};

DecodeShape decode_shape(int n_req, int max_pages, int n_kv_heads) {
  DecodeShape s;
  // about 512 chunk workgroups per launch (two per CU at two waves per SIMD)
  const int64_t ph = (int64_t)n_req * max_pages * n_kv_heads;
  int c3 = 8;
  while (c3 < 64 && (int64_t)c3 * 512 < ph) c3 *= 2;
  s.c3 = c3;
  s.c8 = c3;
  s.max_chunks = (max_pages + s.c8 - 1) / s.c8 + 2;
  return s;
}

// workspace: int32 chunk count per request, then the partials
static size_t header_bytes(int n_req) { return (((size_t)n_req * 4) + 255) / 256 * 256; }

size_t decode_ws_bytes(int n_req, int max_pages, int n_kv_heads, int group, int d) {
  DecodeShape s = decode_shape(n_req, max_pages, n_kv_heads);
  return header_bytes(n_req) +
         (size_t)n_req * n_kv_heads * s.max_chunks * group * (d + 2) * sizeof(float);
}

__device__ __forceinline__ half8 h8(half2v a, half2v b, half2v c, half2v d) {
  half8 r;
  r[0] = a[0]; r[1] = a[1]; r[2] = b[0]; r[3] = b[1];
  r[4] = c[0]; r[5] = c[1]; r[6] = d[0]; r[7] = d[1];
  return r;
}
__device__ __forceinline__ half2v cvt_lo(uint32_t w) {
  return __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, false);
}
__device__ __forceinline__ half2v cvt_hi(uint32_t w) {
  return __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, true);
}
__device__ __forceinline__ float exp2_safe(float s, float m) {
  return s == -INFINITY ? 0.0f : exp2f(s - m);
}

template <int D>
struct WaveState {
  float4v acc[D / 16];  // rows (page parity, head) x channels, see below
  float m_run;          // running max of this lane's column (base-2 units)
  float l_run;          // partial denominator over this lane's tokens
};

// Online-softmax step: sc[4] are this lane's base-2 scores (tokens 4*lg + i of
// the page that owns column ln).  Weights are returned in place.  The
// accumulator rows 4*lg + i belong to columns 4*lg + i, whose rescale factors
// are fetched from those lanes when the reference max moves.
template <int D>
__device__ __forceinline__ void softmax_step(WaveState<D>& st, float* sc, int lg) {
  float mx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  // lazy rescale: keep the reference max while new scores stay within 2^8
  const bool need = mx > st.m_run + 8.0f;
  if (__any(need)) {
    const float m_new = need ? mx : st.m_run;
    const float alpha = st.m_run == -INFINITY ? 0.0f : exp2f(st.m_run - m_new);
    st.l_run *= alpha;
    st.m_run = m_new;
    float ar[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ar[i] = __shfl(alpha, 4 * lg + i, 64);
#pragma unroll
    for (int m = 0; m < D / 16; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) st.acc[m][i] *= ar[i];
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sc[i] = exp2_safe(sc[i], st.m_run);
    st.l_run += sc[i];
  }
}

// P^T operand of the PV product: row ln = this lane's column; tokens
// (4*lg + j) of page a for j < 4 and of page b for j >= 4 (block-diagonal:
// page-a rows see only page-a tokens).
__device__ __forceinline__ half8 p_operand(const float* p, bool row_is_b) {
  half8 r;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const _Float16 v = (_Float16)p[j];
    r[j] = row_is_b ? (_Float16)0.0f : v;
    r[4 + j] = row_is_b ? v : (_Float16)0.0f;
  }
  return r;
}

template <int D>
__global__ __launch_bounds__(256, 2) void decode_kernel(DecodeArgs a) {
  constexpr int CL = D / 16, NDW = 3 * D / 128, CB = 3 * D / 32, NS = D / 32;
  extern __shared__ float smem[];
  __shared__ int scr[8];
  __shared__ int2 s_list[64];
  __shared__ int s_slice[MAX_SLICES];
  const PoolView& P = a.P;
  const int r = blockIdx.z, h = blockIdx.y, chunk = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int G = P.group, H = P.n_kv_heads, Hq = H * G;
  const int mp = a.max_pages;
  const int S = a.seq_lens[r];

  if (S < 1 || S > mp * PAGE) {
    if (chunk == 0) {
      for (int i = tid; i < G * D; i += 256) a.out[((int64_t)r * Hq + h * G) * D + i] = 0.0f;
      if (a.lse && tid < G) a.lse[(int64_t)r * Hq + h * G + tid] = -INFINITY;
      if (tid == 0 && h == 0) {
        atomicOr(&P.ctrl[CTRL_ERR], (int)MKV_DEVERR_RANGE);
        a.totals[r] = 0;
      }
    }
    return;
  }
  const int np = (S + PAGE - 1) / PAGE;

  // ---- 1. partition the request's pages by format; pick this chunk's pages.
  // Pages are visited in slices of 1024 (4 consecutive tags per thread, so each
  // load instruction is coalesced).  Pass 1 counts FP8 / TQ3 pages per slice;
  // pass 2 re-reads only the slices that hold this chunk's ranks and scans them.
  const uint8_t* trow = a.tags + (int64_t)r * mp;
  const int n_slices = (np + 1023) / 1024;
  {
    for (int i = tid; i < n_slices; i += 256) s_slice[i] = 0;
    __syncthreads();
    int bad = 0;
    for (int it = 0; it < n_slices; ++it) {
      const int p0 = it * 1024 + tid * 4;
      int c8 = 0, c3 = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int p = p0 + b;
        const int tg = p < np ? trow[p] : -1;
        c3 += tg == TAG_S;
        c8 += (tg == TAG_R || tg == TAG_A);
        bad |= (p < np && tg != TAG_S && tg != TAG_R && tg != TAG_A);
      }
      int packed = c8 | (c3 << 16);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) packed += __shfl_xor(packed, o, 64);
      if (lane == 0) atomicAdd(&s_slice[it], packed);
    }
    if (bad && chunk == 0) atomicOr(&P.ctrl[CTRL_ERR], (int)MKV_DEVERR_BAD_TAG);
    __syncthreads();
  }
  int n8 = 0, n3 = 0;
  for (int it = 0; it < n_slices; ++it) {
    n8 += s_slice[it] & 0xFFFF;
    n3 += s_slice[it] >> 16;
  }
  const int nch8 = (n8 + a.c8 - 1) / a.c8, nch3 = (n3 + a.c3 - 1) / a.c3;
  const int total = nch8 + nch3;
  if (chunk == 0 && h == 0 && tid == 0) a.totals[r] = total;
  if (chunk >= total) return;
  const bool is8 = chunk < nch8;
  const int lo = is8 ? chunk * a.c8 : (chunk - nch8) * a.c3;
  const int hi = min(lo + (is8 ? a.c8 : a.c3), is8 ? n8 : n3);
  {
    const int32_t* brow = a.bt + (int64_t)r * mp;
    const int n_ids = is8 ? P.n_fp8 : P.n_tq3;
    int base = 0;
    for (int it = 0; it < n_slices; ++it) {
      const int cnt = is8 ? (s_slice[it] & 0xFFFF) : (s_slice[it] >> 16);
      if (base < hi && base + cnt > lo) {  // uniform across the workgroup
        const int p0 = it * 1024 + tid * 4;
        int tg4[4], c = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int p = p0 + b;
          const int tg = p < np ? trow[p] : -1;
          tg4[b] = is8 ? (tg == TAG_R || tg == TAG_A) : (tg == TAG_S);
          c += tg4[b];
        }
        int tot;
        int rank = base + block_excl_scan(c, scr, &tot);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          if (tg4[b]) {
            if (rank >= lo && rank < hi) {
              const int p = p0 + b;
              int id = brow[p], lp = p;
              if (id < 0 || id >= n_ids) {
                // out-of-range physical id: read page 0 instead, mask every token
                atomicOr(&P.ctrl[CTRL_ERR], (int)MKV_DEVERR_RANGE);
                id = 0;
                lp = 0x3FFFFFFF / PAGE;
              }
              s_list[rank - lo] = make_int2(lp, id);
            }
            rank++;
          }
        }
      }
      base += cnt;
    }
  }

  // ---- 2. queries of the GQA group -> fp16 MFMA operands in LDS
  float* qs = smem;  // [G][D]
  for (int i = tid; i < G * D; i += 256) {
    const int n = i / D, c = i % D;
    float x = bf16_to_f32(a.q[((int64_t)r * Hq + h * G + n) * D + c]);
    if (!is8) x *= (float)P.sigma[c];
    qs[i] = x;
  }
  __syncthreads();
  if (!is8) {
    for (int s = 1; s < D; s <<= 1) {
      for (int b = tid; b < G * D / 2; b += 256) {
        const int n = b / (D / 2), bb = b % (D / 2);
        const int i = n * D + (bb / s) * 2 * s + (bb % s);
        const float x0 = qs[i], x1 = qs[i + s];
        qs[i] = x0 + x1;
        qs[i + s] = x0 - x1;
      }
      __syncthreads();
    }
  }
  // Columns of the score tile: with G <= 8 two pages share one MFMA tile,
  // columns [0, 8) holding the heads for page a and [8, 16) for page b.
  const bool pair = G <= 8;
  const float qscale = is8 ? 1.0f : rsqrtf((float)D);
  const int ln = lane & 15, lg = lane >> 4;
  const int col_head = pair ? (ln & 7) : ln;
  const bool col_valid = col_head < G;
  const bool col_b = pair && ln >= 8;        // this column scores page b
  const bool row_b = pair && lg >= 2;        // accumulator rows 4*lg+i hold page b
  // fp16 query operands in MFMA lane order: qop[s][lane] (16 B each)
  half8* qop = reinterpret_cast<half8*>(smem + G * D);
  for (int i = tid; i < NS * 64; i += 256) {
    const int s = i / 64, l = i % 64;
    const int lln = l & 15, llg = l >> 4;
    const int ch = pair ? (lln & 7) : lln;
    half8 v;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      v[j] = (_Float16)(ch < G ? qs[ch * D + (D / 4) * llg + 8 * s + j] * qscale : 0.0f);
    qop[i] = v;
  }
  __syncthreads();

  // ---- 3. per-wave scan over page pairs
  WaveState<D> st;
#pragma unroll
  for (int m = 0; m < CL; ++m) st.acc[m] = float4v{0.f, 0.f, 0.f, 0.f};
  st.m_run = -INFINITY;
  st.l_run = 0.0f;

  const int npg = hi - lo;
  const int per_wave = (is8 ? a.c8 : a.c3) / 4;
  const int w0 = wid * per_wave, w1 = min(npg, w0 + per_wave);
  const int step = pair ? 2 : 1;
  const int layer = a.layer;
  const float smk = a.sm_log2;
  const float4v zero4 = {0.f, 0.f, 0.f, 0.f};

  if (!is8) {
    for (int ia = w0; ia < w1; ia += step) {
      const bool hasb = pair && ia + 1 < w1;
      const int2 ea = s_list[ia];
      const int2 eb = hasb ? s_list[ia + 1] : ea;
      const uint8_t* ra = P.tq3 + (((int64_t)layer * P.n_tq3 + ea.y) * H + h) * tq3_region_bytes(D);
      const uint8_t* rb = P.tq3 + (((int64_t)layer * P.n_tq3 + eb.y) * H + h) * tq3_region_bytes(D);
      const uint8_t* rown = row_b ? rb : ra;
      uint32_t kA[NDW], kB[NDW], vA[NDW], vB[NDW];
      {
        const uint32_t* pkA = reinterpret_cast<const uint32_t*>(ra + (ln * 4 + lg) * CB);
        const uint32_t* pkB = reinterpret_cast<const uint32_t*>(rb + (ln * 4 + lg) * CB);
        const uint32_t* pvA = reinterpret_cast<const uint32_t*>(ra + 6 * D + (ln * 4 + lg) * CB);
        const uint32_t* pvB = reinterpret_cast<const uint32_t*>(rb + 6 * D + (ln * 4 + lg) * CB);
#pragma unroll
        for (int w = 0; w < NDW; ++w) {
          kA[w] = pkA[w];
          kB[w] = pkB[w];
          vA[w] = pvA[w];
          vB[w] = pvB[w];
        }
      }
      const uint2 gw = *reinterpret_cast<const uint2*>((col_b ? rb : ra) + 12 * D + 8 * lg);
      // per-channel V scale of this lane's row page, V zero of both pages
      half2v sO[CL / 2], zA[CL / 2], zB[CL / 2];
      {
        const half2v* s0 = reinterpret_cast<const half2v*>(rown + 12 * D + 32 + 2 * CL * ln);
        const half2v* z0 = reinterpret_cast<const half2v*>(ra + 14 * D + 32 + 2 * CL * ln);
        const half2v* z1 = reinterpret_cast<const half2v*>(rb + 14 * D + 32 + 2 * CL * ln);
#pragma unroll
        for (int i = 0; i < CL / 2; ++i) {
          sO[i] = s0[i];
          zA[i] = z0[i];
          zB[i] = z1[i];
        }
      }
      // QK^T: rows = tokens of the page, columns = (page, head)
      float4v sa = zero4, sb = zero4;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const half8 qv = qop[s * 64 + lane];
        const uint32_t a0 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kA, 2 * s));
        const uint32_t a1 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kA, 2 * s + 1));
        sa = __builtin_amdgcn_mfma_f32_16x16x32_f16(h8(cvt_lo(a0), cvt_hi(a0), cvt_lo(a1), cvt_hi(a1)),
                                                     qv, sa, 0, 0, 0);
        if (pair) {
          const uint32_t b0 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kB, 2 * s));
          const uint32_t b1 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kB, 2 * s + 1));
          sb = __builtin_amdgcn_mfma_f32_16x16x32_f16(
              h8(cvt_lo(b0), cvt_hi(b0), cvt_lo(b1), cvt_hi(b1)), qv, sb, 0, 0, 0);
        }
      }
      float sc[4];
      {
        const int vcnt = col_b ? (hasb ? S - eb.x * PAGE : 0) : S - ea.x * PAGE;
        const _Float16* gh = reinterpret_cast<const _Float16*>(&gw);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float sv = col_b ? sb[i] : sa[i];
          sc[i] = (col_valid && 4 * lg + i < vcnt) ? sv * (float)gh[i] * smk : -INFINITY;
        }
      }
      softmax_step<D>(st, sc, lg);
      const half8 pT = p_operand(sc, col_b);
      // PV: codes enter the MFMA exactly; per-channel scale folded in fp32,
      // the zero term added by a second MFMA against the broadcast zeros
#pragma unroll
      for (int m = 0; m < CL; ++m) {
        const uint32_t ua = __builtin_amdgcn_perm(VLUT_HI, VLUT_LO, quad_sel<NDW>(vA, m));
        const uint32_t ub = __builtin_amdgcn_perm(VLUT_HI, VLUT_LO, quad_sel<NDW>(vB, m));
        const float4v X = __builtin_amdgcn_mfma_f32_16x16x32_f16(
            pT, h8(cvt_lo(ua), cvt_hi(ua), cvt_lo(ub), cvt_hi(ub)), zero4, 0, 0, 0);
        const float sm = (float)sO[m >> 1][m & 1];
        st.acc[m] += sm * X;
        const _Float16 za = zA[m >> 1][m & 1], zb = zB[m >> 1][m & 1];
        half8 zz;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          zz[j] = za;
          zz[4 + j] = zb;
        }
        st.acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(pT, zz, st.acc[m], 0, 0, 0);
      }
    }
  } else {
    for (int ia = w0; ia < w1; ia += step) {
      const bool hasb = pair && ia + 1 < w1;
      const int2 ea = s_list[ia];
      const int2 eb = hasb ? s_list[ia + 1] : ea;
      const int64_t pha = ((int64_t)layer * P.n_fp8 + ea.y) * H + h;
      const int64_t phb = ((int64_t)layer * P.n_fp8 + eb.y) * H + h;
      const uint8_t* ra = P.fp8 + pha * fp8_region_bytes(D);
      const uint8_t* rb = P.fp8 + phb * fp8_region_bytes(D);
      constexpr int KW = D / 16;  // dwords of K per lane (D/4 bytes)
      uint32_t kA[KW], kB[KW], vA[CL], vB[CL];
      {
        const uint4* pkA = reinterpret_cast<const uint4*>(ra + ln * D + (D / 4) * lg);
        const uint4* pkB = reinterpret_cast<const uint4*>(rb + ln * D + (D / 4) * lg);
        const uint4* pvA = reinterpret_cast<const uint4*>(ra + PAGE * D + (ln * 4 + lg) * 4 * CL);
        const uint4* pvB = reinterpret_cast<const uint4*>(rb + PAGE * D + (ln * 4 + lg) * 4 * CL);
#pragma unroll
        for (int w = 0; w < KW / 4; ++w) {
          const uint4 x = pkA[w], y = pkB[w];
          kA[4 * w] = x.x; kA[4 * w + 1] = x.y; kA[4 * w + 2] = x.z; kA[4 * w + 3] = x.w;
          kB[4 * w] = y.x; kB[4 * w + 1] = y.y; kB[4 * w + 2] = y.z; kB[4 * w + 3] = y.w;
        }
#pragma unroll
        for (int w = 0; w < CL / 4; ++w) {
          const uint4 x = pvA[w], y = pvB[w];
          vA[4 * w] = x.x; vA[4 * w + 1] = x.y; vA[4 * w + 2] = x.z; vA[4 * w + 3] = x.w;
          vB[4 * w] = y.x; vB[4 * w + 1] = y.y; vB[4 * w + 2] = y.z; vB[4 * w + 3] = y.w;
        }
      }
      const float sK = P.fp8_scales[(col_b ? phb : pha) * 2];
      const float sV = P.fp8_scales[(row_b ? phb : pha) * 2 + 1];
      float4v sa = zero4, sb = zero4;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const half8 qv = qop[s * 64 + lane];
        sa = __builtin_amdgcn_mfma_f32_16x16x32_f16(
            h8(cvt_lo(kA[2 * s]), cvt_hi(kA[2 * s]), cvt_lo(kA[2 * s + 1]), cvt_hi(kA[2 * s + 1])),
            qv, sa, 0, 0, 0);
        if (pair)
          sb = __builtin_amdgcn_mfma_f32_16x16x32_f16(
              h8(cvt_lo(kB[2 * s]), cvt_hi(kB[2 * s]), cvt_lo(kB[2 * s + 1]), cvt_hi(kB[2 * s + 1])),
              qv, sb, 0, 0, 0);
      }
      float sc[4];
      {
        const int vcnt = col_b ? (hasb ? S - eb.x * PAGE : 0) : S - ea.x * PAGE;
        const float kk = sK * smk;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float sv = col_b ? sb[i] : sa[i];
          sc[i] = (col_valid && 4 * lg + i < vcnt) ? sv * kk : -INFINITY;
        }
      }
      softmax_step<D>(st, sc, lg);
      const half8 pT = p_operand(sc, col_b);
#pragma unroll
      for (int m = 0; m < CL; ++m) {
        const float4v X = __builtin_amdgcn_mfma_f32_16x16x32_f16(
            pT, h8(cvt_lo(vA[m]), cvt_hi(vA[m]), cvt_lo(vB[m]), cvt_hi(vB[m])), zero4, 0, 0, 0);
        st.acc[m] += sV * X;
      }
    }
  }

  // ---- 4. rows -> heads: fetch each accumulator row's (m, l); merge the two
  // page parities (rows h and h + 8 sit in lanes l and l ^ 32); then merge the
  // four waves in LDS into one (m_j, l_j, O_j) partial per chunk
  float l_col = st.l_run;
  l_col += __shfl_xor(l_col, 16, 64);
  l_col += __shfl_xor(l_col, 32, 64);
  float mrow[4], lrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    mrow[i] = __shfl(st.m_run, 4 * lg + i, 64);
    lrow[i] = __shfl(l_col, 4 * lg + i, 64);
  }
  if (pair) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float m2 = __shfl_xor(mrow[i], 32, 64), l2 = __shfl_xor(lrow[i], 32, 64);
      const float M = fmaxf(lrow[i] > 0.0f ? mrow[i] : -INFINITY, l2 > 0.0f ? m2 : -INFINITY);
      const float f1 = lrow[i] > 0.0f ? exp2f(mrow[i] - M) : 0.0f;
      const float f2 = l2 > 0.0f ? exp2f(m2 - M) : 0.0f;
#pragma unroll
      for (int m = 0; m < CL; ++m) {
        const float o2 = __shfl_xor(st.acc[m][i], 32, 64);
        st.acc[m][i] = f1 * st.acc[m][i] + f2 * o2;
      }
      lrow[i] = f1 * lrow[i] + f2 * l2;
      mrow[i] = M;
    }
  }
  float* macc = smem;                 // [4][G][D]
  float* mm = smem + 4 * G * D;       // [4][G]
  float* ml = mm + 4 * G;             // [4][G]
  __syncthreads();                    // qop region is reused below
  if (!row_b) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int head = 4 * lg + i;
      if (head < G) {
#pragma unroll
        for (int m = 0; m < CL; ++m) macc[(wid * G + head) * D + CL * ln + m] = st.acc[m][i];
        if (ln == 0) {
          mm[wid * G + head] = mrow[i];
          ml[wid * G + head] = lrow[i];
        }
      }
    }
  }
  __syncthreads();
  float* part = a.partials + (((int64_t)r * H + h) * a.max_chunks + chunk) * G * (D + 2);
  for (int i = tid; i < G * D; i += 256) {
    const int n = i / D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w)
      if (ml[w * G + n] > 0.0f) M = fmaxf(M, mm[w * G + n]);
    float L = 0.0f, O = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float lw = ml[w * G + n];
      if (lw > 0.0f) {
        const float f = exp2f(mm[w * G + n] - M);
        L += f * lw;
        O += f * macc[(w * G + n) * D + (i % D)];
      }
    }
    part[i] = O / L;
    if (i % D == 0) {
      part[G * D + n] = M;
      part[G * D + G + n] = L;
    }
  }
}

// Merge stage (Eq. softmax-merge): one workgroup per (request, KV head, query
// head of the group).  The chunk partials' (m_j, l_j) go to LDS; each of the 4
// waves then folds a quarter of the partials' normalized outputs, four
// channels per lane with 16-byte loads, and the waves combine in LDS.
template <int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(int G, int H, int max_chunks,
                                                           const int32_t* totals,
                                                           const float* partials, float* out,
                                                           float* lse) {
  constexpr int C4 = D / 4;  // float4 lanes per row
  __shared__ float s_w[1024];
  __shared__ float4 s_acc[4][C4];
  __shared__ float s_red[8];
  const int n = blockIdx.x, h = blockIdx.y, r = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int Hq = H * G;
  const int total = min(totals[r], max_chunks);
  float* o = out + ((int64_t)r * Hq + h * G + n) * D;
  if (total <= 0) {
    for (int c = tid; c < D; c += 256) o[c] = 0.0f;
    if (lse && tid == 0) lse[(int64_t)r * Hq + h * G + n] = -INFINITY;
    return;
  }
  const float* base = partials + ((int64_t)r * H + h) * max_chunks * G * (D + 2);
  const int stride = G * (D + 2);
  // max over the partials' m_j (empty partials have l_j = 0)
  float M = -INFINITY;
  for (int k = tid; k < total; k += 256) {
    const float* pk = base + (int64_t)k * stride;
    const float lk = pk[G * D + G + n];
    if (lk > 0.0f) M = fmaxf(M, pk[G * D + n]);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, __shfl_xor(M, off, 64));
  if (lane == 0) s_red[wid] = M;
  __syncthreads();
  M = fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3]));
  __syncthreads();
  float L = 0.0f;
  for (int k0 = 0; k0 < total; k0 += 1024) {
    for (int k = k0 + tid; k < min(total, k0 + 1024); k += 256) {
      const float* pk = base + (int64_t)k * stride;
      const float lk = pk[G * D + G + n];
      const float wk = lk > 0.0f ? exp2f(pk[G * D + n] - M) * lk : 0.0f;
      s_w[k - k0] = wk;
      L += wk;
    }
    __syncthreads();
    if (lane < C4) {
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      const int kend = min(total, k0 + 1024);
#pragma unroll 8
      for (int k = k0 + wid; k < kend; k += 4) {
        const float wk = s_w[k - k0];
        const float4 v = *reinterpret_cast<const float4*>(base + (int64_t)k * stride + n * D + 4 * lane);
        acc.x += wk * v.x;
        acc.y += wk * v.y;
        acc.z += wk * v.z;
        acc.w += wk * v.w;
      }
      if (k0 == 0) s_acc[wid][lane] = acc;
      else {
        s_acc[wid][lane].x += acc.x; s_acc[wid][lane].y += acc.y;
        s_acc[wid][lane].z += acc.z; s_acc[wid][lane].w += acc.w;
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) L += __shfl_xor(L, off, 64);
  if (lane == 0) s_red[4 + wid] = L;
  __syncthreads();
  L = s_red[4] + s_red[5] + s_red[6] + s_red[7];
  const float inv = 1.0f / L;
  if (tid < C4) {
    float4 t = s_acc[0][tid];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      t.x += s_acc[w][tid].x; t.y += s_acc[w][tid].y;
      t.z += s_acc[w][tid].z; t.w += s_acc[w][tid].w;
    }
    t.x *= inv; t.y *= inv; t.z *= inv; t.w *= inv;
    *reinterpret_cast<float4*>(o + 4 * tid) = t;
  }
  if (lse && tid == 0) lse[(int64_t)r * Hq + h * G + n] = (M + log2f(L)) * 0.69314718055994531f;
}

hipError_t launch_decode(const PoolView& P, int layer, int n_req, const uint16_t* q,
                         const int32_t* bt, const uint8_t* tags, int max_pages,
                         const int32_t* seq_lens, float* out, float* lse, void* ws,
                         hipStream_t s) {
  DecodeShape sh = decode_shape(n_req, max_pages, P.n_kv_heads);
  DecodeArgs a;
  a.P = P;
  a.layer = layer;
  a.n_req = n_req;
  a.max_pages = max_pages;
  a.q = q;
  a.bt = bt;
  a.tags = tags;
  a.seq_lens = seq_lens;
  a.out = out;
  a.lse = lse;
  a.totals = reinterpret_cast<int32_t*>(ws);
  a.partials = reinterpret_cast<float*>(reinterpret_cast<uint8_t*>(ws) + header_bytes(n_req));
  a.c3 = sh.c3;
  a.c8 = sh.c8;
  a.max_chunks = sh.max_chunks;
  a.sm_log2 = 1.4426950408889634f / sqrtf((float)P.d);
  const size_t merge_f = (size_t)(4 * P.group * P.d + 8 * P.group);
  const size_t qop_f = (size_t)P.group * P.d + (size_t)(P.d / 32) * 64 * 4;
  const size_t lds = (merge_f > qop_f ? merge_f : qop_f) * sizeof(float);
  dim3 grid(sh.max_chunks, P.n_kv_heads, n_req);
  dim3 mgrid(P.group, P.n_kv_heads, n_req);
  if (P.d == 256) {
    hipLaunchKernelGGL(decode_kernel<256>, grid, dim3(256), lds, s, a);
    hipLaunchKernelGGL(decode_merge_kernel<256>, mgrid, dim3(256), 0, s, P.group, P.n_kv_heads,
                       sh.max_chunks, a.totals, a.partials, out, lse);
  } else {
    hipLaunchKernelGGL(decode_kernel<128>, grid, dim3(256), lds, s, a);
    hipLaunchKernelGGL(decode_merge_kernel<128>, mgrid, dim3(256), 0, s, P.group, P.n_kv_heads,
                       sh.max_chunks, a.totals, a.partials, out, lse);
  }
  return hipGetLastError();
}

}  // namespace mkv
