// Causal chunked-prefill attention over mixed FP8/TQ3 pages on MFMA (the
// query chunk makes it a dense contraction).  The paper runs prefill on a
// generic dense path (Sec. 4.1); this variant keeps the pages in their two
// physical formats and applies the same score algebra as decode (Sec. 3.3):
// rotated queries against TQ3 key codes times the FP16 key-norm correction,
// plain queries against FP8 keys, one online softmax per query row.
//
// Launch: one partition kernel (compact per-format lists, Sec. 4.1) and one
// attention kernel.  Grid (row block, KV head, request); 256 threads = 4
// waves, one workgroup per CU.  A query row is a (query token, head of the
// GQA group) pair; each wave owns 32 (d = 256) or 48 (d = 128) rows and streams
// every page of its request, TQ3 pairs first and FP8 pages after, through a
// two-slot LDS ring fed by direct HBM -> LDS copies:
//   S^T = K Q^T  on v_mfma_f32_16x16x32_f16: M = 16 tokens of a page,
//                N = 16 query rows, K = 32 channels; TQ3 codes -> E4M3
//                codebook bytes (one v_perm per 4 codes) -> fp16, against
//                the rotated query as an fp16 hi + lo pair (two MFMAs);
//   online softmax per query row in base 2 (lazy rescale, threshold 2^8),
//                causal mask token <= position of the query;
//   O^T += V^T P^T on the same MFMA: M = 16 channels, N = 16 query rows,
//                K = 32 tokens (two pages); weights as an fp16 hi + lo pair;
//                TQ3 values as three exact fp16 operands (high and low parts
//                of scale * code, and the zero); FP8 values exact, the
//                page's V scale folded into the weights.
// The workgroups of one (request, KV head) read the same pages at about the
// same time, so the page bytes come from L2 after the first reader.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "mkv_attn.h"
#include "mkv_internal.h"
#include "../../include/minima_kv.h"

namespace mkv {

constexpr int CW = 4;  // waves per chunk workgroup
// 16-row query tiles per wave: as many as the registers hold next to the
// O^T accumulators (d/16 x tiles x 4 floats per lane)
template <int D> constexpr int chunk_tiles() { return D == 256 ? 2 : 3; }
constexpr int CMASK_LP = 0x3FFFFFFF / PAGE;

struct ChunkArgs {
  PoolView P;
  int layer, n_req, max_pages, n_q_total;
  const uint16_t* q;
  const int32_t* cu_q;
  const int32_t* seq_lens;
  float* out;
  const int32_t* list8;   // [n_req][max_pages][2] (logical page, physical id)
  const int32_t* list3;
  const int32_t* counts;  // [n_req][2] (n_fp8, n_tq3)
  float sm_log2;          // log2(e) / sqrt(d)
};

static size_t al256(size_t b) { return (b + 255) / 256 * 256; }

// workspace: the two compact lists and their counts
size_t chunk_ws_bytes(int n_req, int max_pages, int n_q_total, int n_kv_heads, int group, int d) {
  (void)n_q_total; (void)n_kv_heads; (void)group; (void)d;
  return 2 * al256((size_t)n_req * max_pages * 2 * sizeof(int32_t)) +
         al256((size_t)n_req * 2 * sizeof(int32_t));
}

// fp16 value with its low 3 significand bits cleared (8 significant bits left)
__device__ __forceinline__ _Float16 hi8(_Float16 x) {
  const uint16_t b = __builtin_bit_cast(uint16_t, x);
  return __builtin_bit_cast(_Float16, (uint16_t)(b & 0xFFF8u));
}

template <int D>
__global__ __launch_bounds__(64 * CW, 1) void chunk_kernel(ChunkArgs a) {
  constexpr int CRT = chunk_tiles<D>(), CROWS = 16 * CRT;  // query rows per wave
  constexpr int NDW = 3 * D / 128, CB = 3 * D / 32, CL = D / 16, NS = D / 32, QQ = D / 4;
  constexpr int R3 = (int)tq3_region_bytes(D);
  constexpr int R8 = (int)fp8_region_bytes(D);
  constexpr int STAGE = 2 * R3;  // a TQ3 page pair, or one FP8 page + its two scales
  constexpr int OPS3 = 2 * dma_ops<R3>(), OPS8 = dma_ops<R8>() + 1;
  static_assert(dma_ops<R8>() == 2 * (D / 64), "dma_fp8_page issues 2 d / 64 copies");
  static_assert(R8 + 8 <= STAGE, "an FP8 page and its scales fit one stage");
  extern __shared__ __align__(16) uint8_t smem[];
  const PoolView& P = a.P;
  const int r = blockIdx.z, h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ln = lane & 15, lg = lane >> 4;
  const int G = P.group, H = P.n_kv_heads, Hq = H * G;
  const int mp = a.max_pages;

  // ---- request and rows of this wave
  const int q0 = a.cu_q[r], q1 = a.cu_q[r + 1];
  const int nq = q1 - q0;
  const int S = a.seq_lens[r];
  const bool range_ok = q0 >= 0 && nq >= 0 && q1 <= a.n_q_total;
  const int rows_r = range_ok ? nq * G : 0;
  const int rb = blockIdx.x * (CW * CROWS) + wid * CROWS;
  if (!range_ok || nq < 1 || S < nq || S > mp * PAGE) {
    if (blockIdx.x == 0 && tid == 0) atomicOr(&P.ctrl[CTRL_ERR], (int)MKV_DEVERR_RANGE);
    // rows that can be located get zeros
    for (int rt = 0; rt < CRT; ++rt) {
      const int rho = rb + 16 * rt + ln;
      if (rho < rows_r) {
        float* o = a.out + ((int64_t)(q0 + rho / G) * Hq + h * G + rho % G) * D;
        for (int c = lg; c < D; c += 4) o[c] = 0.0f;
      }
    }
    return;
  }
  if (rb >= rows_r) return;  // waves are independent: no workgroup barrier below
  const int P0 = S - nq;     // position of the chunk's first query

  // lane's query row per tile: position (-1 for rows past the request's rows)
  int posr[CRT];
#pragma unroll
  for (int rt = 0; rt < CRT; ++rt) {
    const int rho = rb + 16 * rt + ln;
    posr[rt] = rho < rows_r ? P0 + rho / G : -1;
  }

  // ---- query operands: B of S^T = K Q^T; lane (ln, lg) holds, for k-step s,
  // channels QQ lg + 8 s + j (j < 8) of query row 16 rt + ln.  TQ3 pages use
  // q_rot = R q (R = d^-1/2 H diag(sigma)), FP8 pages the plain q.
  half8 qop[CRT][NS];
  // the rotated query's fp16 low part (q_rot = hi + lo to fp32 accuracy)
  // lives in LDS after the rings: [wave][tile][k-step][lane]
  half8* qlo = reinterpret_cast<half8*>(smem + CW * 2 * STAGE) + wid * CRT * NS * 64;
  auto build_q = [&](bool rotated) {
#pragma unroll
    for (int rt = 0; rt < CRT; ++rt) {
      const int rho = min(rb + 16 * rt + ln, rows_r - 1);
      const uint16_t* qrow = a.q + ((int64_t)(q0 + rho / G) * Hq + h * G + rho % G) * D + QQ * lg;
      float x[NS][8];
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const uint4 raw = *reinterpret_cast<const uint4*>(qrow + 8 * s);
        const uint16_t* hb = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
        for (int j = 0; j < 8; ++j) x[s][j] = bf16_to_f32(hb[j]);
      }
      if (rotated) {
        const int8_t* sg = P.sigma + QQ * lg;
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
          for (int j = 0; j < 8; ++j) x[s][j] *= (float)sg[8 * s + j];
        // Walsh-Hadamard butterflies over the channel bits: j (strides 1-4)
        // and s (strides 8 .. 4 NS) inside the lane, lg (strides QQ, 2 QQ)
        // across lanes l ^ 16 and l ^ 32; the stages commute
#pragma unroll
        for (int st = 1; st < 8; st <<= 1)
#pragma unroll
          for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int j = 0; j < 8; ++j)
              if (!(j & st)) {
                const float x0 = x[s][j], x1 = x[s][j + st];
                x[s][j] = x0 + x1;
                x[s][j + st] = x0 - x1;
              }
#pragma unroll
        for (int st = 1; st < NS; st <<= 1)
#pragma unroll
          for (int s = 0; s < NS; ++s)
            if (!(s & st)) {
#pragma unroll
              for (int j = 0; j < 8; ++j) {
                const float x0 = x[s][j], x1 = x[s + st][j];
                x[s][j] = x0 + x1;
                x[s + st][j] = x0 - x1;
              }
            }
        const float sgn16 = (lane & 16) ? -1.0f : 1.0f, sgn32 = (lane & 32) ? -1.0f : 1.0f;
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            x[s][j] = fmaf(sgn16, x[s][j], lane_xor<16>(x[s][j], lane));
            x[s][j] = fmaf(sgn32, x[s][j], lane_xor<32>(x[s][j], lane));
          }
        const float qscale = rsqrtf((float)D);
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
          for (int j = 0; j < 8; ++j) x[s][j] *= qscale;
      }
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        half8 lo;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          qop[rt][s][j] = (_Float16)x[s][j];
          lo[j] = (_Float16)(x[s][j] - (float)qop[rt][s][j]);
        }
        if (rotated) qlo[(rt * NS + s) * 64 + lane] = lo;
      }
    }
  };

  // ---- stage list: TQ3 pairs (list3 entries 2k, 2k+1), then FP8 pages
  const int n8 = a.counts[2 * r], n3 = a.counts[2 * r + 1];
  const int st3 = (n3 + 1) / 2, n_st = st3 + n8;
  const int2* l3 = reinterpret_cast<const int2*>(a.list3) + (int64_t)r * mp;
  const int2* l8 = reinterpret_cast<const int2*>(a.list8) + (int64_t)r * mp;
  // (logical page, physical id) of a list entry; out-of-range ids read page 0
  // with every token masked and are reported after the loop (no memory
  // writes while copies are in flight)
  bool bad_id = false;
  auto checked = [&](int2 e, int n_ids) {
    if (e.y < 0 || e.y >= n_ids) {
      bad_id = true;
      return make_int2(CMASK_LP, 0);
    }
    return e;
  };
  // List entries reach the wave 64 at a time (lane k holds entry base + k)
  // and are read out with v_readlane, so the loop issues one vector load per
  // 64 entries (its wait also drains the copies in flight) instead of one per
  // stage.
  int2 cache = make_int2(0, 0);
  int cache_tag = -1;  // 2 * base + list (0: TQ3, 1: FP8)
  auto entry = [&](int list, int k) {
    const int base = k & ~63, tag = 2 * base + list;
    if (tag != cache_tag) {
      const int2* l = list ? l8 : l3;
      const int n = list ? n8 : n3;
      cache = l[min(base + lane, n - 1)];
      cache_tag = tag;
    }
    return make_int2(__builtin_amdgcn_readlane(cache.x, k - base),
                     __builtin_amdgcn_readlane(cache.y, k - base));
  };
  // stage j -> {lp_a, id_a, lp_b, id_b}; id_b < 0 marks an FP8 stage
  auto stage_at = [&](int j) {
    if (j < st3) {
      const int2 ea = checked(entry(0, 2 * j), P.n_tq3);
      int2 eb = 2 * j + 1 < n3 ? checked(entry(0, 2 * j + 1), P.n_tq3) : make_int2(CMASK_LP, ea.y);
      return make_int4(ea.x, ea.y, eb.x, eb.y);
    }
    const int2 e = checked(entry(1, j - st3), P.n_fp8);
    return make_int4(e.x, e.y, 0, -1);
  };
  const int layer = a.layer;
  const uint8_t* tq3_l = P.tq3 + (int64_t)layer * P.n_tq3 * H * R3;
  const uint8_t* fp8_l = P.fp8 + (int64_t)layer * P.n_fp8 * H * R8;
  const uint8_t* scl_l = reinterpret_cast<const uint8_t*>(P.fp8_scales + (int64_t)layer * P.n_fp8 * H * 2);
  uint8_t* wring = smem + wid * 2 * STAGE;
  const uint32_t wring_lds = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)wring);
  const DmaLanes dl = {16u * lane, 4096u + 16u * lane};
  auto issue = [&](const int4& e, int slot) {
    const uint32_t dst = wring_lds + slot * STAGE;
    if (e.w >= 0) {
      dma_region<R3>(dst, tq3_l + ((int64_t)e.y * H + h) * R3, dl, lane);
      dma_region<R3>(dst + R3, tq3_l + ((int64_t)e.w * H + h) * R3, dl, lane);
    } else {
      dma_fp8_page<D>(dst, fp8_l + ((int64_t)e.y * H + h) * R8, lane);
      if (lane < 2) dma4(4 * lane, scl_l + ((int64_t)e.y * H + h) * 8, dst + R8);
    }
  };
  auto begin_stage = [&](int j) {
    const int nops = j + 1 < n_st ? (j + 1 < st3 ? OPS3 : OPS8) : 0;
    if (nops == OPS3)
      wait_vmcnt<OPS3>();
    else if (nops == OPS8)
      wait_vmcnt<OPS8>();
    else
      wait_vmcnt<0>();
  };

  // ---- accumulators: O^T tiles (16 channels x 16 query rows) per channel
  // tile m and row tile rt; lane (ln, lg) holds channels CL (4 lg + i) + m of
  // query row 16 rt + ln
  float4v acc[CL][CRT];
#pragma unroll
  for (int m = 0; m < CL; ++m)
#pragma unroll
    for (int rt = 0; rt < CRT; ++rt) acc[m][rt] = float4v{0.f, 0.f, 0.f, 0.f};
  float m_run[CRT], l_run[CRT];
#pragma unroll
  for (int rt = 0; rt < CRT; ++rt) {
    m_run[rt] = -INFINITY;
    l_run[rt] = 0.0f;
  }
  const float smk = a.sm_log2;
  const float4v zero4 = {0.f, 0.f, 0.f, 0.f};

  // Online softmax over this stage's scores sc[rt][k] (k < NK: this lane's
  // tokens) of query row 16 rt + ln; returns the weights in place.
  auto softmax = [&](float (*sc)[8], auto nkc) {
    constexpr int NK = decltype(nkc)::value;
#pragma unroll
    for (int rt = 0; rt < CRT; ++rt) {
      float mx = sc[rt][0];
#pragma unroll
      for (int k = 1; k < NK; ++k) mx = fmaxf(mx, sc[rt][k]);
      mx = max4rows(mx);
      const bool need = mx > m_run[rt] + 8.0f;
      if (__any(need)) {
        const float m_new = need ? mx : m_run[rt];
        const float alpha = m_run[rt] == -INFINITY ? 0.0f : exp2f(m_run[rt] - m_new);
        m_run[rt] = m_new;
        l_run[rt] *= alpha;
#pragma unroll
        for (int m = 0; m < CL; ++m) acc[m][rt] *= alpha;  // column = this lane's row
      }
#pragma unroll
      for (int k = 0; k < NK; ++k) {
        sc[rt][k] = exp2_safe(sc[rt][k], m_run[rt]);
        l_run[rt] += sc[rt][k];
      }
    }
  };

  const int n_pre = min(2, n_st);
  for (int k = 0; k < n_pre; ++k) issue(stage_at(k), k);
  build_q(true);
  for (int j = 0; j < st3; ++j) {
    const int slot = j & 1;
    const int4 e = stage_at(j);
    begin_stage(j);
    const bool refill = j + 2 < n_st;
    const int4 e2 = refill ? stage_at(j + 2) : e;
    const uint8_t* ra = wring + slot * STAGE;
    // ---------------- TQ3 pair
    const uint8_t* rb2 = ra + R3;
    uint32_t kA[NDW], kB[NDW], vA[NDW], vB[NDW];
    read_chunk<NDW>(kA, ra, 16 * lg + ln);
    read_chunk<NDW>(kB, rb2, 16 * lg + ln);
    read_chunk<NDW>(vA, ra + 6 * D, 16 * lg + ln);
    read_chunk<NDW>(vB, rb2 + 6 * D, 16 * lg + ln);
    const uint2 gA = *reinterpret_cast<const uint2*>(ra + 12 * D + 8 * lg);
    const uint2 gB = *reinterpret_cast<const uint2*>(rb2 + 12 * D + 8 * lg);
    half2v sA[CL / 2], zA[CL / 2], sB[CL / 2], zB[CL / 2];
#pragma unroll
    for (int i = 0; i < CL / 2; ++i) {
      sA[i] = reinterpret_cast<const half2v*>(ra + 12 * D + 32 + 2 * CL * ln)[i];
      zA[i] = reinterpret_cast<const half2v*>(ra + 14 * D + 32 + 2 * CL * ln)[i];
      sB[i] = reinterpret_cast<const half2v*>(rb2 + 12 * D + 32 + 2 * CL * ln)[i];
      zB[i] = reinterpret_cast<const half2v*>(rb2 + 14 * D + 32 + 2 * CL * ln)[i];
    }
    wait_lgkm0();  // the stage is in registers: refill its slot
    if (refill) issue(e2, slot);
    // S^T for both pages
    float4v st[2][CRT];
#pragma unroll
    for (int pg = 0; pg < 2; ++pg)
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt) st[pg][rt] = zero4;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const uint32_t a0 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kA, 2 * s));
      const uint32_t a1 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kA, 2 * s + 1));
      const uint32_t b0 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kB, 2 * s));
      const uint32_t b1 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kB, 2 * s + 1));
      const half8 Ka = h8(cvt_lo(a0), cvt_hi(a0), cvt_lo(a1), cvt_hi(a1));
      const half8 Kb = h8(cvt_lo(b0), cvt_hi(b0), cvt_lo(b1), cvt_hi(b1));
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt) {
        const half8 ql = qlo[(rt * NS + s) * 64 + lane];
        st[0][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(Ka, qop[rt][s], st[0][rt], 0, 0, 0);
        st[1][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(Kb, qop[rt][s], st[1][rt], 0, 0, 0);
        st[0][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(Ka, ql, st[0][rt], 0, 0, 0);
        st[1][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(Kb, ql, st[1][rt], 0, 0, 0);
      }
    }
    // scores (tokens 4 lg + i of pages a and b), causal and length masks
    float sc[CRT][8];
    {
      const _Float16* ga = reinterpret_cast<const _Float16*>(&gA);
      const _Float16* gb = reinterpret_cast<const _Float16*>(&gB);
      const int ta = e.x * PAGE + 4 * lg, tb = e.z * PAGE + 4 * lg;
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t0 = ta + i, t1 = tb + i;
          sc[rt][i] = (t0 < S && t0 <= posr[rt]) ? st[0][rt][i] * (float)ga[i] * smk : -INFINITY;
          sc[rt][4 + i] = (t1 < S && t1 <= posr[rt]) ? st[1][rt][i] * (float)gb[i] * smk : -INFINITY;
        }
    }
    softmax(sc, std::integral_constant<int, 8>{});
    // weights as an fp16 hi + lo pair: one token can carry most of a row's
    // mass, and its weight, taken relative to a lagging reference max, is
    // then not a power of two; a single fp16 rounding of it moves the output
    // by up to 2^-12 of that token's value
    half8 pH[CRT], pL[CRT];
#pragma unroll
    for (int rt = 0; rt < CRT; ++rt)
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const _Float16 hi = (_Float16)sc[rt][k];
        pH[rt][k] = hi;
        pL[rt][k] = (_Float16)(sc[rt][k] - (float)hi);
      }
    // O^T += V^T P^T with exact V operands: v = zero + scale * code is split
    // as scale_hi * code + scale_lo * code + zero, scale_hi keeping 8
    // significant bits of the fp16 scale (so 3-bit codes times it are exact
    // in fp16) and scale_lo the remaining 3; the products that reach fp32
    // accuracy are (hi + lo weights) x (scale_hi term, zero) and hi weights x
    // scale_lo term (lo x scale_lo sits below 2^-19 of the value)
#pragma unroll
    for (int m = 0; m < CL; ++m) {
      const uint32_t ua = quad_sel<NDW>(vA, m), ub = quad_sel<NDW>(vB, m);
      const half2v ca01 = cvt_code<false>(ua), ca23 = cvt_code<true>(ua);
      const half2v cb01 = cvt_code<false>(ub), cb23 = cvt_code<true>(ub);
      const _Float16 sa = sA[m >> 1][m & 1], za = zA[m >> 1][m & 1];
      const _Float16 sb = sB[m >> 1][m & 1], zb = zB[m >> 1][m & 1];
      const _Float16 sa_hi = hi8(sa), sb_hi = hi8(sb);
      const _Float16 sa_lo = sa - sa_hi, sb_lo = sb - sb_hi;  // exact
      const half2v sah = {sa_hi, sa_hi}, sal = {sa_lo, sa_lo};
      const half2v sbh = {sb_hi, sb_hi}, sbl = {sb_lo, sb_lo};
      const half8 A1 = h8(ca01 * sah, ca23 * sah, cb01 * sbh, cb23 * sbh);
      const half8 A2 = h8(ca01 * sal, ca23 * sal, cb01 * sbl, cb23 * sbl);
      const half2v za2 = {za, za}, zb2 = {zb, zb};
      const half8 A3 = h8(za2, za2, zb2, zb2);
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt) {
        acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A1, pH[rt], acc[m][rt], 0, 0, 0);
        acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A2, pH[rt], acc[m][rt], 0, 0, 0);
        acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A3, pH[rt], acc[m][rt], 0, 0, 0);
        acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A1, pL[rt], acc[m][rt], 0, 0, 0);
        acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A3, pL[rt], acc[m][rt], 0, 0, 0);
      }
    }
  }
  if (st3 < n_st) build_q(false);  // plain queries for the FP8 pages
  for (int j = st3; j < n_st; ++j) {
    const int slot = j & 1;
    const int4 e = stage_at(j);
    begin_stage(j);
    const bool refill = j + 2 < n_st;
    const int4 e2 = refill ? stage_at(j + 2) : e;
    const uint8_t* ra = wring + slot * STAGE;
    // ---------------- one FP8 page
    constexpr int KW = D / 16;
    uint32_t kA[KW], vA[CL];
    {
      // block-permuted page (see dma_fp8_page): lane l's w-th 16 bytes at 64 w + l
      const uint4* pk = reinterpret_cast<const uint4*>(ra) + lane;
      const uint4* pv = reinterpret_cast<const uint4*>(ra + PAGE * D) + lane;
#pragma unroll
      for (int w = 0; w < KW / 4; ++w) {
        const uint4 x = pk[64 * w];
        kA[4 * w] = x.x; kA[4 * w + 1] = x.y; kA[4 * w + 2] = x.z; kA[4 * w + 3] = x.w;
      }
#pragma unroll
      for (int w = 0; w < CL / 4; ++w) {
        const uint4 x = pv[64 * w];
        vA[4 * w] = x.x; vA[4 * w + 1] = x.y; vA[4 * w + 2] = x.z; vA[4 * w + 3] = x.w;
      }
    }
    const float2 ksv = *reinterpret_cast<const float2*>(ra + R8);
    wait_lgkm0();
    if (refill) issue(e2, slot);
    float4v st[CRT];
#pragma unroll
    for (int rt = 0; rt < CRT; ++rt) st[rt] = zero4;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const half8 Ka = h8(cvt_lo(kA[2 * s]), cvt_hi(kA[2 * s]), cvt_lo(kA[2 * s + 1]), cvt_hi(kA[2 * s + 1]));
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt)
        st[rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(Ka, qop[rt][s], st[rt], 0, 0, 0);
    }
    float sc[CRT][8];
    {
      const int ta = e.x * PAGE + 4 * lg;
      const float kk = ksv.x * smk;
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t0 = ta + i;
          sc[rt][i] = (t0 < S && t0 <= posr[rt]) ? st[rt][i] * kk : -INFINITY;
        }
    }
    softmax(sc, std::integral_constant<int, 4>{});
    // the page's V scale folded into the weights, carried as an fp16 pair
    // (hi + lo) so the products keep fp32 accuracy
    half8 pH[CRT], pL[CRT];
#pragma unroll
    for (int rt = 0; rt < CRT; ++rt)
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float w = k < 4 ? sc[rt][k] * ksv.y : 0.0f;
        const _Float16 hi = (_Float16)w;
        pH[rt][k] = hi;
        pL[rt][k] = (_Float16)(w - (float)hi);
      }
    const half2v z2 = {(_Float16)0.0f, (_Float16)0.0f};
#pragma unroll
    for (int m = 0; m < CL; ++m) {
      const half8 Av = h8(cvt_lo(vA[m]), cvt_hi(vA[m]), z2, z2);
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt) {
        acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(Av, pH[rt], acc[m][rt], 0, 0, 0);
        acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(Av, pL[rt], acc[m][rt], 0, 0, 0);
      }
    }
  }

  if (__any(bad_id) && lane == 0) atomicOr(&P.ctrl[CTRL_ERR], (int)MKV_DEVERR_RANGE);
  // ---- normalize and store: lane (ln, lg) holds channels CL (4 lg + i) + m
  // (m < CL, contiguous) of query row 16 rt + ln
#pragma unroll
  for (int rt = 0; rt < CRT; ++rt) {
    const float L = sum4rows(l_run[rt]);
    const int rho = rb + 16 * rt + ln;
    if (rho >= rows_r) continue;
    const float inv = L > 0.0f ? 1.0f / L : 0.0f;
    float* o = a.out + ((int64_t)(q0 + rho / G) * Hq + h * G + rho % G) * D;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int m4 = 0; m4 < CL / 4; ++m4)
        *reinterpret_cast<float4*>(o + CL * (4 * lg + i) + 4 * m4) =
            make_float4(acc[4 * m4][rt][i] * inv, acc[4 * m4 + 1][rt][i] * inv,
                        acc[4 * m4 + 2][rt][i] * inv, acc[4 * m4 + 3][rt][i] * inv);
  }
}

hipError_t launch_chunk(const PoolView& P, int layer, int n_req, const uint16_t* q,
                        const int32_t* cu_q, int n_q_total, const int32_t* bt, const uint8_t* tags,
                        int max_pages, const int32_t* seq_lens, float* out, void* ws,
                        hipStream_t s) {
  ChunkArgs a;
  a.P = P;
  a.layer = layer;
  a.n_req = n_req;
  a.max_pages = max_pages;
  a.n_q_total = n_q_total;
  a.q = q;
  a.cu_q = cu_q;
  a.seq_lens = seq_lens;
  a.out = out;
  uint8_t* w = reinterpret_cast<uint8_t*>(ws);
  const size_t lb = al256((size_t)n_req * max_pages * 2 * sizeof(int32_t));
  int32_t* list8 = reinterpret_cast<int32_t*>(w);
  int32_t* list3 = reinterpret_cast<int32_t*>(w + lb);
  int32_t* counts = reinterpret_cast<int32_t*>(w + 2 * lb);
  a.list8 = list8;
  a.list3 = list3;
  a.counts = counts;
  a.sm_log2 = 1.4426950408889634f / sqrtf((float)P.d);
  hipError_t e = launch_partition(n_req, bt, tags, max_pages, seq_lens, list8, list3, counts,
                                  P.ctrl + CTRL_ERR, s);
  if (e != hipSuccess) return e;
  const int tiles = P.d == 256 ? chunk_tiles<256>() : chunk_tiles<128>();
  const size_t lds = (size_t)CW * 2 * 2 * tq3_region_bytes(P.d) +  // rings
                     (size_t)CW * tiles * (P.d / 32) * 64 * 16;    // rotated-query low parts
  const void* kern = P.d == 256 ? (const void*)chunk_kernel<256> : (const void*)chunk_kernel<128>;
  e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  // rows of one request: at most n_q_total queries x group heads
  const int64_t rows = (int64_t)n_q_total * P.group;
  const int wg_rows = CW * 16 * (P.d == 256 ? chunk_tiles<256>() : chunk_tiles<128>());
  const int blocks = (int)((rows + wg_rows - 1) / wg_rows);
  dim3 grid(blocks, P.n_kv_heads, n_req);
  void* args[] = {&a};
  e = hipLaunchKernel(kern, grid, dim3(64 * CW), args, lds, s);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace mkv
