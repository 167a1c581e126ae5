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
// GQA group) pair; each wave owns 32 (d = 256) or 48 (d = 128) rows.  The
// workgroup streams every page of its request, TQ3 pairs first and FP8 pages
// after, through one LDS ring shared by its waves: each wave issues a quarter
// of every stage's direct HBM -> LDS copies, and one barrier per stage both
// publishes the stage and frees the slot read before it.
//   S^T = K Q^T  on v_mfma_f32_16x16x32_f16: M = 16 tokens of a page, N = 16
//                query rows, K = 32 channels; TQ3 codes -> E4M3 codebook
//                bytes (one v_perm per 4 codes) -> fp16, against the rotated
//                query as an fp16 hi + lo pair (two MFMAs); FP8 keys -> fp16
//                against the plain query (exact in fp16, one MFMA);
//   online softmax per query row in base 2 (lazy rescale, threshold 2^8),
//                causal mask token <= position of the query;
//   O^T += V^T P^T on v_mfma_f32_16x16x32_f16: M = 16 channels, N = 16 query
//                rows, K = 32 tokens (two pages); weights as an fp16 hi + lo
//                pair; TQ3 values as exact fp16 operands (high and low parts
//                of scale * code) with the zero term as one rank-2 product of
//                the pages' zeros and weight sums per stage; FP8 values exact,
//                the page's V scale folded into the weights.
// The workgroups of one (request, KV head) read the same pages at about the
// same time, so the page bytes come from L2 after the first reader.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "mkv_attn.h"
#include "mkv_internal.h"
#include "../../include/minima_kv.h"

namespace mkv {

constexpr int CW = 4;        // waves per chunk workgroup
constexpr int CSLOTS = 7;    // stages in the shared ring
// 16-row query tiles per wave: as many as the registers hold next to the
// O^T accumulators (d/16 x tiles x 4 floats per lane) and the query terms
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
__device__ __forceinline__ half2v hi8x2(half2v x) {
  const uint32_t b = __builtin_bit_cast(uint32_t, x);
  return __builtin_bit_cast(half2v, b & 0xFFF8FFF8u);
}
__device__ __forceinline__ half2v bcast(_Float16 x) { return half2v{x, x}; }
// (a, b) as fp16 pairs hi = (a, b) rounded to nearest, lo = the rounded
// remainders: together 22 significant bits.  (The round-toward-zero packed
// conversion flushes fp16 subnormals, so the low part of every weight below
// 2^-4 vanished and chunk outputs moved by up to 1.3e-3.)
__device__ __forceinline__ void split2(float a, float b, uint32_t& hi, uint32_t& lo) {
  const half2v h = {(_Float16)a, (_Float16)b};
  const half2v l = {(_Float16)(a - (float)h[0]), (_Float16)(b - (float)h[1])};
  hi = __builtin_bit_cast(uint32_t, h);
  lo = __builtin_bit_cast(uint32_t, l);
}
__device__ __forceinline__ half8 h8u(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  typedef uint32_t u4v __attribute__((ext_vector_type(4)));
  return __builtin_bit_cast(half8, u4v{a, b, c, d});
}
constexpr float CM_INIT = -1.0e30f;  // running max before the first score (finite: no inf - inf)

template <int D>
__global__ __launch_bounds__(64 * CW, 1) void chunk_kernel(ChunkArgs a) {
  constexpr int CRT = chunk_tiles<D>(), CROWS = 16 * CRT;  // query rows per wave
  constexpr int NDW = 3 * D / 128, CL = D / 16, NS = D / 32, QQ = D / 4;
  constexpr int R3 = (int)tq3_region_bytes(D);
  constexpr int R8 = (int)fp8_region_bytes(D);
  constexpr int STAGE = 2 * R3;       // a TQ3 page pair, or one FP8 page + its two scales
  constexpr int MAIN_KB = 16 * D / 1024;  // whole KiB of a TQ3 page (its last 32 bytes aside)
  constexpr int OPS_W = 2 * MAIN_KB / CW;  // 1-KiB copies per wave per stage
  constexpr int NI = D / 64;               // 1-KiB copies per half of an FP8 page
  static_assert(2 * MAIN_KB % CW == 0 && 2 * NI == CW * OPS_W, "copies split evenly");
  static_assert(R3 == 1024 * MAIN_KB + 32, "TQ3 page = whole KiB + a 32-byte tail");
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
  if (!range_ok || nq < 1 || S < nq || S > mp * PAGE) {  // workgroup-uniform
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
  if (blockIdx.x * (CW * CROWS) >= rows_r) return;  // whole workgroup past the rows
  // Waves whose rows all lie past the request's rows still take part in the
  // copies and barriers; their scores are all masked.
  const int P0 = S - nq;  // position of the chunk's first query

  // lane's query row per tile: position (-1 for rows past the request's rows)
  int posr[CRT];
#pragma unroll
  for (int rt = 0; rt < CRT; ++rt) {
    const int rho = rb + 16 * rt + ln;
    posr[rt] = rho < rows_r ? P0 + rho / G : -1;
  }

  // ---- query operands: B of S^T = K Q^T; lane (ln, lg) holds, for k-step
  // s, channels QQ lg + 8 s + j (j < 8) of query row 16 rt + ln.  TQ3 pages
  // use q_rot = R q (R = d^-1/2 H diag(sigma)) as an fp16 pair hi + lo (fp32
  // accuracy: two MFMAs), FP8 pages the plain q (bf16 -> fp16 is exact: one
  // MFMA).  The keys enter as fp16 too: the fp8 MFMA adds its products in
  // groups aligned to the group's largest one and keeps only about 15 bits
  // there, which moved chunk outputs by up to 2e-3 where keys carry large
  // norms.
  half8 qop[CRT][NS];
  // the rotated query's fp16 low part lives in this wave's LDS area after the
  // ring: [tile][k-step][lane]
  half8* qlo = reinterpret_cast<half8*>(smem + CSLOTS * STAGE) + wid * CRT * NS * 64;
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
  // and are read out with v_readlane: one vector load per 64 entries (its
  // wait also drains the copies in flight).  Two caches: one for the stage
  // being copied, one for the stage being computed, which lags it.
  struct ListCache {
    int2 v;
    int tag;  // 2 * base + list (0: TQ3, 1: FP8)
  };
  ListCache c_iss{make_int2(0, 0), -1}, c_cmp{make_int2(0, 0), -1};
  auto entry = [&](ListCache& c, int list, int k) {
    const int base = k & ~63, tag = 2 * base + list;
    if (tag != c.tag) {
      const int2* l = list ? l8 : l3;
      const int n = list ? n8 : n3;
      c.v = l[min(base + lane, n - 1)];
      c.tag = tag;
    }
    return make_int2(__builtin_amdgcn_readlane(c.v.x, k - base),
                     __builtin_amdgcn_readlane(c.v.y, k - base));
  };
  // stage j -> {lp_a, id_a, lp_b, id_b}; id_b < 0 marks an FP8 stage
  auto stage_at = [&](ListCache& c, int j) {
    if (j < st3) {
      const int2 ea = checked(entry(c, 0, 2 * j), P.n_tq3);
      int2 eb = 2 * j + 1 < n3 ? checked(entry(c, 0, 2 * j + 1), P.n_tq3) : make_int2(CMASK_LP, ea.y);
      return make_int4(ea.x, ea.y, eb.x, eb.y);
    }
    const int2 e = checked(entry(c, 1, j - st3), P.n_fp8);
    return make_int4(e.x, e.y, 0, -1);
  };
  const int layer = a.layer;
  const uint8_t* tq3_l = P.tq3 + (int64_t)layer * P.n_tq3 * H * R3;
  const uint8_t* fp8_l = P.fp8 + (int64_t)layer * P.n_fp8 * H * R8;
  const uint8_t* scl_l = reinterpret_cast<const uint8_t*>(P.fp8_scales + (int64_t)layer * P.n_fp8 * H * 2);
  const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)smem);
  // FP8 pages land block-permuted (see dma_fp8_page): per-lane source offsets
  const uint32_t vk = 16u * (uint32_t)(ln * (D / 16) + lg * NI);
  const uint32_t vv = 16u * (uint32_t)((ln * 4 + lg) * NI);
  // This wave's share of stage e's copies into ring slot `slot`: OPS_W whole
  // KiB (TQ3: KiB w OPS_W .. of the two pages laid end to end; FP8: copies
  // w OPS_W .. of the page's 2 NI), and for waves 0 and 1 one small copy
  // (TQ3: the 32-byte tail of page a resp. b; FP8: the two scales, copied by
  // both so that every stage costs each wave the same number of copies).
  auto issue = [&](const int4& e, int slot) {
    const uint32_t dst = ring_lds + slot * STAGE;
    if (e.w >= 0) {
#pragma unroll
      for (int i = 0; i < OPS_W; ++i) {
        const int g = wid * OPS_W + i, pg = g / MAIN_KB, kb = g % MAIN_KB;
        const int id = pg ? e.w : e.y;
        dma16<0>(16u * lane + 1024u * kb, tq3_l + ((int64_t)id * H + h) * R3,
                 dst + pg * R3 + 1024 * kb);
      }
      if (wid < 2) {
        const int id = wid ? e.w : e.y;
        if (lane < 8) dma4(16 * D + 4 * lane, tq3_l + ((int64_t)id * H + h) * R3, dst + wid * R3 + 16 * D);
      }
    } else {
      const uint8_t* src = fp8_l + ((int64_t)e.y * H + h) * R8;
#pragma unroll
      for (int i = 0; i < OPS_W; ++i) {
        const int op = wid * OPS_W + i;
        if (op < NI)
          dma16<0>(vk, src + 16 * op, dst + 1024 * op);
        else
          dma16<0>(vv, src + 16 * D + 16 * (op - NI), dst + 16 * D + 1024 * (op - NI));
      }
      if (wid < 2 && lane < 2) dma4(4 * lane, scl_l + ((int64_t)e.y * H + h) * 8, dst + R8);
    }
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
    m_run[rt] = CM_INIT;
    l_run[rt] = 0.0f;
  }
  const float4v zero4 = {0.f, 0.f, 0.f, 0.f};
  const float smk = a.sm_log2;

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
        const float alpha = __builtin_amdgcn_exp2f(m_run[rt] - m_new);
        m_run[rt] = m_new;
        l_run[rt] *= alpha;
#pragma unroll
        for (int m = 0; m < CL; ++m) acc[m][rt] *= alpha;  // column = this lane's row
      }
#pragma unroll
      for (int k = 0; k < NK; ++k) {
        sc[rt][k] = __builtin_amdgcn_exp2f(sc[rt][k] - m_run[rt]);  // -inf -> 0
        l_run[rt] += sc[rt][k];
      }
    }
  };
  // S^T tile of one page for every row tile: A = the page's key bytes for
  // k-step S (from kop), B = the query terms
  // S^T tiles of NP pages (st[p][rt]); kop(p, s) gives page p's keys for
  // k-step s as fp16; LO adds the rotated query's low part
  auto qk = [&](float4v (*st)[CRT], auto np, auto loc, auto kop) {
    constexpr int NP = decltype(np)::value;
    constexpr bool LO = decltype(loc)::value;
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt) st[p][rt] = zero4;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      half8 K[NP];
#pragma unroll
      for (int p = 0; p < NP; ++p) K[p] = kop(p, s);
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt) {
#pragma unroll
        for (int p = 0; p < NP; ++p)
          st[p][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(K[p], qop[rt][s], st[p][rt], 0, 0, 0);
        if constexpr (LO) {
          const half8 ql = qlo[(rt * NS + s) * 64 + lane];
#pragma unroll
          for (int p = 0; p < NP; ++p)
            st[p][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(K[p], ql, st[p][rt], 0, 0, 0);
        }
      }
    }
  };

  // ---- the stage loop.  The TQ3 phase is software-pipelined: pass j runs the
  // PV product of stage j - 1 and the scores and softmax of stage j in one
  // straight-line block, so the matrix pipe keeps working through the
  // softmax.  A pass reads two ring slots (j - 1 and j); the barrier at its
  // start frees the slot of stage j - 2 for stage j + CSLOTS - 2.
  const int n_pre = min(CSLOTS - 2, n_st);
  for (int k = 0; k < n_pre; ++k) issue(stage_at(c_iss, k), k);
  build_q(true);
  // Stage j's copies have landed (this wave's by its vmcnt, everyone's by the
  // barrier); every wave is done with stage j - 2.
  auto next_stage = [&](int j) {
    if (j + CSLOTS - 2 <= n_st) {
      if (wid < 2)
        wait_vmcnt<(CSLOTS - 3) * (OPS_W + 1)>();
      else
        wait_vmcnt<(CSLOTS - 3) * OPS_W>();
    } else {
      wait_vmcnt<0>();
    }
    wait_lgkm0();  // this wave's reads of earlier stages are done
    __builtin_amdgcn_s_barrier();
    __asm__ __volatile__("" ::: "memory");
    if (j + CSLOTS - 2 < n_st) issue(stage_at(c_iss, j + CSLOTS - 2), (j + CSLOTS - 2) % CSLOTS);
  };
  // last token each row may see: min(S - 1, its position); -1 for rows past
  // the request's rows (all masked)
  int lim[CRT];
#pragma unroll
  for (int rt = 0; rt < CRT; ++rt) lim[rt] = min(S - 1, posr[rt]);

  // Scores and weights of the TQ3 pair e in ring slot ra: weights into pH,
  // pL (fp16 hi + lo: one token can carry most of a row's mass, and its
  // weight, taken against a lagging reference max, is then not a power of
  // two; a single fp16 rounding of it moves the output by up to 2^-12 of that
  // token's value) and Bz (this lane's weight sums of pages a and b, hi then
  // lo, for the zero term).  The reference max moves (lazily, when a score
  // passes it by 2^8) without a branch: alpha[rt] is the factor the
  // accumulators still owe, 1 where the reference stayed; the return value
  // says whether any row of the wave moved.
  auto tq3_scores = [&](const uint8_t* ra, const int4& e, half8* pH, half8* pL, half8* Bz,
                        float* alpha) {
    const uint8_t* rb2 = ra + R3;
    uint32_t kA[NDW], kB[NDW];
    read_chunk<NDW>(kA, ra, 16 * lg + ln);
    read_chunk<NDW>(kB, rb2, 16 * lg + ln);
    const uint2 gA = *reinterpret_cast<const uint2*>(ra + 12 * D + 8 * lg);
    const uint2 gB = *reinterpret_cast<const uint2*>(rb2 + 12 * D + 8 * lg);
    float4v st2[2][CRT];
    qk(st2, std::integral_constant<int, 2>{}, std::true_type{}, [&](int p, int sk) {
      const uint32_t* kc = p ? kB : kA;
      const uint32_t c0 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kc, 2 * sk));
      const uint32_t c1 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kc, 2 * sk + 1));
      return h8(cvt_lo(c0), cvt_hi(c0), cvt_lo(c1), cvt_hi(c1));
    });
    // scores (tokens 4 lg + i of pages a and b), causal and length masks
    const _Float16* ga = reinterpret_cast<const _Float16*>(&gA);
    const _Float16* gb = reinterpret_cast<const _Float16*>(&gB);
    const int ta = e.x * PAGE + 4 * lg, tb = e.z * PAGE + 4 * lg;
    bool moved = false;
#pragma unroll
    for (int rt = 0; rt < CRT; ++rt) {
      float sc[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sc[i] = ta + i <= lim[rt] ? st2[0][rt][i] * ((float)ga[i] * smk) : -INFINITY;
        sc[4 + i] = tb + i <= lim[rt] ? st2[1][rt][i] * ((float)gb[i] * smk) : -INFINITY;
      }
      float mx = sc[0];
#pragma unroll
      for (int k = 1; k < 8; ++k) mx = fmaxf(mx, sc[k]);
      mx = max4rows(mx);
      const bool need = mx > m_run[rt] + 8.0f;
      const float m_new = need ? mx : m_run[rt];
      alpha[rt] = __builtin_amdgcn_exp2f(m_run[rt] - m_new);
      m_run[rt] = m_new;
      moved |= need;
      float lsum = 0.0f;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        sc[k] = __builtin_amdgcn_exp2f(sc[k] - m_new);  // -inf -> 0
        lsum += sc[k];
      }
      l_run[rt] = fmaf(l_run[rt], alpha[rt], lsum);
      uint32_t hh[4], ll[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) split2(sc[2 * k], sc[2 * k + 1], hh[k], ll[k]);
      pH[rt] = h8u(hh[0], hh[1], hh[2], hh[3]);
      pL[rt] = h8u(ll[0], ll[1], ll[2], ll[3]);
      const float ra_ = (sc[0] + sc[1]) + (sc[2] + sc[3]);
      const float rb_ = (sc[4] + sc[5]) + (sc[6] + sc[7]);
      uint32_t zh, zl;
      split2(ra_, rb_, zh, zl);
      Bz[rt] = h8u(zh, zl, 0u, 0u);
    }
    return __any(moved);
  };
  // O^T += V^T P^T for the TQ3 pair in ring slot ra, with exact V operands:
  // v = zero + scale * code is split as scale_hi * code + scale_lo * code +
  // zero, scale_hi keeping 8 significant bits of the fp16 scale (so 3-bit
  // codes times it are exact in fp16) and scale_lo the remaining 3.  The
  // products that reach fp32 accuracy: (hi + lo weights) x scale_hi term, hi
  // weights x scale_lo term (lo x scale_lo sits below 2^-19 of the value), and
  // the zero term as zero_a (sum of weights over page a) + zero_b (same for
  // b), whose sums the MFMA completes across the four lane groups.
  auto tq3_pv = [&](const uint8_t* ra, const half8* pH, const half8* pL, const half8* Bz) {
    const uint8_t* rb2 = ra + R3;
    uint32_t vA[NDW], vB[NDW];
    read_chunk<NDW>(vA, ra + 6 * D, 16 * lg + ln);
    read_chunk<NDW>(vB, rb2 + 6 * D, 16 * lg + ln);
    const half2v* sca = reinterpret_cast<const half2v*>(ra + 12 * D + 32 + 2 * CL * ln);
    const half2v* zra = reinterpret_cast<const half2v*>(ra + 14 * D + 32 + 2 * CL * ln);
    const half2v* scb = reinterpret_cast<const half2v*>(rb2 + 12 * D + 32 + 2 * CL * ln);
    const half2v* zrb = reinterpret_cast<const half2v*>(rb2 + 14 * D + 32 + 2 * CL * ln);
#pragma unroll
    for (int m2 = 0; m2 < CL / 2; ++m2) {
      const half2v s2a = sca[m2], s2b = scb[m2], z2a = zra[m2], z2b = zrb[m2];
      const half2v sha = hi8x2(s2a), shb = hi8x2(s2b);
      const half2v sla = s2a - sha, slb = s2b - shb;  // exact
#pragma unroll
      for (int mm = 0; mm < 2; ++mm) {
        const int m = 2 * m2 + mm;
        const uint32_t ua = quad_sel<NDW>(vA, m), ub = quad_sel<NDW>(vB, m);
        const half2v ca01 = cvt_code<false>(ua), ca23 = cvt_code<true>(ua);
        const half2v cb01 = cvt_code<false>(ub), cb23 = cvt_code<true>(ub);
        const half2v sah = bcast(sha[mm]), sal = bcast(sla[mm]);
        const half2v sbh = bcast(shb[mm]), sbl = bcast(slb[mm]);
        const half8 A1 = h8(ca01 * sah, ca23 * sah, cb01 * sbh, cb23 * sbh);
        const half8 A2 = h8(ca01 * sal, ca23 * sal, cb01 * sbl, cb23 * sbl);
        const _Float16 za = z2a[mm], zb = z2b[mm];
        const half8 Az = half8{za, zb, za, zb, (_Float16)0.0f, (_Float16)0.0f, (_Float16)0.0f,
                               (_Float16)0.0f};
#pragma unroll
        for (int rt = 0; rt < CRT; ++rt) {
          acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A1, pH[rt], acc[m][rt], 0, 0, 0);
          acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A2, pH[rt], acc[m][rt], 0, 0, 0);
          acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A1, pL[rt], acc[m][rt], 0, 0, 0);
          acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(Az, Bz[rt], acc[m][rt], 0, 0, 0);
        }
      }
    }
  };
  auto rescale = [&](const float* alpha) {
#pragma unroll
    for (int m = 0; m < CL; ++m)
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt) acc[m][rt] *= alpha[rt];  // column = this lane's row
  };

  {
    half8 pH[CRT], pL[CRT], Bz[CRT];  // weights of the stage whose PV is pending
    if (st3 > 0) {
      next_stage(0);
      float alpha[CRT];
      (void)tq3_scores(smem, stage_at(c_cmp, 0), pH, pL, Bz, alpha);  // accumulators still zero
    }
    for (int j = 1; j < st3; ++j) {
      next_stage(j);
      const int4 e = stage_at(c_cmp, j);
      tq3_pv(smem + ((j - 1) % CSLOTS) * STAGE, pH, pL, Bz);
      half8 nH[CRT], nL[CRT], nZ[CRT];
      float alpha[CRT];
      if (tq3_scores(smem + (j % CSLOTS) * STAGE, e, nH, nL, nZ, alpha)) rescale(alpha);
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt) {
        pH[rt] = nH[rt];
        pL[rt] = nL[rt];
        Bz[rt] = nZ[rt];
      }
    }
    if (st3 > 0) tq3_pv(smem + ((st3 - 1) % CSLOTS) * STAGE, pH, pL, Bz);
  }
  if (st3 < n_st) build_q(false);  // plain queries for the FP8 pages
  for (int j = st3; j < n_st; ++j) {
    next_stage(j);
    const int4 e = stage_at(c_cmp, j);
    const uint8_t* ra = smem + (j % CSLOTS) * STAGE;
    {
      // ---------------- one FP8 page
      // block-permuted page (see dma_fp8_page): lane l's w-th 16 bytes at 64 w + l
      const uint4* pk = reinterpret_cast<const uint4*>(ra) + lane;
      const uint32_t* pv = reinterpret_cast<const uint32_t*>(ra + PAGE * D);
      const float2 ksv = *reinterpret_cast<const float2*>(ra + R8);
      float4v st1[1][CRT];
      qk(st1, std::integral_constant<int, 1>{}, std::false_type{}, [&](int, int sk) {
        // lane l's K bytes: channels QQ lg + 16 w .. at LDS block 64 w + l
        const uint2 kw = reinterpret_cast<const uint2*>(pk + 64 * (sk >> 1))[sk & 1];
        return h8(cvt_lo(kw.x), cvt_hi(kw.x), cvt_lo(kw.y), cvt_hi(kw.y));
      });
      float sc[CRT][8];
      {
        const int ta = e.x * PAGE + 4 * lg;
        const float kk = ksv.x * smk;
#pragma unroll
        for (int rt = 0; rt < CRT; ++rt)
#pragma unroll
          for (int i = 0; i < 4; ++i) sc[rt][i] = ta + i <= lim[rt] ? st1[0][rt][i] * kk : -INFINITY;
      }
      softmax(sc, std::integral_constant<int, 4>{});
      // the page's V scale folded into the weights, carried as an fp16 pair
      // (hi in k-slots 0-3, lo in 4-7, against the four values twice)
      half8 pB[CRT];
#pragma unroll
      for (int rt = 0; rt < CRT; ++rt) {
        uint32_t h01, l01, h23, l23;
        split2(sc[rt][0] * ksv.y, sc[rt][1] * ksv.y, h01, l01);
        split2(sc[rt][2] * ksv.y, sc[rt][3] * ksv.y, h23, l23);
        pB[rt] = h8u(h01, h23, l01, l23);
      }
      // lane-chunk (ln, lg) of V: dword m = tokens 4 lg .. 4 lg + 3 of channel CL ln + m
#pragma unroll
      for (int m4 = 0; m4 < CL / 4; ++m4) {
        const uint4 x = reinterpret_cast<const uint4*>(pv)[64 * m4 + lane];
        const uint32_t vw[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int mm = 0; mm < 4; ++mm) {
          const int m = 4 * m4 + mm;
          const half2v v01 = cvt_lo(vw[mm]), v23 = cvt_hi(vw[mm]);
          const half8 Av = h8(v01, v23, v01, v23);
#pragma unroll
          for (int rt = 0; rt < CRT; ++rt)
            acc[m][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(Av, pB[rt], acc[m][rt], 0, 0, 0);
        }
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
  const size_t lds = (size_t)CSLOTS * 2 * tq3_region_bytes(P.d) +  // the shared ring
                     (size_t)CW * tiles * (P.d / 32) * 64 * 16;      // rotated-query low parts
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
