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
// GQA group) pair; each wave owns one tile of 32 rows.  The workgroup streams
// every page of its request, TQ3 pairs first and FP8 pages after, through one
// LDS ring shared by its waves: each wave issues a quarter of every stage's
// direct HBM -> LDS copies, and one barrier per stage both publishes the
// stage and frees the slot read two stages before.  All products run on
// v_mfma_f32_32x32x16_f16 (on gfx950 it sustains about 1.7x the rate of the
// 16x16x32 shape):
//   S^T = K Q^T: M = 32 tokens (the two pages of a TQ3 pair; one FP8 page
//                and 16 zero rows), N = the 32 query rows, K = 16 channels;
//                TQ3 codes -> E4M3 codebook bytes (one v_perm per 4 codes)
//                -> fp16 against the rotated query as an fp16 hi + lo pair
//                (two MFMAs), FP8 keys -> fp16 against the plain query (exact
//                in fp16, one MFMA);
//   online softmax per query row in base 2 (lazy rescale, threshold 2^8),
//                causal mask token <= position of the query;
//   O^T += V^T P^T: M = 32 channels, N = the 32 query rows, K = the 16
//                tokens of one page: a lane's score outputs are exactly the 8
//                tokens per page its weight operand holds, so the weights
//                never move between lanes.  Weights as an fp16 hi + lo pair;
//                TQ3 values as exact fp16 operands (high and low parts of
//                scale * code) with the zero term as one rank-2 product of
//                the pages' zeros and weight sums per stage; FP8 values
//                exact, the page's V scale folded into the weights.
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

// Byte selector of the codes of quad 2 mb + h of a chunk (h = 0 or 1, per
// lane): quad_sel with the quad's low bit taken from a lane value.
template <int NDW>
__device__ __forceinline__ uint32_t quad_pair_sel(const uint32_t* Dw, int mb, int h) {
  if (mb < NDW) return (Dw[mb] >> (3 * h)) & 0x07070707u;
  const int p = mb - NDW;
  const uint32_t q0 = ((Dw[3 * p] >> 6) & 0x03030303u) | ((Dw[3 * p + 1] >> 4) & 0x04040404u);
  const uint32_t q1 = ((Dw[3 * p + 1] >> 7) & 0x01010101u) | ((Dw[3 * p + 2] >> 5) & 0x06060606u);
  return h ? q1 : q0;
}
// half h of x broadcast to both halves
__device__ __forceinline__ half2v bcast_half(half2v x, int h) {
  const uint32_t b = __builtin_bit_cast(uint32_t, x);
  return __builtin_bit_cast(half2v, __builtin_amdgcn_perm(b, b, h ? 0x03020302u : 0x01000100u));
}

template <int D>
__global__ __launch_bounds__(64 * CW, 1) void chunk_kernel(ChunkArgs a) {
  constexpr int NDW = 3 * D / 128, CL = D / 16, QQ = D / 4;
  constexpr int NKS = D / 16;   // k-steps of the score product (16 channels each)
  constexpr int NMB = D / 32;   // 32-channel blocks of the output
  constexpr int KPC = QQ / 8;   // k-steps per key chunk (a chunk holds QQ channels)
  constexpr int R3 = (int)tq3_region_bytes(D);
  constexpr int R8 = (int)fp8_region_bytes(D);
  constexpr int STAGE = 2 * R3;       // a TQ3 page pair, or one FP8 page + its two scales
  constexpr int MAIN_KB = 16 * D / 1024;  // whole KiB of a TQ3 page (its last 32 bytes aside)
  constexpr int OPS_W = 2 * MAIN_KB / CW;  // 1-KiB copies per wave per stage
  constexpr int NI = D / 64;               // 1-KiB copies per half of an FP8 page
  static_assert(2 * MAIN_KB % CW == 0 && 2 * NI == CW * OPS_W, "copies split evenly");
  static_assert(R3 == 1024 * MAIN_KB + 32, "TQ3 page = whole KiB + a 32-byte tail");
  static_assert(R8 + 8 <= STAGE, "an FP8 page and its scales fit one stage");
  static_assert(CL == 2 * NMB, "a lane's chunk row covers two channels per block");
  extern __shared__ __align__(16) uint8_t smem[];
  const PoolView& P = a.P;
  const int r = blockIdx.z, h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  // MFMA lane roles: li = lane % 32 (row of A, column of B and of the
  // output), lg = lane / 32 (k-slot group)
  const int li = lane & 31, lg = lane >> 5;
  const int ln = lane & 15, l4 = lane >> 4;  // the copy layout's view of the lane
  const int G = P.group, H = P.n_kv_heads, Hq = H * G;
  const int mp = a.max_pages;

  // ---- request and rows of this wave
  const int q0 = a.cu_q[r], q1 = a.cu_q[r + 1];
  const int nq = q1 - q0;
  const int S = a.seq_lens[r];
  const bool range_ok = q0 >= 0 && nq >= 0 && q1 <= a.n_q_total;
  const int rows_r = range_ok ? nq * G : 0;
  const int rb = blockIdx.x * (CW * 32) + wid * 32;
  if (!range_ok || nq < 1 || S < nq || S > mp * PAGE) {  // workgroup-uniform
    if (blockIdx.x == 0 && tid == 0) atomicOr(&P.ctrl[CTRL_ERR], (int)MKV_DEVERR_RANGE);
    // rows that can be located get zeros
    const int rho = rb + li;
    if (rho < rows_r) {
      float* o = a.out + ((int64_t)(q0 + rho / G) * Hq + h * G + rho % G) * D;
      for (int c = lg; c < D; c += 2) o[c] = 0.0f;
    }
    return;
  }
  if (blockIdx.x * (CW * 32) >= rows_r) return;  // whole workgroup past the rows
  // Waves whose rows all lie past the request's rows still take part in the
  // copies and barriers; their scores are all masked.
  const int P0 = S - nq;  // position of the chunk's first query
  // this lane's query row rb + li: last token it may see, min(S - 1,
  // position); -1 for rows past the request's rows (all masked)
  const int rho_l = rb + li;
  const int lim = rho_l < rows_r ? min(S - 1, P0 + rho_l / G) : -1;

  // ---- query operand: B of S^T = K Q^T.  Lane (li, lg) holds, for k-step s,
  // channels (D/2) lg + 8 s + b (b < 8) of query row rb + li (the MFMA pairs
  // slot b of lane group lg in A and B; the key operands use the same
  // channel order).  TQ3 pages use q_rot = R q (R = d^-1/2 H diag(sigma)) as
  // an fp16 pair hi + lo (fp32 accuracy: two MFMAs), FP8 pages the plain q
  // (bf16 -> fp16 is exact: one MFMA).  Keys enter as fp16 too: the fp8 MFMA
  // adds its products in groups aligned to the group's largest one and keeps
  // only about 15 bits there, which moved chunk outputs by up to 2e-3 where
  // keys carry large norms.
  half8 qop[NKS];
  // the rotated query's fp16 low part lives in this wave's LDS area after the
  // ring: [k-step][lane]
  half8* qlo = reinterpret_cast<half8*>(smem + CSLOTS * STAGE) + wid * NKS * 64;
  auto build_q = [&](bool rotated) {
    const int rho = min(rho_l, rows_r - 1);
    const uint16_t* qrow = a.q + ((int64_t)(q0 + rho / G) * Hq + h * G + rho % G) * D + (D / 2) * lg;
    float x[NKS][8];
#pragma unroll
    for (int s = 0; s < NKS; ++s) {
      const uint4 raw = *reinterpret_cast<const uint4*>(qrow + 8 * s);
      const uint16_t* hb = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
      for (int j = 0; j < 8; ++j) x[s][j] = bf16_to_f32(hb[j]);
    }
    if (rotated) {
      const int8_t* sg = P.sigma + (D / 2) * lg;
#pragma unroll
      for (int s = 0; s < NKS; ++s)
#pragma unroll
        for (int j = 0; j < 8; ++j) x[s][j] *= (float)sg[8 * s + j];
      // Walsh-Hadamard butterflies over the channel bits: j (strides 1-4)
      // and s (strides 8 .. D/4) inside the lane, lg (stride D/2) across
      // lanes l ^ 32; the stages commute
#pragma unroll
      for (int st = 1; st < 8; st <<= 1)
#pragma unroll
        for (int s = 0; s < NKS; ++s)
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (!(j & st)) {
              const float x0 = x[s][j], x1 = x[s][j + st];
              x[s][j] = x0 + x1;
              x[s][j + st] = x0 - x1;
            }
#pragma unroll
      for (int st = 1; st < NKS; st <<= 1)
#pragma unroll
        for (int s = 0; s < NKS; ++s)
          if (!(s & st)) {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              const float x0 = x[s][j], x1 = x[s + st][j];
              x[s][j] = x0 + x1;
              x[s + st][j] = x0 - x1;
            }
          }
      const float sgn32 = (lane & 32) ? -1.0f : 1.0f;
      const float qscale = rsqrtf((float)D);
#pragma unroll
      for (int s = 0; s < NKS; ++s)
#pragma unroll
        for (int j = 0; j < 8; ++j)
          x[s][j] = fmaf(sgn32, x[s][j], lane_xor<32>(x[s][j], lane)) * qscale;
    }
#pragma unroll
    for (int s = 0; s < NKS; ++s) {
      half8 lo;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        qop[s][j] = (_Float16)x[s][j];
        lo[j] = (_Float16)(x[s][j] - (float)qop[s][j]);
      }
      if (rotated) qlo[s * 64 + lane] = lo;
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
  const uint32_t vk = 16u * (uint32_t)(ln * (D / 16) + l4 * NI);
  const uint32_t vv = 16u * (uint32_t)((ln * 4 + l4) * NI);
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

  // ---- accumulators: O^T tile (32 channels x the 32 query rows) per block
  // mb.  Lane (li, lg), element e holds query row rb + li and tile row rr =
  // 8 (e / 4) + 4 lg + e % 4, which is channel CL (rr % 16) + 2 mb + rr / 16
  // (a lane's V chunk row rr % 16 then serves every block).
  float16v acc[NMB];
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb) acc[mb] = float16v{};
  float m_run = CM_INIT, l_run = 0.0f;  // this lane's row; l_run over its tokens
  const float smk = a.sm_log2;
  const int hh = li >> 4;   // which of the block's two channels of the chunk row
  const int rrow = li & 15; // this lane's chunk row (A operands of PV)

  // Online softmax over the scores sc[16] of this lane's query row (its 16
  // tokens of the tile; the other 16 sit in lane l ^ 32), given before the
  // softmax scale log2(e)/sqrt(d), which enters with the max subtraction.  The reference max
  // moves (lazily, when a score passes it by 2^8) without a branch: alpha is
  // the factor the accumulators still owe, 1 where the reference stayed; the
  // return value says whether any row of the wave moved.
  auto softmax = [&](float* sc, float& alpha) {
    float mx = sc[0];
#pragma unroll
    for (int k = 1; k < 16; ++k) mx = fmaxf(mx, sc[k]);
    mx = fmaxf(mx, lane_xor<32>(mx, lane)) * smk;
    const bool need = mx > m_run + 8.0f;
    const float m_new = need ? mx : m_run;
    alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    float lsum = 0.0f;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      sc[k] = __builtin_amdgcn_exp2f(fmaf(sc[k], smk, -m_new));  // -inf -> 0
      lsum += sc[k];
    }
    l_run = fmaf(l_run, alpha, lsum);
    return __any(need);
  };
  // weights p[0..7] as an fp16 hi + lo pair (one token can carry most of a
  // row's mass, and its weight, taken against a lagging reference max, is
  // then not a power of two; a single fp16 rounding of it moves the output
  // by up to 2^-12 of that token's value)
  auto split8 = [&](const float* p, half8& hi, half8& lo) {
    uint32_t hh4[4], ll4[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) split2(p[2 * k], p[2 * k + 1], hh4[k], ll4[k]);
    hi = h8u(hh4[0], hh4[1], hh4[2], hh4[3]);
    lo = h8u(ll4[0], ll4[1], ll4[2], ll4[3]);
  };
  struct TqW {
    half8 ha, la, hb, lb, z;  // weights of pages a and b (hi, lo); zero-term operand
  };

  // Scores and weights of the TQ3 pair e in ring slot ra.  The score tile's
  // rows are the pair's 32 tokens (page a, then page b); lane (li, lg)
  // receives tokens 4 lg .. 4 lg + 3 and 8 + 4 lg .. of each page, which are
  // exactly the k-slots of its weight operand.
  auto tq3_scores = [&](const uint8_t* ra, const int4& e, TqW& w, float& alpha) {
    const uint8_t* pg = ra + (li >= 16 ? R3 : 0);
    uint32_t kc0[NDW], kc1[NDW];
    read_chunk<NDW>(kc0, pg, 16 * (2 * lg) + rrow);
    read_chunk<NDW>(kc1, pg, 16 * (2 * lg + 1) + rrow);
    const uint2 ga0 = *reinterpret_cast<const uint2*>(ra + 12 * D + 8 * lg);
    const uint2 ga1 = *reinterpret_cast<const uint2*>(ra + 12 * D + 16 + 8 * lg);
    const uint2 gb0 = *reinterpret_cast<const uint2*>(ra + R3 + 12 * D + 8 * lg);
    const uint2 gb1 = *reinterpret_cast<const uint2*>(ra + R3 + 12 * D + 16 + 8 * lg);
    float16v st = {};
#pragma unroll
    for (int s = 0; s < NKS; ++s) {
      const uint32_t* kc = s < KPC ? kc0 : kc1;
      const int qd = 2 * (s % KPC);
      const uint32_t c0 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kc, qd));
      const uint32_t c1 = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kc, qd + 1));
      const half8 K = h8(cvt_lo(c0), cvt_hi(c0), cvt_lo(c1), cvt_hi(c1));
      st = __builtin_amdgcn_mfma_f32_32x32x16_f16(K, qop[s], st, 0, 0, 0);
      st = __builtin_amdgcn_mfma_f32_32x32x16_f16(K, qlo[s * 64 + lane], st, 0, 0, 0);
    }
    // element e: token 8 (e / 4) + 4 lg + e % 4 of the pair (page a below 16)
    const _Float16* gam[4] = {reinterpret_cast<const _Float16*>(&ga0), reinterpret_cast<const _Float16*>(&ga1),
                              reinterpret_cast<const _Float16*>(&gb0), reinterpret_cast<const _Float16*>(&gb1)};
    float sc[16];
    if ((max(e.x, e.z) + 1) * PAGE <= P0 + 1) {
      // the pair lies wholly before the chunk's first query: no mask
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4)
#pragma unroll
        for (int u = 0; u < 4; ++u) sc[4 * e4 + u] = st[4 * e4 + u] * (float)gam[e4][u];
    } else {
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int t0 = (e4 < 2 ? e.x : e.z) * PAGE + 8 * (e4 & 1) + 4 * lg;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          sc[4 * e4 + u] = t0 + u <= lim ? st[4 * e4 + u] * (float)gam[e4][u] : -INFINITY;
      }
    }
    const bool moved = softmax(sc, alpha);
    split8(sc, w.ha, w.la);
    split8(sc + 8, w.hb, w.lb);
    const float ra_ = ((sc[0] + sc[1]) + (sc[2] + sc[3])) + ((sc[4] + sc[5]) + (sc[6] + sc[7]));
    const float rb_ = ((sc[8] + sc[9]) + (sc[10] + sc[11])) + ((sc[12] + sc[13]) + (sc[14] + sc[15]));
    uint32_t zh, zl;
    split2(ra_, rb_, zh, zl);
    w.z = h8u(zh, zl, 0u, 0u);  // (R_a, R_b) hi, then lo
    return moved;
  };
  // O^T += V^T P^T for the TQ3 pair in ring slot ra, with exact V operands:
  // v = zero + scale * code is split as scale_hi * code + scale_lo * code +
  // zero, scale_hi keeping 8 significant bits of the fp16 scale (so 3-bit
  // codes times it are exact in fp16) and scale_lo the remaining 3.  The
  // products that reach fp32 accuracy: (hi + lo weights) x scale_hi term, hi
  // weights x scale_lo term (lo x scale_lo sits below 2^-19 of the value), and
  // the zero term as zero_a (sum of weights over page a) + zero_b (same for
  // b), whose sums the MFMA completes across the two lane groups.
  auto tq3_pv = [&](const uint8_t* ra, const TqW& w) {
    uint32_t va0[NDW], va2[NDW], vb0[NDW], vb2[NDW];
    read_chunk<NDW>(va0, ra + 6 * D, 16 * lg + rrow);
    read_chunk<NDW>(va2, ra + 6 * D, 16 * (lg + 2) + rrow);
    read_chunk<NDW>(vb0, ra + R3 + 6 * D, 16 * lg + rrow);
    read_chunk<NDW>(vb2, ra + R3 + 6 * D, 16 * (lg + 2) + rrow);
    const half2v* sca = reinterpret_cast<const half2v*>(ra + 12 * D + 32 + 2 * CL * rrow);
    const half2v* zra = reinterpret_cast<const half2v*>(ra + 14 * D + 32 + 2 * CL * rrow);
    const half2v* scb = reinterpret_cast<const half2v*>(ra + R3 + 12 * D + 32 + 2 * CL * rrow);
    const half2v* zrb = reinterpret_cast<const half2v*>(ra + R3 + 14 * D + 32 + 2 * CL * rrow);
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
      const half2v s2a = sca[mb], s2b = scb[mb];
      const half2v sha = hi8x2(s2a), shb = hi8x2(s2b);
      const half2v sah = bcast_half(sha, hh), sal = bcast_half(s2a - sha, hh);  // exact split
      const half2v sbh = bcast_half(shb, hh), sbl = bcast_half(s2b - shb, hh);
      const uint32_t ua0 = quad_pair_sel<NDW>(va0, mb, hh), ua2 = quad_pair_sel<NDW>(va2, mb, hh);
      const uint32_t ub0 = quad_pair_sel<NDW>(vb0, mb, hh), ub2 = quad_pair_sel<NDW>(vb2, mb, hh);
      const half2v a01 = cvt_code<false>(ua0), a23 = cvt_code<true>(ua0);
      const half2v a45 = cvt_code<false>(ua2), a67 = cvt_code<true>(ua2);
      const half2v b01 = cvt_code<false>(ub0), b23 = cvt_code<true>(ub0);
      const half2v b45 = cvt_code<false>(ub2), b67 = cvt_code<true>(ub2);
      const half8 A1a = h8(a01 * sah, a23 * sah, a45 * sah, a67 * sah);
      const half8 A2a = h8(a01 * sal, a23 * sal, a45 * sal, a67 * sal);
      const half8 A1b = h8(b01 * sbh, b23 * sbh, b45 * sbh, b67 * sbh);
      const half8 A2b = h8(b01 * sbl, b23 * sbl, b45 * sbl, b67 * sbl);
      const _Float16 za = bcast_half(zra[mb], hh)[0], zb = bcast_half(zrb[mb], hh)[0];
      const half8 Az = half8{za, zb, za, zb, (_Float16)0.0f, (_Float16)0.0f, (_Float16)0.0f,
                             (_Float16)0.0f};
      acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(A1a, w.ha, acc[mb], 0, 0, 0);
      acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(A2a, w.ha, acc[mb], 0, 0, 0);
      acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(A1a, w.la, acc[mb], 0, 0, 0);
      acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(A1b, w.hb, acc[mb], 0, 0, 0);
      acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(A2b, w.hb, acc[mb], 0, 0, 0);
      acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(A1b, w.lb, acc[mb], 0, 0, 0);
      acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(Az, w.z, acc[mb], 0, 0, 0);
    }
  };
  auto rescale = [&](float alpha) {
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) acc[mb] *= alpha;  // column = this lane's row
  };

  // ---- the stage loop.  The TQ3 phase is software-pipelined: pass j runs the
  // PV product of stage j - 1 and the scores and softmax of stage j in one
  // straight-line block.  A pass reads two ring slots (j - 1 and j); the
  // barrier at its start frees the slot of stage j - 2 for stage j + CSLOTS - 2.
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
  {
    TqW w;  // weights of the stage whose PV is pending
    if (st3 > 0) {
      next_stage(0);
      float alpha;
      (void)tq3_scores(smem, stage_at(c_cmp, 0), w, alpha);  // accumulators still zero
    }
    for (int j = 1; j < st3; ++j) {
      next_stage(j);
      const int4 e = stage_at(c_cmp, j);
      tq3_pv(smem + ((j - 1) % CSLOTS) * STAGE, w);
      TqW wn;
      float alpha;
      if (tq3_scores(smem + (j % CSLOTS) * STAGE, e, wn, alpha)) rescale(alpha);
      w = wn;
    }
    if (st3 > 0) tq3_pv(smem + ((st3 - 1) % CSLOTS) * STAGE, w);
  }
  if (st3 < n_st) build_q(false);  // plain queries for the FP8 pages
  for (int j = st3; j < n_st; ++j) {
    next_stage(j);
    const int4 e = stage_at(c_cmp, j);
    const uint8_t* ra = smem + (j % CSLOTS) * STAGE;
    // ---------------- one FP8 page: score rows 0-15 are its tokens, 16-31 zero
    // block-permuted page (see dma_fp8_page): 16-byte block 64 w + 16 Q + t
    // holds bytes 16 w .. of token t's channel quarter Q (K), and of the
    // lane-chunk (t, Q) (V)
    const uint2* pk = reinterpret_cast<const uint2*>(ra);
    const float2 ksv = *reinterpret_cast<const float2*>(ra + R8);
    float16v st = {};
#pragma unroll
    for (int s = 0; s < NKS; ++s) {
      const int Q = 2 * lg + s / KPC, off = 8 * (s % KPC);
      half8 K = {};
      if (li < 16) {
        const uint2 kw = pk[2 * (64 * (off / 16) + 16 * Q + li) + (off / 8) % 2];
        K = h8(cvt_lo(kw.x), cvt_hi(kw.x), cvt_lo(kw.y), cvt_hi(kw.y));
      }
      st = __builtin_amdgcn_mfma_f32_32x32x16_f16(K, qop[s], st, 0, 0, 0);
    }
    float sc[16];
    {
      const float kk = ksv.x;
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int t0 = e.x * PAGE + 8 * (e4 & 1) + 4 * lg;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          sc[4 * e4 + u] = (e4 < 2 && t0 + u <= lim) ? st[4 * e4 + u] * kk : -INFINITY;
      }
    }
    float alpha;
    if (softmax(sc, alpha)) rescale(alpha);
    // the page's V scale folded into the weights
    float pw[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) pw[k] = sc[k] * ksv.y;
    half8 pH, pL;
    split8(pw, pH, pL);
    // lane-chunks (rrow, lg) and (rrow, lg + 2) of V: dword m = tokens
    // 4 g' .. 4 g' + 3 of channel CL rrow + m
    const uint2* pv = reinterpret_cast<const uint2*>(ra + PAGE * D);
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
      const int blk = 64 * (mb / 2);
      const uint2 v0 = pv[2 * (blk + 16 * lg + rrow) + (mb & 1)];
      const uint2 v2 = pv[2 * (blk + 16 * (lg + 2) + rrow) + (mb & 1)];
      const uint32_t w0 = hh ? v0.y : v0.x, w2 = hh ? v2.y : v2.x;
      const half8 Av = h8(cvt_lo(w0), cvt_hi(w0), cvt_lo(w2), cvt_hi(w2));
      acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(Av, pH, acc[mb], 0, 0, 0);
      acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(Av, pL, acc[mb], 0, 0, 0);
    }
  }

  if (__any(bad_id) && lane == 0) atomicOr(&P.ctrl[CTRL_ERR], (int)MKV_DEVERR_RANGE);
  // ---- normalize and store: tile row rr = 8 kk + 4 lg + u (kk, u: the
  // lane's elements 4 kk + u and 8 + 4 kk + u) is chunk row rr % 16 = rr
  // for both halves hh = 0, 1 of every block, so channels CL rr .. CL rr + CL
  // - 1 are contiguous: channel CL rr + 2 mb + hh <- acc[mb][4 kk + 8 hh + u]
  const float L = l_run + lane_xor<32>(l_run, lane);
  if (rho_l < rows_r) {
    const float inv = L > 0.0f ? 1.0f / L : 0.0f;
    float* o = a.out + ((int64_t)(q0 + rho_l / G) * Hq + h * G + rho_l % G) * D;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int rr = 8 * kk + 4 * lg + u;
#pragma unroll
        for (int v = 0; v < NMB / 2; ++v)
          *reinterpret_cast<float4*>(o + CL * rr + 4 * v) =
              make_float4(acc[2 * v][4 * kk + u] * inv, acc[2 * v][4 * kk + 8 + u] * inv,
                          acc[2 * v + 1][4 * kk + u] * inv, acc[2 * v + 1][4 * kk + 8 + u] * inv);
      }
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
  const size_t lds = (size_t)CSLOTS * 2 * tq3_region_bytes(P.d) +  // the shared ring
                     (size_t)CW * (P.d / 16) * 64 * 16;              // rotated-query low parts
  const void* kern = P.d == 256 ? (const void*)chunk_kernel<256> : (const void*)chunk_kernel<128>;
  e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  // rows of one request: at most n_q_total queries x group heads
  const int64_t rows = (int64_t)n_q_total * P.group;
  const int wg_rows = CW * 32;
  const int blocks = (int)((rows + wg_rows - 1) / wg_rows);
  dim3 grid(blocks, P.n_kv_heads, n_req);
  void* args[] = {&a};
  e = hipLaunchKernel(kern, grid, dim3(64 * CW), args, lds, s);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace mkv
