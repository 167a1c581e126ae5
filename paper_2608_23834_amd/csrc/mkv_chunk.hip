// Causal chunked-prefill attention over mixed FP8/TQ3 pages on MFMA (the
// query chunk makes it a dense contraction).  The paper runs prefill on a
// generic dense path (Sec. 4.1); this variant keeps the pages in their two
// physical formats and applies the same score algebra as decode (Sec. 3.3):
// rotated queries against TQ3 key codes times the FP16 key-norm correction,
// plain queries against FP8 keys, one online softmax per query row.
//
// Launch: the partition kernel (compact per-format lists, Sec. 4.1), a stage
// table kernel (per request: the TQ3 pages in pairs, then the FP8 pages), a
// row-block table kernel (first 128-row block of each request) and the
// attention kernel.  Grid (row block over all requests, KV head); 512
// threads = 8 waves, one workgroup per CU, two waves per SIMD.  A query row
// is a (query token, head of the GQA group) pair; a workgroup owns 128 rows:
//  * four score waves of 32 rows each hold their rows' rotated queries as
//    three E4M3 terms in registers, copy their share of every stage (direct
//    HBM -> LDS copies into a ring of eight stages) and of the stage table,
//    unpack TQ3 pairs into MFMA operand layouts in LDS (key codes -> E4M3
//    codebook bytes, value codes as bytes, the V scale split for exact fp16
//    products).  Pass p issues S^T = K Q^T of pair p on
//    v_mfma_f32_32x32x64_f8f6f4 (M = the pair's 32 tokens, N = the 32 rows,
//    K = 64 channels; three MFMAs per k-step, one per query term) and,
//    between those MFMAs, finishes pair p - 1: the causal mask, the online
//    softmax in base 2 (lazy rescale, threshold 2^8) and the weights as fp16
//    hi + lo pairs, handed over in LDS;
//  * four PV waves, wave v owning the 32-channel blocks 2v, 2v + 1 of all
//    128 rows, hold O^T accumulators (32 channels x 32 rows per block and
//    score wave) and compute O^T += V^T P^T on v_mfma_f32_32x32x16_f16 (M =
//    32 channels, N = 32 rows, K = the 16 tokens of one page; a lane's score
//    outputs are exactly the 8 tokens per page its weight operand holds):
//    values as exact fp16 operands (scale_hi * code, scale_lo * code), the
//    zero term as one rank-2 product of the pages' zeros and weight sums,
//    applying the rescale the score waves passed along first.
// Pass p (one barrier): the score waves issue pair p's product and finish
// pair p - 1 while the PV waves take pair p - 2.  FP8 pages: the score waves
// score them on the f16 MFMA against the plain query (the fp8 MFMA keeps too
// few bits where FP8 keys carry large norms) with one zero-padded half of
// the tile, and fold the page's V scale into the weights; the PV waves read
// the page's values from the ring.  The workgroups of one (request, KV head)
// read the same pages at about the same time, so the page bytes come from
// L2 after the first reader.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "mkv_attn.h"
#include "mkv_internal.h"
#include "../../include/minima_kv.h"

namespace mkv {

constexpr int NSW = 4;       // score waves per chunk workgroup (one PV wave each)
constexpr int CW = 2 * NSW;  // waves per chunk workgroup
constexpr int CSLOTS = 8;    // raw stages in the shared ring
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
  const int4* stages;     // [n_req][max_pages] stage table (chunk_stages_kernel)
  const int32_t* rbo;     // [n_req + 1] first row block of each request (chunk_rows_kernel)
  float sm_log2;          // log2(e) / sqrt(d)
};

static size_t al256(size_t b) { return (b + 255) / 256 * 256; }

// workspace: the two compact lists, their counts and the stage table (one
// int4 per stage; the chunk kernel copies it in 1 KiB blocks, so 1 KiB of
// slack after it keeps the last block inside the workspace)
struct ChunkWs {
  size_t list8, list3, counts, stages, rbo, total;
};
static ChunkWs chunk_ws(int n_req, int max_pages) {
  ChunkWs w;
  const size_t lb = al256((size_t)n_req * max_pages * 2 * sizeof(int32_t));
  w.list8 = 0;
  w.list3 = lb;
  w.counts = 2 * lb;
  w.stages = w.counts + al256((size_t)n_req * 2 * sizeof(int32_t));
  w.rbo = w.stages + al256((size_t)n_req * max_pages * sizeof(int4) + 1024);
  w.total = w.rbo + al256((size_t)(n_req + 1) * sizeof(int32_t));
  return w;
}
size_t chunk_ws_bytes(int n_req, int max_pages, int n_q_total, int n_kv_heads, int group, int d) {
  (void)n_q_total; (void)n_kv_heads; (void)group; (void)d;
  return chunk_ws(n_req, max_pages).total;
}

// Stage table of a chunk call: per request, stage j -> {lp_a, id_a, lp_b,
// id_b}: the TQ3 pages in pairs (list entries 2 j, 2 j + 1; a missing page b
// is masked) first, then the FP8 pages one per stage (id_b = -1).  Ids
// outside the pool become page 0 with every token masked, and set the range
// error bit.
__global__ __launch_bounds__(256) void chunk_stages_kernel(int max_pages, int n_tq3, int n_fp8,
                                                           const int32_t* list8,
                                                           const int32_t* list3,
                                                           const int32_t* counts, int4* stages,
                                                           int32_t* err) {
  const int r = blockIdx.y, j = blockIdx.x * 256 + threadIdx.x;
  const int n8 = counts[2 * r], n3 = counts[2 * r + 1];
  const int st3 = (n3 + 1) / 2, n_st = st3 + n8;  // at most the request's pages
  if (j >= n_st) return;
  const int2* l3 = reinterpret_cast<const int2*>(list3) + (int64_t)r * max_pages;
  const int2* l8 = reinterpret_cast<const int2*>(list8) + (int64_t)r * max_pages;
  bool bad = false;
  auto checked = [&](int2 e, int n_ids) {
    if (e.y < 0 || e.y >= n_ids) {
      bad = true;
      return make_int2(CMASK_LP, 0);
    }
    return e;
  };
  int4 st;
  if (j < st3) {
    const int2 ea = checked(l3[2 * j], n_tq3);
    const int2 eb = 2 * j + 1 < n3 ? checked(l3[2 * j + 1], n_tq3) : make_int2(CMASK_LP, ea.y);
    st = make_int4(ea.x, ea.y, eb.x, eb.y);
  } else {
    const int2 e = checked(l8[j - st3], n_fp8);
    st = make_int4(e.x, e.y, 0, -1);
  }
  stages[(int64_t)r * max_pages + j] = st;
  if (bad) atomicOr(err, (int)MKV_DEVERR_RANGE);
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
// 2^-4 vanished and chunk outputs moved by up to 1.3e-3.)  The remainders
// a - hi are single mixed-precision FMAs (hi read as fp16) with neg1 = -1
// held in a register.
__device__ __forceinline__ void split2(float a, float b, float neg1, uint32_t& hi, uint32_t& lo) {
  const half2v h = {(_Float16)a, (_Float16)b};
  const half2v l = {(_Float16)__builtin_fmaf((float)h[0], neg1, a), (_Float16)__builtin_fmaf((float)h[1], neg1, b)};
  hi = __builtin_bit_cast(uint32_t, h);
  lo = __builtin_bit_cast(uint32_t, l);
}
__device__ __forceinline__ half8 h8u(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  typedef uint32_t u4v __attribute__((ext_vector_type(4)));
  return __builtin_bit_cast(half8, u4v{a, b, c, d});
}
constexpr float CM_INIT = -1.0e30f;  // running max before the first score (finite: no inf - inf)

// LDS of a chunk workgroup (bytes): the ring of raw stages, two buffers of
// unpacked key operands, two of unpacked value operands, two of the weights
// the score waves hand to the PV waves, the rows' softmax denominators for
// the final normalization, and three blocks of the stage table.
template <int D>
struct ChunkLds {
  static constexpr int NK8 = D / 64, NMB = D / 32;
  static constexpr int STAGE = 2 * (int)tq3_region_bytes(D);
  static constexpr int KB = NK8 * 64 * 32;            // key bytes [k-step][lane][32]
  static constexpr int VX = 2 * NMB * 64 * 8;         // value codes [page][block][lane][8]
  static constexpr int SX = 2 * NMB * 32 * 4;         // V scale (hi, lo) fp16 [page][block][row]
  static constexpr int VB = VX + SX + 2 * NMB * 32 * 2;  // + V zero fp16 [page][block][row]
  // weights of one stage from one score wave: 5 half8 operands per lane
  // ([field][lane][16]: page a hi, lo, page b hi, lo, zero term) and the
  // rescale factor per lane
  static constexpr int WF_ALPHA = 5 * 1024, WPW = WF_ALPHA + 256;
  static constexpr int KB0 = CSLOTS * STAGE;
  static constexpr int VB0 = KB0 + 2 * KB;
  static constexpr int WB0 = VB0 + 2 * VB;
  static constexpr int LB0 = WB0 + 2 * NSW * WPW;     // row denominators [score wave][32]
  static constexpr int LS0 = LB0 + NSW * 32 * 4;      // stage-table blocks [3][64 stages][16]
  static constexpr int TOTAL = LS0 + 3 * 1024;
  static_assert(KB % 16 == 0 && VB % 16 == 0 && STAGE % 16 == 0 && WPW % 16 == 0,
                "16-byte aligned buffers");
  static_assert(TOTAL <= 160 * 1024, "one workgroup's LDS");
};

// One 128-row block xb of request r and KV head h (the body of a chunk
// workgroup; every wave of the workgroup runs it).
template <int D>
__device__ __forceinline__ void chunk_block(const ChunkArgs& a, int r, int h, int xb, uint8_t* smem) {
  constexpr int NDW = 3 * D / 128, CL = D / 16, QQ = D / 4;
  constexpr int NKS = D / 16;   // k-steps of the FP8-page score product (16 channels each)
  constexpr int NK8 = D / 64;   // k-steps of the TQ3 score product (64 channels each)
  constexpr int NMB = D / 32;   // 32-channel blocks of the output
  constexpr int KPC = QQ / 8;   // FP8-page k-steps per channel quarter
  constexpr int R3 = (int)tq3_region_bytes(D);
  constexpr int R8 = (int)fp8_region_bytes(D);
  constexpr int STAGE = 2 * R3;       // a TQ3 page pair, or one FP8 page + its two scales
  constexpr int MAIN_KB = 16 * D / 1024;  // whole KiB of a TQ3 page (its last 32 bytes aside)
  constexpr int OPS_W = 2 * MAIN_KB / NSW;  // 1-KiB copies per score wave per stage
  constexpr int NI = D / 64;                // 1-KiB copies per half of an FP8 page
  using LY = ChunkLds<D>;
  static_assert(2 * MAIN_KB % NSW == 0 && 2 * NI == NSW * OPS_W, "copies split evenly");
  static_assert(R3 == 1024 * MAIN_KB + 32, "TQ3 page = whole KiB + a 32-byte tail");
  static_assert(R8 + 8 <= STAGE, "an FP8 page and its scales fit one stage");
  static_assert(CL == 2 * NMB, "a chunk row of V covers two channels per block");
  static_assert(CW == 2 * NSW, "one PV wave per score wave");
  const PoolView& P = a.P;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool score_wave = wid < NSW;
  const int sw = wid % NSW;  // score wave: its rows (PV waves: unused)
  // MFMA lane roles: li = lane % 32 (row of A, column of B and of the
  // output), lg = lane / 32 (k-slot group)
  const int li = lane & 31, lg = lane >> 5;
  const int ln = lane & 15, l4 = lane >> 4;  // the copy layout's view of the lane
  const int G = P.group, H = P.n_kv_heads, Hq = H * G;
  const int mp = a.max_pages;

  // ---- request and rows of this wave pair
  const int q0 = a.cu_q[r], q1 = a.cu_q[r + 1];
  const int nq = q1 - q0;
  const int S = a.seq_lens[r];
  const bool range_ok = q0 >= 0 && nq >= 0 && q1 <= a.n_q_total;
  const int rows_r = range_ok ? nq * G : 0;
  const int rb = xb * (NSW * 32) + sw * 32;
  if (!range_ok || nq < 1 || S < nq || S > mp * PAGE) {  // workgroup-uniform
    if (xb == 0 && tid == 0) atomicOr(&P.ctrl[CTRL_ERR], (int)MKV_DEVERR_RANGE);
    // rows that can be located get zeros
    const int rho = rb + li;
    if (score_wave && rho < rows_r) {
      float* o = a.out + ((int64_t)(q0 + rho / G) * Hq + h * G + rho % G) * D;
      for (int c = lg; c < D; c += 2) o[c] = 0.0f;
    }
    return;
  }
  if (xb * (NSW * 32) >= rows_r) return;  // whole workgroup past the rows (not with the row-block table)
  // Score waves whose rows all lie past the request's rows still take part
  // in the copies, the unpacking and the barriers; their scores are all
  // masked.
  const int P0 = S - nq;  // position of the chunk's first query
  // this lane's query row rb + li: last token it may see, min(S - 1,
  // position); -1 for rows past the request's rows (all masked)
  const int rho_l = rb + li;
  const int lim = rho_l < rows_r ? min(S - 1, P0 + rho_l / G) : -1;
  const int n8 = a.counts[2 * r], n3 = a.counts[2 * r + 1];
  const int st3 = (n3 + 1) / 2, n_st = st3 + n8;
  uint8_t* const kbuf = smem + LY::KB0;
  uint8_t* const vbuf = smem + LY::VB0;
  uint8_t* const wbuf = smem + LY::WB0;
  float* const lbuf = reinterpret_cast<float*>(smem + LY::LB0);
  auto barrier = [&]() {
    wait_lgkm0();  // this wave's LDS reads and writes are done
    __builtin_amdgcn_s_barrier();
    __asm__ __volatile__("" ::: "memory");
  };
  struct TqW {
    half8 ha, la, hb, lb, z;  // weights of pages a and b (hi, lo); zero-term operand
  };
  // this pair's weight slot of stage j
  auto wslot = [&](int j) { return wbuf + ((j & 1) * NSW + sw) * LY::WPW; };

  // Stage j of the loops below is a TQ3 pair for j < st3, else an FP8 page.
  // Pass p (one barrier each, p = 0 .. n_st): the score waves issue stage
  // p's score product and finish stage p - 1 (scores, softmax, weights into
  // LDS) while the PV waves take stage p - 2 with the weights handed over in
  // pass p - 1.
  if (score_wave) {
    // ======================= score waves =======================
    // The score waves' instructions go first on the SIMD (their weights gate
    // the next pass); the PV waves fill the gaps.
    __builtin_amdgcn_s_setprio(2);
    float neg1 = -1.0f;  // kept in a register (see split2)
    __asm__ __volatile__("" : "+v"(neg1));
    const int rho_c = min(rho_l, rows_r - 1);  // a valid row to load for masked lanes
    const uint16_t* qrow_ptr = a.q + ((int64_t)(q0 + rho_c / G) * Hq + h * G + rho_c % G) * D;
    const uint8_t* stab = reinterpret_cast<const uint8_t*>(a.stages + (int64_t)r * mp);
    // The stage table reaches LDS in blocks of 64 stages (1 KiB), three
    // buffers, copied by every score wave itself with the counted copies of
    // the pages (so its own wait for a page makes the block visible to it);
    // block k + 1 is copied just before the first page of block k.
    const uint8_t* lsb = smem + LY::LS0;
    // stage j -> {lp_a, id_a, lp_b, id_b}; id_b < 0 marks an FP8 stage.  Two
    // readers (c = 0: the stage being scored, c = 1: the next stage to copy)
    // each keep one block in registers, lane l holding stage 64 k + l, and
    // take an entry with lane reads: one LDS read per 64 stages.
    int4 blk_v[2] = {make_int4(0, 0, 0, 0), make_int4(0, 0, 0, 0)};
    int blk_k[2] = {-1, -1};
    auto stage_at = [&](int j, int c) {
      j = __builtin_amdgcn_readfirstlane(j);
      if (j >= n_st) return make_int4(CMASK_LP, 0, CMASK_LP, 0);  // past the list: never used
      if ((j >> 6) != blk_k[c]) {
        blk_k[c] = j >> 6;
        blk_v[c] = *reinterpret_cast<const int4*>(lsb + ((j >> 6) % 3) * 1024 + lane * 16);
        wait_lgkm0();  // here, so that the lane reads after the join wait for nothing
      }
      const int l = j & 63;
      return make_int4(__builtin_amdgcn_readlane(blk_v[c].x, l), __builtin_amdgcn_readlane(blk_v[c].y, l),
                       __builtin_amdgcn_readlane(blk_v[c].z, l), __builtin_amdgcn_readlane(blk_v[c].w, l));
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
    // This wave's share of stage e's copies into ring slot `slot`: OPS_W
    // whole KiB (TQ3: KiB w OPS_W .. of the two pages laid end to end; FP8:
    // copies w OPS_W .. of the page's 2 NI), and for waves 0 and 1 one small
    // copy (TQ3: the 32-byte tail of page a resp. b; FP8: the two scales,
    // copied by both so that every stage costs each wave the same number of
    // copies).  Only the score waves copy.
    auto issue = [&](int4 e, int slot) {
      // wave-uniform by construction; said so for the scalar operands of the copies
      slot = __builtin_amdgcn_readfirstlane(slot);
      e.y = __builtin_amdgcn_readfirstlane(e.y);
      e.w = __builtin_amdgcn_readfirstlane(e.w);
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
    // Ring bookkeeping: stage s sits in slot s % CSLOTS; `issued` stages have
    // been copied so far.  The slot of a TQ3 pair s is free from pass s + 2
    // on (its keys are unpacked in pass s - 1, its values and key-norm
    // corrections read in pass s + 1), that of an FP8 page s from pass s + 3
    // on (read by the score waves in pass s, by the PV waves in pass
    // s + 2).  A wait for stage s lets the copies of the
    // stages after it stay in flight (every stage costs a wave the same
    // copies).
    const uint32_t lst_lds = ring_lds + LY::LS0;
    auto issue_list = [&](int k) {  // block k of the stage table -> buffer k % 3
      dma16<0>(16u * lane, stab + 1024 * k, lst_lds + (k % 3) * 1024);
    };
    const int n_blk = (n_st + 63) / 64;
    int issued = 0;
    issue_list(0);
    if (n_blk > 1) issue_list(1);
    wait_vmcnt<0>();
    int4 e_iss = stage_at(0, 1);  // the entries of stage `issued`
    auto refill = [&](int pass) {
      bool fresh = true;  // e_iss holds stage `issued`
      while (issued < n_st) {
        const int prev = issued - CSLOTS;
        if (prev >= 0 && (prev < st3 ? prev + 2 : prev + 3) > pass) break;
        if (!fresh) e_iss = stage_at(issued, 1);
        if ((issued & 63) == 0 && issued > 0 && (issued >> 6) + 1 < n_blk) issue_list((issued >> 6) + 1);
        issue(e_iss, issued % CSLOTS);
        ++issued;
        fresh = false;
      }
    };
    // entries of the next stage to copy, loaded at the end of a pass (the
    // barrier's wait covers their latency)
    auto prefetch_iss = [&]() { e_iss = stage_at(issued, 1); };
    auto wait_for = [&](int s) {
      const int later = max(0, min(issued - 1 - s, CSLOTS - 1));
#define MKV_CHUNK_WAIT(n)                                   \
  case n:                                                  \
    if (wid < 2) wait_vmcnt<(n) * (OPS_W + 1)>();          \
    else wait_vmcnt<(n) * OPS_W>();                        \
    break;
      switch (later) {
        MKV_CHUNK_WAIT(1)
        MKV_CHUNK_WAIT(2)
        MKV_CHUNK_WAIT(3)
        MKV_CHUNK_WAIT(4)
        MKV_CHUNK_WAIT(5)
        MKV_CHUNK_WAIT(6)
        MKV_CHUNK_WAIT(7)
        default: wait_vmcnt<0>(); break;
      }
#undef MKV_CHUNK_WAIT
    };
    static_assert(CSLOTS <= 8 && (CSLOTS - 1) * (OPS_W + 1) < 64,
                  "wait_for covers up to seven stages in flight");
    refill(-1);
    prefetch_iss();

    // ---- rotated query of this lane's row, q_rot = R q (R = d^-1/2 H
    // diag(sigma)), times the softmax scale log2(e)/sqrt(d) (scores come out
    // in base 2) and a power-of-two row scale qsc that puts the row's
    // largest entry in [128, 256), as three E4M3 terms t0 + t1 + t2 (each
    // the E4M3 rounding of what the earlier ones left; the remainder sits
    // below E4M3's subnormal step, about 2^-17 of the largest entry).  B
    // operand of the 32x32x64 fp8 MFMA: lane (li, lg) holds, for k-step s,
    // channels 64 s + 32 lg + j (j < 32) of row rb + li; the key operand
    // uses the same order.
    v8i qt[3][NK8];
    float qinv;
    {
      float x[NK8][32];
#pragma unroll
      for (int s = 0; s < NK8; ++s)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const uint4 raw = *reinterpret_cast<const uint4*>(qrow_ptr + 64 * s + 32 * lg + 8 * v);
          const uint16_t* hb = reinterpret_cast<const uint16_t*>(&raw);
          // the signs sit 4-byte aligned in the control buffer
          const uint32_t* sgw = reinterpret_cast<const uint32_t*>(P.sigma + 64 * s + 32 * lg + 8 * v);
          const uint2 sg2 = make_uint2(sgw[0], sgw[1]);
          const int8_t* sg = reinterpret_cast<const int8_t*>(&sg2);
#pragma unroll
          for (int j = 0; j < 8; ++j) x[s][8 * v + j] = bf16_to_f32(hb[j]) * (float)sg[j];
        }
      // Walsh-Hadamard butterflies over the channel bits: j (strides 1-16)
      // and s (strides 64 ..) inside the lane, lg (stride 32) across lanes
      // l ^ 32; the stages commute
#pragma unroll
      for (int st = 1; st < 32; st <<= 1)
#pragma unroll
        for (int s = 0; s < NK8; ++s)
#pragma unroll
          for (int j = 0; j < 32; ++j)
            if (!(j & st)) {
              const float x0 = x[s][j], x1 = x[s][j + st];
              x[s][j] = x0 + x1;
              x[s][j + st] = x0 - x1;
            }
#pragma unroll
      for (int st = 1; st < NK8; st <<= 1)
#pragma unroll
        for (int s = 0; s < NK8; ++s)
          if (!(s & st)) {
#pragma unroll
            for (int j = 0; j < 32; ++j) {
              const float x0 = x[s][j], x1 = x[s + st][j];
              x[s][j] = x0 + x1;
              x[s + st][j] = x0 - x1;
            }
          }
      const float sgn32 = (lane & 32) ? -1.0f : 1.0f;
      const float qscale = rsqrtf((float)D) * a.sm_log2;
      float amax = 0.0f;
#pragma unroll
      for (int s = 0; s < NK8; ++s)
#pragma unroll
        for (int j = 0; j < 32; ++j) {
          x[s][j] = fmaf(sgn32, x[s][j], lane_xor<32>(x[s][j], lane)) * qscale;
          amax = fmaxf(amax, fabsf(x[s][j]));
        }
      amax = fmaxf(amax, lane_xor<32>(amax, lane));
      int ex = 0;
      (void)frexpf(amax, &ex);  // amax in [2^(ex-1), 2^ex)
      const bool ok = rho_l < rows_r && amax > 0.0f;
      const float qsc = ok ? ldexpf(1.0f, 8 - ex) : 0.0f;
      qinv = ok ? ldexpf(1.0f, ex - 8) : 1.0f;  // (the terms of such a row are all zero)
#pragma unroll
      for (int s = 0; s < NK8; ++s)
#pragma unroll
        for (int w = 0; w < 8; ++w) {
          uint32_t b0 = 0, b1 = 0, b2 = 0;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            float v = x[s][4 * w + k] * qsc;
            const uint32_t e0 = f32_to_e4m3(v);
            v -= e4m3_to_f32(e0);
            const uint32_t e1 = f32_to_e4m3(v);
            v -= e4m3_to_f32(e1);
            const uint32_t e2 = f32_to_e4m3(v);
            b0 |= e0 << (8 * k);
            b1 |= e1 << (8 * k);
            b2 |= e2 << (8 * k);
          }
          qt[0][s][w] = (int)b0;
          qt[1][s][w] = (int)b1;
          qt[2][s][w] = (int)b2;
        }
    }

    float m_run = CM_INIT, l_run = 0.0f;  // this lane's row; l_run over its tokens
    const float smk = a.sm_log2;
    // Online softmax over the base-2 scores sc[16] of this lane's query row
    // (its 16 tokens of the tile; the other 16 sit in lane l ^ 32).  The
    // reference max moves (lazily, when a score passes it by 2^8): alpha is
    // the factor the PV accumulators still owe, exactly 1 where the
    // reference stayed (the PV wave skips the rescale when no row of its
    // tile moved).
    auto softmax = [&](float* sc, float& alpha) {
      float mx = sc[0];
#pragma unroll
      for (int k = 1; k < 16; ++k) mx = fmaxf(mx, sc[k]);
      mx = fmaxf(mx, lane_xor<32>(mx, lane));
      const float m_new = mx > m_run + 8.0f ? mx : m_run;
      alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      float lsum = 0.0f;
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        sc[k] = __builtin_amdgcn_exp2f(sc[k] - m_new);  // -inf -> 0
        lsum += sc[k];
      }
      l_run = fmaf(l_run, alpha, lsum);
    };
    // weights p[0..7] as an fp16 hi + lo pair (one token can carry most of
    // a row's mass, and its weight, taken against a lagging reference max,
    // is then not a power of two; a single fp16 rounding of it moves the
    // output by up to 2^-12 of that token's value)
    auto split8 = [&](const float* p, half8& hi, half8& lo) {
      uint32_t hh4[4], ll4[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) split2(p[2 * k], p[2 * k + 1], neg1, hh4[k], ll4[k]);
      hi = h8u(hh4[0], hh4[1], hh4[2], hh4[3]);
      lo = h8u(ll4[0], ll4[1], ll4[2], ll4[3]);
    };
    // hand the weights of stage j (and the rescale the PV accumulators owe
    // before them) to the PV wave of this pair
    auto put_weights = [&](int j, const TqW& w, float alpha) {
      uint8_t* ws = wslot(j);
      *reinterpret_cast<half8*>(ws + 0 * 1024 + 16 * lane) = w.ha;
      *reinterpret_cast<half8*>(ws + 1 * 1024 + 16 * lane) = w.la;
      *reinterpret_cast<half8*>(ws + 2 * 1024 + 16 * lane) = w.hb;
      *reinterpret_cast<half8*>(ws + 3 * 1024 + 16 * lane) = w.lb;
      *reinterpret_cast<half8*>(ws + 4 * 1024 + 16 * lane) = w.z;
      reinterpret_cast<float*>(ws + LY::WF_ALPHA)[lane] = alpha;
    };

    // ---- unpacking of a TQ3 pair (the 256 threads of the score waves, from
    // the raw stage at rs):
    //  keys: threads 0-127, one code chunk (token, channel quarter) each:
    //    codes -> E4M3 codebook bytes (one v_perm per 4 codes) in the score
    //    product's A layout, kb[k-step][lane (32 lg + token of the pair)][32];
    //  values: threads 128-255, one code chunk (16 channels, 4 tokens) each:
    //    code bytes in the PV product's A layout, vb[page][block][lane][8]
    //    (lane 32 hk + rr: channel CL (rr % 16) + 2 mb + rr / 16, tokens 4
    //    hk .. 4 hk + 3 then 8 + 4 hk .. 8 + 4 hk + 3, the order in which
    //    the score tile hands each lane its weights);
    //  per (page, block, row rr): the V scale split as (hi, lo) fp16 (hi
    //    keeps 8 significant bits, so code x hi is exact in fp16) and the V
    //    zero.
    // The keys of a pair are unpacked one pass before its score product, its
    // values one pass after it (with its scores).
    auto unpack_k = [&](const uint8_t* rs, uint8_t* kb) {  // threads 0-127
      const int p = tid >> 6, tok = tid & 15, g = (tid >> 4) & 3;
      uint32_t dw[NDW];
      read_chunk<NDW>(dw, rs + p * R3, 16 * g + tok);
#pragma unroll
      for (int q8 = 0; q8 < CL / 8; ++q8) {
        uint32_t o[8];
#pragma unroll
        for (int w = 0; w < 8; ++w) o[w] = __builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(dw, 8 * q8 + w));
        const int c0 = g * QQ + 32 * q8;  // first channel of these 32 bytes
        uint4* dst = reinterpret_cast<uint4*>(kb + ((c0 / 64) * 64 + 32 * ((c0 / 32) & 1) + 16 * p + tok) * 32);
        dst[0] = make_uint4(o[0], o[1], o[2], o[3]);
        dst[1] = make_uint4(o[4], o[5], o[6], o[7]);
      }
    };
    auto unpack_v = [&](const uint8_t* rs, uint8_t* vb) {  // threads 128-255
      const int u = tid - 128;
      const int p = u >> 6, r0 = u & 15, g = (u >> 4) & 3;
      uint32_t dw[NDW];
      read_chunk<NDW>(dw, rs + p * R3 + 6 * D, 16 * g + r0);
      uint8_t* base = vb + (p * NMB * 64 + 32 * (g & 1) + r0) * 8 + 4 * (g >> 1);
#pragma unroll
      for (int q = 0; q < CL; ++q)
        *reinterpret_cast<uint32_t*>(base + ((q >> 1) * 64 + 16 * (q & 1)) * 8) = quad_sel<NDW>(dw, q);
    };
    auto unpack_side = [&](const uint8_t* rs, uint8_t* vb) {
      if (NMB * 32 >= 64 * NSW || tid < NMB * 32) {  // whole waves (every score wave at d = 256)
        const int mb = tid >> 5, rr = tid & 31, ch = CL * (rr & 15) + 2 * mb + (rr >> 4);
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const half2v s1 = bcast(*reinterpret_cast<const _Float16*>(rs + p * R3 + 12 * D + 32 + 2 * ch));
          const half2v sh = hi8x2(s1);
          const half2v sp = {sh[0], s1[0] - sh[0]};  // exact split
          *reinterpret_cast<half2v*>(vb + LY::VX + ((p * NMB + mb) * 32 + rr) * 4) = sp;
          *reinterpret_cast<_Float16*>(vb + LY::VX + LY::SX + ((p * NMB + mb) * 32 + rr) * 2) =
              *reinterpret_cast<const _Float16*>(rs + p * R3 + 14 * D + 32 + 2 * ch);
        }
      }
    };

    // S^T = K Q^T of the pair whose keys are unpacked in kb: M = the pair's
    // 32 tokens (page a, then page b), N = the wave's 32 rows, one chain of
    // three MFMAs (one per query term) per k-step
    auto tq3_qk = [&](const uint8_t* kb, float16v& st, auto rev) {
      st = float16v{};
#pragma unroll
      for (int s_ = 0; s_ < NK8; ++s_) {
        const int s = decltype(rev)::value ? NK8 - 1 - s_ : s_;
        const v8i A = *reinterpret_cast<const v8i*>(kb + (s * 64 + lane) * 32);
#pragma unroll
        for (int t = 0; t < 3; ++t)
          st = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A, qt[t][s], st, 0, 0, 0, 0, 0, 0);
      }
    };
    // Scores and weights of the TQ3 pair e from its score product st and the
    // key-norm corrections gamma in its raw stage rs.  Lane (li, lg)
    // receives tokens 4 lg .. 4 lg + 3 and 8 + 4 lg .. of each page, which
    // are exactly the k-slots of its weight operand.  `masked`: some token
    // of the pair lies past the chunk's first query.
    auto tq3_scores = [&](const uint8_t* rs, const float16v& st, const int4& e, TqW& w, float& alpha,
                          auto masked) {
      // element e: token 8 (e / 4) + 4 lg + e % 4 of the pair (page a below 16)
      uint2 gw[4];
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4)
        gw[e4] = *reinterpret_cast<const uint2*>(rs + (e4 >> 1) * R3 + 12 * D + 16 * (e4 & 1) + 8 * lg);
      float sc[16];
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int t0 = (e4 < 2 ? e.x : e.z) * PAGE + 8 * (e4 & 1) + 4 * lg;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float v = st[4 * e4 + u] * qinv * (float)reinterpret_cast<const _Float16*>(&gw[e4])[u];
          if constexpr (decltype(masked)::value)
            sc[4 * e4 + u] = t0 + u <= lim ? v : -INFINITY;
          else
            sc[4 * e4 + u] = v;
        }
      }
      softmax(sc, alpha);
      split8(sc, w.ha, w.la);
      split8(sc + 8, w.hb, w.lb);
      const float ra_ = ((sc[0] + sc[1]) + (sc[2] + sc[3])) + ((sc[4] + sc[5]) + (sc[6] + sc[7]));
      const float rb_ = ((sc[8] + sc[9]) + (sc[10] + sc[11])) + ((sc[12] + sc[13]) + (sc[14] + sc[15]));
      uint32_t zh, zl;
      split2(ra_, rb_, neg1, zh, zl);
      w.z = h8u(zh, zl, 0u, 0u);  // (R_a, R_b) hi, then lo
    };
    // a pair whose pages both end before the chunk's first query needs no mask
    auto unmasked = [&](const int4& e) { return (max(e.x, e.z) + 1) * PAGE <= P0 + 1; };

    // ---- passes over the TQ3 pairs.  Pass p (after barrier p + 1) issues
    // the score product of pair p (keys unpacked in pass p - 1) and, while
    // the matrix unit works on it, finishes pair p - 1 (scores from the
    // product issued in pass p - 1, softmax, weights into LDS) and unpacks
    // the keys of pair p + 1 and the values of pair p - 1; the PV waves take
    // pair p - 2.  One straight block per wave kind; scheduling fences place
    // the twelve MFMAs between segments of the VALU and LDS work (left to
    // itself the compiler issued all twelve first).
    float16v st_prev = {};                // score product of stage p - 1
    int4 e_prev = make_int4(0, 0, 0, 0);  // entries of stage p - 1
    auto tq3_pass = [&](int p, float16v& st, auto masked, auto key_kind) {
      constexpr bool KK = decltype(key_kind)::value;  // this wave unpacks keys (else values)
      const uint8_t* kb = kbuf + (p & 1) * LY::KB;
      uint8_t* kb_next = kbuf + ((p + 1) & 1) * LY::KB;
      uint8_t* vb_prev = vbuf + ((p + 1) & 1) * LY::VB;  // buffer (p - 1) & 1
      const uint8_t* rs_prev = smem + ((p + CSLOTS - 1) % CSLOTS) * STAGE;
      const uint8_t* rs_next = smem + ((p + 1) % CSLOTS) * STAGE;
      // k-step of the i-th step of the product (the two kinds take the
      // k-steps in opposite orders, which keeps the compiler from merging
      // the two blocks' products)
      auto kstep = [&](int i) { return KK ? i : NK8 - 1 - i; };
      auto ld_a = [&](int i) { return *reinterpret_cast<const v8i*>(kb + (kstep(i) * 64 + lane) * 32); };
      v8i A[2];
      A[0] = ld_a(0);
      A[1] = ld_a(1);
      uint2 gw[4];
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4)
        gw[e4] = *reinterpret_cast<const uint2*>(rs_prev + (e4 >> 1) * R3 + 12 * D + 16 * (e4 & 1) + 8 * lg);
      st = float16v{};
      // MFMA m of the product (k-step m / 3, query term m % 3); the operand of
      // the k-step after next is read once the last MFMA of a k-step is issued
      auto mf = [&](int m) {
        const int i = m / 3, t = m % 3;
        if (i >= NK8) return;  // d = 128: six MFMAs
        st = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A[i & 1], qt[t][kstep(i)], st, 0, 0, 0, 0, 0,
                                                             0);
        if (t == 2 && i + 2 < NK8) A[i & 1] = ld_a(i + 2);
        __builtin_amdgcn_sched_barrier(0);
      };
      // pair p - 1: scores, softmax and weights, between the MFMAs
      float sc[16];
      auto scores = [&](int e4) {
        const int t0 = (e4 < 2 ? e_prev.x : e_prev.z) * PAGE + 8 * (e4 & 1) + 4 * lg;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          // st * gamma as one mixed-precision FMA; the power-of-two row
          // factor qinv enters with the max and the exponent (exact)
          const float v = __builtin_fmaf((float)reinterpret_cast<const _Float16*>(&gw[e4])[u], st_prev[4 * e4 + u], 0.0f);
          if constexpr (decltype(masked)::value)
            sc[4 * e4 + u] = t0 + u <= lim ? v : -INFINITY;
          else
            sc[4 * e4 + u] = v;
        }
      };
      float m_new, alpha, lsum = 0.0f;
      auto ex = [&](int k0, int k1) {
#pragma unroll
        for (int k = k0; k < k1; ++k) {
          sc[k] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[k], qinv, -m_new));  // -inf -> 0
          lsum += sc[k];
        }
      };
      TqW w;
      mf(0);
      scores(0);
      scores(1);
      __builtin_amdgcn_sched_barrier(0);
      mf(1);
      scores(2);
      scores(3);
      __builtin_amdgcn_sched_barrier(0);
      mf(2);
      {
        float mx = sc[0];
#pragma unroll
        for (int k = 1; k < 16; ++k) mx = fmaxf(mx, sc[k]);
        mx = fmaxf(mx, lane_xor<32>(mx, lane)) * qinv;
        m_new = mx > m_run + 8.0f ? mx : m_run;
        alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
      }
      __builtin_amdgcn_sched_barrier(0);
      mf(3);
      ex(0, 6);
      __builtin_amdgcn_sched_barrier(0);
      mf(4);
      ex(6, 11);
      __builtin_amdgcn_sched_barrier(0);
      mf(5);
      ex(11, 16);
      l_run = fmaf(l_run, alpha, lsum);
      __builtin_amdgcn_sched_barrier(0);
      mf(6);
      split8(sc, w.ha, w.la);
      __builtin_amdgcn_sched_barrier(0);
      mf(7);
      split8(sc + 8, w.hb, w.lb);
      __builtin_amdgcn_sched_barrier(0);
      mf(8);
      {
        const float ra_ = ((sc[0] + sc[1]) + (sc[2] + sc[3])) + ((sc[4] + sc[5]) + (sc[6] + sc[7]));
        const float rb_ = ((sc[8] + sc[9]) + (sc[10] + sc[11])) + ((sc[12] + sc[13]) + (sc[14] + sc[15]));
        uint32_t zh, zl;
        split2(ra_, rb_, neg1, zh, zl);
        w.z = h8u(zh, zl, 0u, 0u);  // (R_a, R_b) hi, then lo
      }
      put_weights(p - 1, w, alpha);
      __builtin_amdgcn_sched_barrier(0);
      // then this wave's share of the unpacking: keys of pair p + 1 or
      // values of pair p - 1, and the values' side data of pair p - 1
      mf(9);
      if constexpr (KK)
        unpack_k(rs_next, kb_next);
      else
        unpack_v(rs_prev, vb_prev);
      __builtin_amdgcn_sched_barrier(0);
      mf(10);
      unpack_side(rs_prev, vb_prev);
      __builtin_amdgcn_sched_barrier(0);
      mf(11);
    };
    if (st3 > 0) wait_for(0);
    barrier();
    if (st3 > 0 && wid < 2) unpack_k(smem, kbuf);
    for (int p = 0; p < st3; ++p) {
      if (p + 1 < st3) wait_for(p + 1);
      barrier();  // keys of pair p unpacked; raw pair p + 1 landed
      // (in the last pass the key unpacking reads a slot that holds no pair
      // and writes a buffer nobody reads any more)
      float16v st;
      if (p == 0) {
        if (wid < 2) {
          tq3_qk(kbuf, st, std::false_type{});
          unpack_k(smem + (1 % CSLOTS) * STAGE, kbuf + LY::KB);
        } else {
          tq3_qk(kbuf, st, std::true_type{});
        }
      } else if (unmasked(e_prev)) {
        if (wid < 2)
          tq3_pass(p, st, std::false_type{}, std::true_type{});
        else
          tq3_pass(p, st, std::false_type{}, std::false_type{});
      } else {
        if (wid < 2)
          tq3_pass(p, st, std::true_type{}, std::true_type{});
        else
          tq3_pass(p, st, std::true_type{}, std::false_type{});
      }
      refill(p);
      st_prev = st;
      e_prev = stage_at(p, 0);
      prefetch_iss();
    }
    // ---- passes over the FP8 pages: pass p scores page p with plain
    // queries as fp16 (bf16 -> fp16 is exact for the query range) against
    // its FP8 keys, straight from the ring, and finishes the weights of
    // stage p - 1 (for p = st3 the last TQ3 pair, whose values it also
    // unpacks); the last pass only finishes.  Lane (li, lg) holds, for
    // k-step s, channels (D/2) lg + 8 s + b (b < 8) of its row.
    {
      half8 qop[NKS];
      if (st3 < n_st) {
        const uint16_t* qrow = qrow_ptr + (D / 2) * lg;
#pragma unroll
        for (int s = 0; s < NKS; ++s) {
          const uint4 raw = *reinterpret_cast<const uint4*>(qrow + 8 * s);
          const uint16_t* hb = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
          for (int j = 0; j < 8; ++j) qop[s][j] = (_Float16)bf16_to_f32(hb[j]);
        }
      }
      float2 ks_prev = make_float2(0.0f, 0.0f);  // key and value scales of FP8 stage p - 1
      for (int p = st3; p <= n_st; ++p) {
        if (p < n_st) wait_for(p);
        barrier();  // page p visible
        refill(p);
        float16v st = {};
        float2 ksv = make_float2(0.0f, 0.0f);
        if (p < n_st) {
          const uint8_t* ra = smem + (p % CSLOTS) * STAGE;
          // block-permuted page (see dma_fp8_page): 16-byte block 64 w + 16
          // Q + t holds bytes 16 w .. of token t's channel quarter Q (K);
          // score rows 0-15 are the page's tokens, 16-31 zero
          const uint2* pk = reinterpret_cast<const uint2*>(ra);
          ksv = *reinterpret_cast<const float2*>(ra + R8);
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
        }
        if (p > 0) {
          TqW w;
          float alpha;
          if (p == st3) {  // the last TQ3 pair
            const uint8_t* rs_prev = smem + ((p + CSLOTS - 1) % CSLOTS) * STAGE;
            uint8_t* vb_prev = vbuf + ((p + 1) & 1) * LY::VB;
            if (unmasked(e_prev))
              tq3_scores(rs_prev, st_prev, e_prev, w, alpha, std::false_type{});
            else
              tq3_scores(rs_prev, st_prev, e_prev, w, alpha, std::true_type{});
            if (wid >= 2) unpack_v(rs_prev, vb_prev);
            unpack_side(rs_prev, vb_prev);
          } else {
            float sc[16];
            const float kk = ks_prev.x * smk;
#pragma unroll
            for (int e4 = 0; e4 < 4; ++e4) {
              const int t0 = e_prev.x * PAGE + 8 * (e4 & 1) + 4 * lg;
#pragma unroll
              for (int u = 0; u < 4; ++u)
                sc[4 * e4 + u] = (e4 < 2 && t0 + u <= lim) ? st_prev[4 * e4 + u] * kk : -INFINITY;
            }
            softmax(sc, alpha);
            // the page's V scale folded into the weights
            float pw[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) pw[k] = sc[k] * ks_prev.y;
            split8(pw, w.ha, w.la);
            w.hb = w.la;
            w.lb = w.la;
            w.z = w.la;
          }
          put_weights(p - 1, w, alpha);
        }
        st_prev = st;
        ks_prev = ksv;
        e_prev = stage_at(p, 0);
        prefetch_iss();
      }
    }
    barrier();  // the PV waves' last pass
    const float L = l_run + lane_xor<32>(l_run, lane);
    if (lg == 0) lbuf[sw * 32 + li] = L;
    barrier();
  } else {
    // ========================= PV waves =========================
    // PV wave v owns the 32-channel blocks mb = NBW v .. NBW v + NBW - 1 of
    // the output for all 128 rows of the workgroup (the rows of every score
    // wave g), so each value operand is built once per workgroup.
    // Accumulators: O^T tile (32 channels x the 32 rows of score wave g) per
    // (block, g).  Lane (li, lg), element e holds row 32 g + li and tile row
    // rr = 8 (e / 4) + 4 lg + e % 4, which is channel CL (rr % 16) + 2 mb +
    // rr / 16 (the value unpacking lays its operands out for this order).
    constexpr int NBW = NMB / NSW;
    static_assert(NMB % NSW == 0 && NBW <= 2, "whole blocks per PV wave");
    const int pv = wid - NSW;
    float16v acc[NBW][NSW];
#pragma unroll
    for (int b = 0; b < NBW; ++b)
#pragma unroll
      for (int g = 0; g < NSW; ++g) acc[b][g] = float16v{};
    // weights of stage j from score wave g
    auto wsl = [&](int j, int g) { return wbuf + ((j & 1) * NSW + g) * LY::WPW; };
    // the rescales the weights of stage j carry, one per score wave (skipped
    // when every factor is 1: no reference max moved)
    auto rescale = [&](int j) {
      float al[NSW];
      bool any = false;
#pragma unroll
      for (int g = 0; g < NSW; ++g) {
        al[g] = reinterpret_cast<const float*>(wsl(j, g) + LY::WF_ALPHA)[lane];
        any |= al[g] != 1.0f;
      }
      if (__any(any)) {
#pragma unroll
        for (int b = 0; b < NBW; ++b)
#pragma unroll
          for (int g = 0; g < NSW; ++g) acc[b][g] *= al[g];  // column = this lane's row
      }
    };
    auto ld_w = [&](int j, int g, TqW& w) {
      const uint8_t* ws = wsl(j, g);
      w.ha = *reinterpret_cast<const half8*>(ws + 0 * 1024 + 16 * lane);
      w.la = *reinterpret_cast<const half8*>(ws + 1 * 1024 + 16 * lane);
      w.hb = *reinterpret_cast<const half8*>(ws + 2 * 1024 + 16 * lane);
      w.lb = *reinterpret_cast<const half8*>(ws + 3 * 1024 + 16 * lane);
      w.z = *reinterpret_cast<const half8*>(ws + 4 * 1024 + 16 * lane);
    };
    // O^T += V^T P^T for the TQ3 pair of stage j (values unpacked in vb),
    // with exact V operands: v = zero + scale * code is split as scale_hi *
    // code + scale_lo * code + zero.  The products that reach fp32 accuracy:
    // (hi + lo weights) x scale_hi term, hi weights x scale_lo term (lo x
    // scale_lo sits below 2^-19 of the value), and the zero term as zero_a
    // (sum of weights over page a) + zero_b (same for b), whose sums the
    // MFMA completes across the two lane groups.
    auto tq3_pv = [&](int j) {
      const uint8_t* vb = vbuf + (j & 1) * LY::VB;
      const _Float16* zx = reinterpret_cast<const _Float16*>(vb + LY::VX + LY::SX);
      struct Ops {
        half8 A1[2], A2[2], Az;
      };
      // the weights of score wave g + 1 are read while the products of g run
      TqW wb[2];
      ld_w(j, 0, wb[0]);
      Ops op[NBW];
#pragma unroll
      for (int b = 0; b < NBW; ++b) {
        const int mb = NBW * pv + b;
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const uint2 cw = *reinterpret_cast<const uint2*>(vb + ((p * NMB + mb) * 64 + lane) * 8);
          const half2v s2 = *reinterpret_cast<const half2v*>(vb + LY::VX + ((p * NMB + mb) * 32 + li) * 4);
          const half2v sh = bcast(s2[0]), sl = bcast(s2[1]);
          const half2v c01 = cvt_code<false>(cw.x), c23 = cvt_code<true>(cw.x);
          const half2v c45 = cvt_code<false>(cw.y), c67 = cvt_code<true>(cw.y);
          op[b].A1[p] = h8(c01 * sh, c23 * sh, c45 * sh, c67 * sh);
          op[b].A2[p] = h8(c01 * sl, c23 * sl, c45 * sl, c67 * sl);
        }
        const _Float16 za = zx[mb * 32 + li], zb = zx[(NMB + mb) * 32 + li];
        op[b].Az = half8{za, zb, za, zb, (_Float16)0.0f, (_Float16)0.0f, (_Float16)0.0f, (_Float16)0.0f};
      }
      rescale(j);
#pragma unroll
      for (int g = 0; g < NSW; ++g) {
        if (g + 1 < NSW) ld_w(j, g + 1, wb[(g + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
        const TqW& w = wb[g & 1];
        // the blocks' chains interleaved
#define MKV_PV(A, B)                                                                     \
  _Pragma("unroll") for (int b = 0; b < NBW; ++b) acc[b][g] =                            \
      __builtin_amdgcn_mfma_f32_32x32x16_f16(op[b].A, w.B, acc[b][g], 0, 0, 0);
        MKV_PV(A1[0], ha)
        MKV_PV(A2[0], ha)
        MKV_PV(A1[0], la)
        MKV_PV(A1[1], hb)
        MKV_PV(A2[1], hb)
        MKV_PV(A1[1], lb)
        MKV_PV(Az, z)
#undef MKV_PV
      }
    };
    // O^T += V^T P^T for the FP8 page of stage j in ring slot ra (weights hi +
    // lo, the page's V scale already folded in): lane-chunks (rrow, lg) and
    // (rrow, lg + 2) of V, dword m = tokens 4 g' .. 4 g' + 3 of channel CL
    // rrow + m
    auto fp8_pv = [&](const uint8_t* ra, int j) {
      const int rrow = li & 15, hh = li >> 4;
      const uint2* pvp = reinterpret_cast<const uint2*>(ra + PAGE * D);
      half8 Av[NBW];
#pragma unroll
      for (int b = 0; b < NBW; ++b) {
        const int mb = NBW * pv + b;
        const int blk = 64 * (mb / 2);
        const uint2 v0 = pvp[2 * (blk + 16 * lg + rrow) + (mb & 1)];
        const uint2 v2 = pvp[2 * (blk + 16 * (lg + 2) + rrow) + (mb & 1)];
        const uint32_t w0 = hh ? v0.y : v0.x, w2 = hh ? v2.y : v2.x;
        Av[b] = h8(cvt_lo(w0), cvt_hi(w0), cvt_lo(w2), cvt_hi(w2));
      }
      rescale(j);
#pragma unroll
      for (int g = 0; g < NSW; ++g) {
        const uint8_t* ws = wsl(j, g);
        const half8 ha = *reinterpret_cast<const half8*>(ws + 0 * 1024 + 16 * lane);
        const half8 la = *reinterpret_cast<const half8*>(ws + 1 * 1024 + 16 * lane);
#pragma unroll
        for (int b = 0; b < NBW; ++b) acc[b][g] = __builtin_amdgcn_mfma_f32_32x32x16_f16(Av[b], ha, acc[b][g], 0, 0, 0);
#pragma unroll
        for (int b = 0; b < NBW; ++b) acc[b][g] = __builtin_amdgcn_mfma_f32_32x32x16_f16(Av[b], la, acc[b][g], 0, 0, 0);
      }
    };
    barrier();  // the score waves' first key unpacking
    barrier();  // pass 0: the score product of stage 0
    barrier();  // pass 1: the weights of stage 0
    for (int j = 0; j < st3; ++j) {  // pass j + 2
      barrier();
      tq3_pv(j);
    }
    for (int j = st3; j < n_st; ++j) {
      barrier();
      fp8_pv(smem + (j % CSLOTS) * STAGE, j);
    }
    barrier();  // the rows' denominators
    // ---- normalize and store: tile row rr = 8 kk + 4 lg + u (kk, u: the
    // lane's elements 4 kk + u and 8 + 4 kk + u) is chunk row rr % 16 = rr
    // for both halves hh = 0, 1 of every block, so this wave's channels
    // CL rr + 2 NBW pv .. + 2 NBW - 1 are contiguous: channel CL rr + 2 mb +
    // hh <- acc[mb - NBW pv][g][4 kk + 8 hh + u]
#pragma unroll
    for (int g = 0; g < NSW; ++g) {
      const int rho = xb * (NSW * 32) + g * 32 + li;
      if (rho < rows_r) {
        const float L = lbuf[g * 32 + li];
        const float inv = L > 0.0f ? 1.0f / L : 0.0f;
        float* o = a.out + ((int64_t)(q0 + rho / G) * Hq + h * G + rho % G) * D + 2 * NBW * pv;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int rr = 8 * kk + 4 * lg + u;
            if constexpr (NBW == 2)
              *reinterpret_cast<float4*>(o + CL * rr) =
                  make_float4(acc[0][g][4 * kk + u] * inv, acc[0][g][4 * kk + 8 + u] * inv,
                              acc[1][g][4 * kk + u] * inv, acc[1][g][4 * kk + 8 + u] * inv);
            else
              *reinterpret_cast<float2*>(o + CL * rr) =
                  make_float2(acc[0][g][4 * kk + u] * inv, acc[0][g][4 * kk + 8 + u] * inv);
          }
      }
    }
  }
}

// Row blocks of a chunk call: request r gets ceil(n_r G / 128) blocks of 128
// rows (at least one, and one for a request whose query range is invalid, so
// that its error is reported); rbo[r] = the blocks before request r,
// rbo[n_req] = all of them.  Query ranges that do not overlap need at most
// `grid` blocks (the launch's width); ranges that overlap and need more set
// the range error bit and rbo[n_req] = 0: the call writes nothing.  One
// workgroup.
__global__ __launch_bounds__(256) void chunk_rows_kernel(int n_req, const int32_t* cu_q, int n_q_total,
                                                         int group, int grid, int32_t* rbo,
                                                         int32_t* err) {
  __shared__ int part[256];
  const int t = threadIdx.x;
  const int per = (n_req + 255) / 256;
  const int r0 = min(n_req, t * per), r1 = min(n_req, r0 + per);
  auto blocks = [&](int r) {
    const int q0 = cu_q[r], q1 = cu_q[r + 1];
    const bool ok = q0 >= 0 && q1 >= q0 && q1 <= n_q_total;
    return ok ? max(1, (int)(((int64_t)(q1 - q0) * group + NSW * 32 - 1) / (NSW * 32))) : 1;
  };
  int sum = 0;
  for (int r = r0; r < r1; ++r) sum += blocks(r);
  part[t] = sum;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {  // inclusive scan of the thread sums
    const int v = t >= o ? part[t - o] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int base = part[t] - sum;
  for (int r = r0; r < r1; ++r) {
    rbo[r] = base;
    base += blocks(r);
  }
  if (t == 255) {
    const bool fits = part[255] <= grid;
    rbo[n_req] = fits ? part[255] : 0;
    if (!fits) atomicOr(err, (int)MKV_DEVERR_RANGE);
  }
}

// Grid (row block over all requests, KV head): workgroup x takes global row
// block x and finds its request in the row-block table (workgroups past the
// last block return at once).
template <int D>
__global__ __launch_bounds__(64 * CW, 1) void chunk_kernel(ChunkArgs a) {
  extern __shared__ __align__(16) uint8_t smem[];
  const int gb = blockIdx.x;
  if (gb >= a.rbo[a.n_req]) return;
  int lo = 0, hi = a.n_req - 1;  // the last request whose first block is <= gb
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.rbo[mid] <= gb)
      lo = mid;
    else
      hi = mid - 1;
  }
  chunk_block<D>(a, lo, blockIdx.y, gb - a.rbo[lo], smem);
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
  const ChunkWs wl = chunk_ws(n_req, max_pages);
  int32_t* list8 = reinterpret_cast<int32_t*>(w + wl.list8);
  int32_t* list3 = reinterpret_cast<int32_t*>(w + wl.list3);
  int32_t* counts = reinterpret_cast<int32_t*>(w + wl.counts);
  int4* stages = reinterpret_cast<int4*>(w + wl.stages);
  int32_t* rbo = reinterpret_cast<int32_t*>(w + wl.rbo);
  a.list8 = list8;
  a.list3 = list3;
  a.counts = counts;
  a.stages = stages;
  a.rbo = rbo;
  a.sm_log2 = 1.4426950408889634f / sqrtf((float)P.d);
  hipError_t e = launch_partition(n_req, bt, tags, max_pages, seq_lens, list8, list3, counts,
                                  P.ctrl + CTRL_ERR, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(chunk_stages_kernel, dim3((max_pages + 255) / 256, n_req), dim3(256), 0, s,
                     max_pages, P.n_tq3, P.n_fp8, list8, list3, counts, stages, P.ctrl + CTRL_ERR);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // row blocks of all requests: at most ceil(n_q_total G / 128) + n_req when
  // the query ranges do not overlap
  const int64_t rows = (int64_t)n_q_total * P.group;
  const int wg_rows = NSW * 32;
  const int blocks = (int)((rows + wg_rows - 1) / wg_rows) + n_req;
  hipLaunchKernelGGL(chunk_rows_kernel, dim3(1), dim3(256), 0, s, n_req, cu_q, n_q_total, P.group, blocks,
                     rbo, P.ctrl + CTRL_ERR);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds = P.d == 256 ? (size_t)ChunkLds<256>::TOTAL : (size_t)ChunkLds<128>::TOTAL;
  const void* kern = P.d == 256 ? (const void*)chunk_kernel<256> : (const void*)chunk_kernel<128>;
  e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 grid(blocks, P.n_kv_heads);
  void* args[] = {&a};
  e = hipLaunchKernel(kern, grid, dim3(64 * CW), args, lds, s);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace mkv
