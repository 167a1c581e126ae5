// Mixed-format paged decode attention (Sec. 3.3, Eq. softmax-merge; Sec. 4.1
// direct fused decode) for gfx950.
//
// One launch per layer.  Grid (chunk, KV head, request); one workgroup per CU:
// 8 wave64s with one ring slot each when a KV head's query group has at most
// 8 heads (two pages share a score tile), else 8 waves with two slots.  Chunks
// are ranges of logical pages of equal cost: a page wholly outside the Recent
// window costs 2 units, a Recent (FP8) page 5 (its scattered 16-byte copies
// make it cost the scan about 2.5 times a TQ3 page, measured); the unit count
// per chunk is chosen so that the launch is about one workgroup per CU.  Each
// workgroup
//  1. loads its chunk's tags and page ids and the request's length together,
//     and meanwhile builds the query operands in LDS: the plain query as fp16
//     (FP8 pages) and the rotated query q_rot = R q (exact algebra: k_hat =
//     gamma R^T mu_c, so keys are never de-rotated) times the softmax scale,
//     as three E4M3 terms under a power-of-two head scale (TQ3 pages), the
//     Hadamard transform done with DPP / permlane butterflies;
//  2. splits its pages by format into compact lists in logical order (Sec.
//     4.1 per-format lists, per chunk, with wave ballots) and turns them into
//     stages of equal size: a pair of TQ3 pages or one FP8 page; waves claim
//     stages from an LDS counter and raise their priority as they progress;
//  3. each wave streams its stages through its ring slot, fed by direct HBM ->
//     LDS copies (global_load_lds_dwordx4): QK^T of TQ3 pages on
//     v_mfma_scale_f32_16x16x128_f8f6f4 (3-bit codes -> E4M3 codebook bytes by
//     one v_perm per 4 codes, against the three query terms; M = 16 tokens, N
//     = 16 columns = the group's heads against page a and page b), of FP8
//     pages on v_mfma_f32_16x16x32_f16; online softmax in base 2 with a lazy
//     reference max; PV on the f16 MFMA with block-diagonal page rows, the
//     weights as an fp16 hi + lo pair, TQ3 value codes as exact integers and
//     the per-channel scale and zero applied in fp32 to the MFMA output;
//  4. merges its waves' rows in LDS into one (m_j, l_j, O_j) partial per chunk.
// A second kernel merges all partials of a request and query head (Eq.
// softmax-merge).  The workspace holds O(chunks x heads x d) partials, never
// anything the size of the cache.  Instances: APP fuses the decode-step append
// of one token per request into the launch; SCORE also records every page's
// local softmax mass for the attention-score collector.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>
#include <type_traits>

#include "mkv_append.h"
#include "mkv_attn.h"
#include "mkv_internal.h"
#include "../../include/minima_kv.h"

namespace mkv {

// Workgroup shape per instance: with the paired score layout (G <= 8) 8
// waves, each with a one-stage ring slot (a stage is moved into registers as
// soon as it lands and the slot refilled at once); otherwise 8 waves with two
// slots.  One workgroup per CU either way.  Eight one-slot waves beat twelve
// on the long pair (29.7 against 31.0 us per scan): the stage loop is not
// issue-bound with two waves per SIMD, and fewer copies in flight per CU let
// the memory system deliver more (a further L2 prefetch of later stages, or
// four waves, were slower still).
#ifndef MKV_PAIR_NW
#define MKV_PAIR_NW 8
#define MKV_PAIR_SLOTS 1
#endif
template <bool PAIR> struct DecodeCfg {
  static constexpr int NW = PAIR ? MKV_PAIR_NW : 8;  // waves per workgroup
  static constexpr int SLOTS = PAIR ? MKV_PAIR_SLOTS : 2;  // ring slots per wave
  static constexpr int NT = 64 * NW;
};
constexpr int NW_MAX = MKV_PAIR_NW > 8 ? MKV_PAIR_NW : 8;
// Wave priority by progress through a stage (claimed -> 1, scores done -> 2,
// weights done -> 3): among the waves of a SIMD the one furthest into its
// stage issues first, so stages finish roughly in the order they were claimed.
#define STAGE_PRIO(p) __builtin_amdgcn_s_setprio(p)
#define NCH_OF(pair) ((pair) ? 8 : 16)
constexpr int MAX_CHUNK_PAGES = 256;   // pages a chunk may span
// cost of a page in chunk units: wholly outside the Recent window / Recent
constexpr int COST_OLD = 2, COST_REC = 5;
constexpr int COST_MIN = COST_OLD < COST_REC ? COST_OLD : COST_REC;
constexpr int MASK_LP = 0x3FFFFFFF / PAGE;  // logical page whose tokens are all masked

struct DecodeArgs {
  PoolView P;
  int layer, n_req, max_pages;
  const uint16_t* q;
  const int32_t* bt;
  const uint8_t* tags;
  const int32_t* seq_lens;
  float* out;
  float* lse;
  float* partials;
  int cunits, max_chunks;  // cost units per chunk, chunk slots per (request, KV head)
  float sm_log2;  // log2(e) / sqrt(d)
  // decode-step append fused into the call (APP instance): one new token per
  // request, K and V rows [n_req][n_kv_heads][d] (bf16); seq_lens then holds
  // the lengths before the append
  const uint16_t* k_new;
  const uint16_t* v_new;
  int32_t* bt_w;    // the same block table and tags, written by the append
  uint8_t* tags_w;
  // per request: the fresh page's id, or -1 (no fresh page, or the call
  // failed); then the FP8 free-list top after the call, or -1.  Written by
  // the scan, published by the merge kernel.
  int32_t* app_rec;
  // SCORE instance: per (request, logical page, query head) the page's local
  // softmax mass sum_i 2^(s_i - m) and the reference exponent m it was taken
  // against (base 2, units of the scaled scores)
  float2* page_mass;
};

// Cost of a request's pages: n_old pages wholly outside the Recent window and
// n_pages - n_old inside it.  Non-decreasing in the sequence length, so the
// table width bounds every request's cost.
__host__ __device__ inline int64_t request_cost(int64_t n_pages, int64_t n_old) {
  return COST_OLD * n_old + COST_REC * (n_pages - n_old);
}
__host__ __device__ inline int64_t old_pages(int64_t seq_len, int recent) {
  return seq_len > recent ? (seq_len - recent) / PAGE : 0;
}
// first page whose cost prefix is at least c
__device__ inline int page_at_cost(int64_t c, int n_old) {
  const int64_t co = (int64_t)COST_OLD * n_old;
  if (c <= co) return (int)((c + COST_OLD - 1) / COST_OLD);
  return n_old + (int)((c - co + COST_REC - 1) / COST_REC);
}

// Units per chunk: about one workgroup per CU for the whole launch when the
// requests fill their tables (256 CUs), never below 16 old pages' worth and
// never spanning more than MAX_CHUNK_PAGES pages.
DecodeShape decode_shape(int n_req, int max_pages, int n_kv_heads, int recent) {
  DecodeShape s;
  const int64_t tmax = request_cost(max_pages, old_pages((int64_t)max_pages * PAGE, recent));
  const int64_t pairs = (int64_t)n_req * n_kv_heads;
  int64_t u = (tmax * pairs + 255) / 256;
  if (u < 16 * COST_OLD) u = 16 * COST_OLD;
  if (u > (int64_t)(MAX_CHUNK_PAGES - 1) * COST_MIN) u = (int64_t)(MAX_CHUNK_PAGES - 1) * COST_MIN;
  s.cunits = (int)u;
  s.max_chunks = (int)((tmax + u - 1) / u);
  return s;
}

// workspace: the partials, one (O_j[G][d], m_j[G], l_j[G]) block per chunk
// slot, padded to a multiple of 4 floats (16-byte aligned O rows); every slot
// of the grid is written on every call (l_j = 0 when the chunk is empty or
// past the request's end), so the merge needs no count
__host__ __device__ constexpr int part_stride(int G, int D) { return (G * (D + 2) + 3) / 4 * 4; }

// bytes of the split partials; the fused append's per-request records follow
static size_t decode_part_bytes(const DecodeShape& s, int n_req, int n_kv_heads, int group, int d) {
  return (size_t)n_req * n_kv_heads * s.max_chunks * part_stride(group, d) * sizeof(float);
}
size_t decode_ws_bytes(int n_req, int max_pages, int n_kv_heads, int group, int d, int recent) {
  DecodeShape s = decode_shape(n_req, max_pages, n_kv_heads, recent);
  return decode_part_bytes(s, n_req, n_kv_heads, group, d) + ((size_t)(n_req + 1) * 4 + 15) / 16 * 16;
}

template <int D>
struct WaveState {
  float4v acc[D / 16];  // rows (page parity, head) x channels, see below
  float m_run;          // running max of this lane's column (base-2 units)
  float l_run;          // partial denominator over this lane's tokens
};
// Initial reference max: finite, so 2^(s - m) is 0 for masked scores (s = -inf)
// and never NaN; a column with l = 0 takes no part in any merge.
constexpr float M_INIT = -1.0e30f;
// The rotated query enters the TQ3 score product as a sum of E4M3 terms,
// q sc = t0 + t1 + t2 (each term the E4M3 rounding of what the previous ones
// left; sc a power of two that puts the head's largest |q sc| in [128, 256)).
// The residual is below E4M3's subnormal step 2^-9, i.e. about 2^-17 of the
// head's largest entry.
constexpr int QF8_TERMS = 3;

// Column layout of a score tile (and row layout of the PV accumulator).  With
// at most six heads per KV head, heads sit in columns 4 k + i, i < 3, so that
// accumulator element 3 of every lane is padding and its updates are skipped.
template <bool G6>
__device__ __forceinline__ int head_of_col(int c) {
  if constexpr (G6) return (c & 3) == 3 ? -1 : 3 * (c >> 2) + (c & 3);
  else return c;
}

// Online-softmax step: sc[4] are this lane's base-2 scores (tokens 4*lg + i of
// the page that owns column ln).  Weights are returned in place.  The
// accumulator rows 4*lg + i belong to columns 4*lg + i, whose rescale factors
// are fetched from those lanes when the reference max moves.
template <int D, int NI>
__device__ __forceinline__ void softmax_step(WaveState<D>& st, float* sc, int lg) {
  const float mx = max4rows(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3])));
  // lazy rescale: keep the reference max while new scores stay within 2^8
  const bool need = mx > st.m_run + 8.0f;
  if (__any(need)) {
    const float m_new = need ? mx : st.m_run;
    const float alpha = __builtin_amdgcn_exp2f(st.m_run - m_new);
    st.l_run *= alpha;
    st.m_run = m_new;
    float ar[4];
#pragma unroll
    for (int i = 0; i < NI; ++i) ar[i] = __shfl(alpha, 4 * lg + i, 64);
#pragma unroll
    for (int m = 0; m < D / 16; ++m)
#pragma unroll
      for (int i = 0; i < NI; ++i) st.acc[m][i] *= ar[i];
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sc[i] = __builtin_amdgcn_exp2f(sc[i] - st.m_run);  // -inf -> 0
    st.l_run += sc[i];
  }
}

// P^T operand of the PV product: row ln = this lane's column; tokens
// (4*lg + j) of page a for j < 4 and of page b for j >= 4 (block-diagonal:
// page-a rows see only page-a tokens).
// The weights go in as an fp16 hi + lo pair (hi: rounded weight, lo: the
// rounding remainder): a token holding most of a row's mass has, against a
// lagging reference max, a weight that fp16 alone would round by up to 2^-12
// of that token's value.
// hi is the weight rounded to fp16, lo the rounded remainder (together 22
// significant bits; round-to-nearest: the packed round-toward-zero conversion
// flushes fp16 subnormals, which drops the low part of every weight below
// 2^-4).
__device__ __forceinline__ void p_operand(const float* p, bool row_is_b, half8& hi, half8& lo) {
  typedef _Float16 h2t __attribute__((ext_vector_type(2)));
  const h2t h01 = {(_Float16)p[0], (_Float16)p[1]};
  const h2t h23 = {(_Float16)p[2], (_Float16)p[3]};
  const h2t l01 = {(_Float16)(p[0] - (float)h01[0]), (_Float16)(p[1] - (float)h01[1])};
  const h2t l23 = {(_Float16)(p[2] - (float)h23[0]), (_Float16)(p[3] - (float)h23[1])};
  typedef uint32_t u4v __attribute__((ext_vector_type(4)));
  const uint32_t a0 = __builtin_bit_cast(uint32_t, h01), a1 = __builtin_bit_cast(uint32_t, h23);
  const uint32_t b0 = __builtin_bit_cast(uint32_t, l01), b1 = __builtin_bit_cast(uint32_t, l23);
  const u4v H = row_is_b ? u4v{0u, 0u, a0, a1} : u4v{a0, a1, 0u, 0u};
  const u4v L = row_is_b ? u4v{0u, 0u, b0, b1} : u4v{b0, b1, 0u, 0u};
  hi = __builtin_bit_cast(half8, H);
  lo = __builtin_bit_cast(half8, L);
}

// PAIR (query group of at most 8 heads): two pages share one score tile,
// columns [0, 8) scoring page a and [8, 16) page b.  G6: at most six heads
// (see head_of_col).
template <int D, bool PAIR, bool G6, bool APP, bool SCORE = false>
__global__ __launch_bounds__(DecodeCfg<PAIR>::NT, 1) void decode_kernel(DecodeArgs a) {
  static_assert(!(APP && SCORE), "the scoring instance has no fused append");
  constexpr int NW = DecodeCfg<PAIR>::NW, NT = DecodeCfg<PAIR>::NT, SLOTS = DecodeCfg<PAIR>::SLOTS;
  constexpr int NCH = NCH_OF(PAIR);  // query heads a score tile holds
  constexpr int CL = D / 16, NDW = 3 * D / 128, CB = 3 * D / 32, NS = D / 32, QV = D / 64;
  constexpr int NK8 = D / 128;  // 128-channel steps of the TQ3 score product (32 channels per lane group)
  constexpr int R3 = (int)tq3_region_bytes(D);  // K codes, V codes, gamma, V scale, V zero
  constexpr int R8 = (int)fp8_region_bytes(D);  // K codes then V codes
  constexpr int STAGE = 2 * R3;                 // a TQ3 page pair, or one FP8 page + scales
  constexpr int OPS3 = dma_ops<R3>(), OPS8 = dma_ops<R8>() + 1;
  static_assert(dma_ops<R8>() == 2 * (D / 64), "dma_fp8_page issues 2 d / 64 copies");
  static_assert(R8 + 8 <= STAGE, "an FP8 page and its two scales fit one stage");
  static_assert(NW % 4 == 0, "per-head wave statistics are read as float4s");
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ int4 s_stage[MAX_CHUNK_PAGES];  // {lp_a, id_a, lp_b, id_b}; id_b < 0: FP8 stage
  __shared__ int s_next;  // next unclaimed stage (one-slot schedule)
  __shared__ int s_app, s_app_bad;  // fused append: append waves done, error flag
  // per (head, wave): running max and denominator (epilogue)
  __shared__ __align__(16) float s_mlf[2][16 * NW_MAX];
  static_assert(NCH_OF(PAIR) * D * 4 <= SLOTS * 2 * (int)tq3_region_bytes(D),
                "a wave's merged rows fit its own ring slot");
  const PoolView& P = a.P;
  const int r = blockIdx.z, h = blockIdx.y, chunk = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = P.group, H = P.n_kv_heads, Hq = H * G;
  const int mp = a.max_pages;
  constexpr bool pair = PAIR;
  // The arguments the prologue needs come in one batch of loads from the
  // argument segment: otherwise the compiler fetches some of them (the chunk
  // size, the pool and partial pointers) only after the first batch has
  // returned, and the page-table loads wait for a second round trip.
  asm volatile("" ::"s"(a.cunits), "s"(a.bt), "s"(a.tags), "s"(a.seq_lens), "s"(a.q), "s"(P.sigma),
               "s"(P.recent), "s"(mp), "s"(a.n_req), "s"(P.tq3), "s"(P.fp8), "s"(a.partials));
  // LDS: [rotated query as E4M3 terms][plain-query operand][page ring | wave merge]
  uint8_t* qf8 = smem;  // [term][step][lane][32 bytes], see the query build below
  half8* qpl = reinterpret_cast<half8*>(smem + QF8_TERMS * NK8 * 64 * 32);  // plain query (bf16 -> fp16 is exact)
  uint8_t* ring = smem + QF8_TERMS * NK8 * 64 * 32 + NS * 64 * 16;
  __shared__ float s_qinv[16];  // per score column: 1 / the power-of-two scale of its terms

  // ---- 1. queries: wave w owns score columns w and w + NW below NCH (the
  // head of a column: head_of_col); lane l holds channels QV l .. QV l + QV -
  // 1.  The loads go out before anything else so their latency hides behind
  // the page-table loads.
  static_assert(QV == 2 || QV == 4, "QV bf16 channels per lane form one 4- or 8-byte load");
  using qvec = typename std::conditional<QV == 4, uint2, uint32_t>::type;
  float qx[2][QV];
  int sg[QV];
#pragma unroll
  for (int ps = 0; ps < 2; ++ps) {
    const int hd = head_of_col<G6>(wid + NW * ps);
    const bool ok = hd >= 0 && hd < G;
    const int nn = ok ? hd : 0;  // loads stay in bounds; padding columns get zeros
    const qvec raw = *reinterpret_cast<const qvec*>(a.q + ((int64_t)r * Hq + h * G + nn) * D + QV * lane);
    const uint16_t* rh = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
    for (int i = 0; i < QV; ++i) qx[ps][i] = ok ? bf16_to_f32(rh[i]) : 0.0f;
  }
#pragma unroll
  for (int i = 0; i < QV; ++i) sg[i] = P.sigma[QV * lane + i];

  float* part = a.partials + (((int64_t)r * H + h) * a.max_chunks + chunk) * part_stride(G, D);
  // ---- chunk -> logical page range: equal-cost ranges over the table width,
  // known before any load, so the sequence length and the chunk's tags and
  // ids are loaded together; pages at or past the request's end are dropped
  // once the length is in (chunk < max_chunks, so the range is not empty)
  const int n_old_t = (int)old_pages((int64_t)mp * PAGE, P.recent);
  const int64_t c0 = (int64_t)chunk * a.cunits;
  const int p0 = page_at_cost(c0, n_old_t);
  const int p1 = page_at_cost(min(request_cost(mp, n_old_t), c0 + a.cunits), n_old_t);
  const int n_pr = p1 - p0;
  // ---- 2. per-format compact lists of the chunk (logical order) -> stages.
  // Every wave reads the tags and ids of the whole chunk (lane l holds pages
  // l + 64 k), so each finds its first stages from its own ballots and starts
  // their copies before any workgroup barrier; wave 0 writes the stage list
  // that later claims read from LDS.
  constexpr int PW = MAX_CHUNK_PAGES / 64;
  const uint64_t below = (1ull << lane) - 1ull;
  int pg_lp[PW], pg_id[PW];
  uint64_t m3w[PW], m8w[PW];
  int n3 = 0, n8 = 0;
  int tg_w[PW];
#pragma unroll
  for (int k = 0; k < PW; ++k) {  // all loads in flight together (clamped to the chunk)
    const int64_t pi = (int64_t)r * mp + p0 + min(lane + 64 * k, n_pr - 1);
    tg_w[k] = a.tags[pi];
    pg_id[k] = a.bt[pi];
  }
  const int s_in = a.seq_lens[r];
  // with the fused append the request's new token sits at position s_in
  const int S = !APP ? s_in : (s_in >= 0 && s_in < mp * PAGE ? s_in + 1 : -1);
  if (S < 1 || S > mp * PAGE) {
    if (chunk == 0 && h == 0 && tid == 0) atomicOr(&P.ctrl[CTRL_ERR], (int)MKV_DEVERR_RANGE);
    if (APP && chunk == 0 && h == 0 && tid == 0) {  // no workgroup holds this request's token
      a.app_rec[r] = -1;
      if (r == 0) a.app_rec[a.n_req] = -1;
    }
    if (tid < G) part[G * D + G + tid] = 0.0f;  // empty partial: the merge writes zeros
    return;
  }
  const int n_pg = min(p1, (S + PAGE - 1) / PAGE) - p0;  // pages of the chunk before the end
  if (n_pg <= 0) {
    if (tid < G) part[G * D + G + tid] = 0.0f;  // slot past the request's end
    return;
  }
  // ---- query operands, built while the page-table loads are in flight, in MFMA
  // lane order (ln = lane % 16 the score column, lg = lane / 16):
  //  qpl[s][lane] holds channels (D/4) lg + 8 s + j, j < 8 (fp16, FP8 pages);
  //  qf8[t][S][lane] holds term t of channels (D/4) lg + 32 S + j, j < 32 (the
  //  f8f6f4 MFMA pairs byte j of lane l in A with byte j of lane l' in B
  //  whenever l / 16 = l' / 16, so any channel order common to both operands
  //  works; this one matches the key quads)
  {
    _Float16* qp = reinterpret_cast<_Float16*>(qpl);
    // R = d^-1/2 H diag(sigma); the rotated query also carries the softmax
    // scale log2(e)/sqrt(d), so TQ3 scores come out in base-2 units
    const float qscale = rsqrtf((float)D) * a.sm_log2;
#pragma unroll
    for (int ps = 0; ps < 2; ++ps) {
      const int n = wid + NW * ps;
      if (n >= NCH) break;  // wave-uniform
      const int hd = head_of_col<G6>(n);
      const bool ok = hd >= 0 && hd < G;
      float xr[QV];
#pragma unroll
      for (int i = 0; i < QV; ++i) xr[i] = qx[ps][i] * (float)sg[i];
      // fast Walsh-Hadamard transform: strides below QV inside the lane,
      // the rest across lanes (partner lane = lane ^ (stride / QV))
#pragma unroll
      for (int st = 1; st < QV; st <<= 1)
#pragma unroll
        for (int i = 0; i < QV; ++i)
          if (!(i & st)) {
            const float x0 = xr[i], x1 = xr[i + st];
            xr[i] = x0 + x1;
            xr[i + st] = x0 - x1;
          }
      auto stage = [&](auto mc) {
        constexpr int m = decltype(mc)::value;
        const float sg_m = (lane & m) ? -1.0f : 1.0f;  // this lane holds the upper element
#pragma unroll
        for (int i = 0; i < QV; ++i) xr[i] = fmaf(sg_m, xr[i], lane_xor<m>(xr[i], lane));
      };
      stage(std::integral_constant<int, 1>{});
      stage(std::integral_constant<int, 2>{});
      stage(std::integral_constant<int, 4>{});
      stage(std::integral_constant<int, 8>{});
      stage(std::integral_constant<int, 16>{});
      stage(std::integral_constant<int, 32>{});
      // the head's power-of-two scale: largest |q sc| in [128, 256)
      float amax = 0.0f;
#pragma unroll
      for (int i = 0; i < QV; ++i) amax = fmaxf(amax, fabsf(xr[i] * qscale));
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
      int ex = 0;
      (void)frexpf(amax, &ex);  // amax in [2^(ex-1), 2^ex)
      const float qsc = (ok && amax > 0.0f) ? ldexpf(1.0f, 7 - ex + 1) : 1.0f;
      if (lane == 0) {
        s_qinv[n] = 1.0f / qsc;
        if (pair) s_qinv[n + 8] = 1.0f / qsc;
      }
#pragma unroll
      for (int i = 0; i < QV; ++i) {
        const int c = QV * lane + i;
        const int lgc = c / (D / 4), sc = (c % (D / 4)) / 8, j = c % 8;
        const _Float16 vp = (_Float16)(ok ? qx[ps][i] : 0.0f);
        const int e0 = ((sc * 64) + lgc * 16 + n) * 8 + j;
        qp[e0] = vp;
        if (pair) qp[e0 + 8 * 8] = vp;  // column n + 8 scores page b with the same head
        // rotated query times its scale as three E4M3 terms (exact residuals)
        float x = ok ? xr[i] * qscale * qsc : 0.0f;
        const int S = (c % (D / 4)) / 32, slot = c % 32;
#pragma unroll
        for (int t = 0; t < QF8_TERMS; ++t) {
          const uint32_t b = f32_to_e4m3(x);
          x -= e4m3_to_f32(b);
          const int e8 = ((t * NK8 + S) * 64 + lgc * 16 + n) * 32 + slot;
          qf8[e8] = (uint8_t)b;
          if (pair) qf8[e8 + 8 * 32] = (uint8_t)b;
        }
      }
    }
  }

  // fused append: the request's new token lands in logical page p_new (a
  // fresh page when its table entry is negative, whose physical id the
  // workgroup learns later); the chunk that holds p_new counts it as a Recent
  // FP8 page, the last of its FP8 stages
  const int p_new = APP ? s_in / PAGE : -1;
  const bool holds = APP && p_new >= p0 && p_new < p1;
#pragma unroll
  for (int k = 0; k < PW; ++k) {
    const int pi = lane + 64 * k;
    int tg = pi < n_pg ? tg_w[k] : -1;
    int id = pg_id[k];
    if (APP && holds && p0 + pi == p_new) {
      tg = TAG_R;
      if (id < 0) id = 0;  // fresh: placeholder until the append wave has popped the id
    }
    const bool is3 = tg == TAG_S, is8 = (tg == TAG_R || tg == TAG_A);
    if (wid == 0 && pi < n_pg && !is3 && !is8) atomicOr(&P.ctrl[CTRL_ERR], (int)MKV_DEVERR_BAD_TAG);
    int lp = p0 + pi;
    if ((is3 || is8) && (id < 0 || id >= (is3 ? P.n_tq3 : P.n_fp8))) {
      // out-of-range physical id: read page 0 instead, mask every token
      if (wid == 0) atomicOr(&P.ctrl[CTRL_ERR], (int)MKV_DEVERR_RANGE);
      id = 0;
      lp = MASK_LP;
    }
    pg_lp[k] = lp;
    pg_id[k] = id;
    m3w[k] = __ballot(is3);
    m8w[k] = __ballot(is8);
    n3 += __popcll(m3w[k]);
    n8 += __popcll(m8w[k]);
  }
  const int st3 = pair ? (n3 + 1) / 2 : n3;
  const int n_st = st3 + n8;
  // (logical page, id) of the page of rank q among the chunk's TQ3 (fmt 0) or
  // FP8 (fmt 1) pages
  auto page_of = [&](int fmt, int q) {
    int2 res = make_int2(MASK_LP, 0);
    int base = 0;
#pragma unroll
    for (int k = 0; k < PW; ++k) {
      const uint64_t m = fmt ? m8w[k] : m3w[k];
      const int cnt = __popcll(m);
      if (q >= base && q < base + cnt) {
        const uint64_t hit = __ballot(((m >> lane) & 1ull) && base + __popcll(m & below) == q);
        const int src = __builtin_amdgcn_readfirstlane(__ffsll((unsigned long long)hit) - 1);
        res = make_int2(__builtin_amdgcn_readlane(pg_lp[k], src), __builtin_amdgcn_readlane(pg_id[k], src));
      }
      base += cnt;
    }
    return res;
  };
  // stage j -> {lp_a, id_a, lp_b, id_b}; id_b < 0 marks an FP8 stage (the
  // same entries wave 0 writes to s_stage)
  auto stage_of = [&](int j) {
    if (j < st3) {
      const int2 ea = page_of(0, pair ? 2 * j : j);
      const int2 eb = (pair && 2 * j + 1 < n3) ? page_of(0, 2 * j + 1) : make_int2(MASK_LP, ea.y);
      return make_int4(ea.x, ea.y, eb.x, eb.y);
    }
    const int2 e8 = page_of(1, j - st3);
    return make_int4(e8.x, e8.y, 0, -1);
  };
  if (wid == 0) {
    int2* s2 = reinterpret_cast<int2*>(s_stage);
    int base3 = 0, base8 = 0;
#pragma unroll
    for (int k = 0; k < PW; ++k) {
      if ((m3w[k] >> lane) & 1ull) {
        const int rank = base3 + __popcll(m3w[k] & below);
        if (pair) {
          s2[rank] = make_int2(pg_lp[k], pg_id[k]);  // stage rank / 2, half rank % 2
          if (rank == n3 - 1 && !(rank & 1)) s2[rank + 1] = make_int2(MASK_LP, pg_id[k]);
        } else {
          s_stage[rank] = make_int4(pg_lp[k], pg_id[k], MASK_LP, pg_id[k]);
        }
      }
      if ((m8w[k] >> lane) & 1ull)
        s_stage[st3 + base8 + __popcll(m8w[k] & below)] = make_int4(pg_lp[k], pg_id[k], 0, -1);
      base3 += __popcll(m3w[k]);
      base8 += __popcll(m8w[k]);
    }
  }
  if (tid == 0) {
    s_next = NW;
    s_app = 0;
    s_app_bad = 0;
  }

  // ---- 3. per-wave stream over the claimed stages
  WaveState<D> st;
#pragma unroll
  for (int m = 0; m < CL; ++m) st.acc[m] = float4v{0.f, 0.f, 0.f, 0.f};
  st.m_run = M_INIT;
  st.l_run = 0.0f;
  const int ln = lane & 15, lg = lane >> 4;
  const int col_head = head_of_col<G6>(pair ? (ln & 7) : ln);
  const bool col_valid = col_head >= 0 && col_head < G;
  const bool col_b = pair && ln >= 8;  // this column scores page b
  const bool row_b = pair && lg >= 2;  // accumulator rows 4*lg+i hold page b
  const float col_bias = col_valid ? 0.0f : -INFINITY;  // masks padding columns
  const float fp8_bias = (col_valid && !col_b) ? 0.0f : -INFINITY;  // FP8 stages: page a only
  constexpr int NI = G6 ? 3 : 4;  // accumulator elements that hold a head
  // Stage schedule: wave w starts with stage w and claims each later stage
  // from an LDS counter when it begins a stage, so the waves of a SIMD finish
  // together (stages differ in cost and the waves of a SIMD do not get equal
  // issue shares).  With two slots per wave the claimed stage after the
  // current one is already in flight.
  // A SIMD issues the instructions of its oldest wave first: waves 0-3 get
  // most of their SIMD, the later ones what is left.  Near the end of the
  // stage list the younger waves stop claiming (a stage they take would
  // finish last), so the last stages run on the faster waves.
  // With the deterministic schedule wave w takes stages w, w + NW, w + 2 NW,
  // ..., so every call folds the same pages in the same order and the outputs
  // are bit-identical from call to call.
  int det_next = wid + NW;
  auto claim = [&]() {
    if (a.P.deterministic) {
      const int v = min(det_next, n_st);
      det_next += NW;
      return v;
    }
    int v = 0;
    if (lane == 0) {
      const int rank = wid / 4;
      const int keep = rank == 0 ? 0 : rank == 1 ? 3 : 24;  // stages left for older waves
      const int seen = __atomic_load_n(&s_next, __ATOMIC_RELAXED);
      v = (n_st - seen <= keep) ? n_st : atomicAdd(&s_next, 1);
    }
    return __builtin_amdgcn_readfirstlane(v);
  };
  const float smk = a.sm_log2;
  const float4v zero4 = {0.f, 0.f, 0.f, 0.f};
  half8 ones8;
#pragma unroll
  for (int j = 0; j < 8; ++j) ones8[j] = (_Float16)1.0f;
  const int layer = a.layer;
  const uint8_t* tq3_l = P.tq3 + (int64_t)layer * P.n_tq3 * H * R3;
  const uint8_t* fp8_l = P.fp8 + (int64_t)layer * P.n_fp8 * H * R8;
  const uint8_t* scl_l = reinterpret_cast<const uint8_t*>(P.fp8_scales + (int64_t)layer * P.n_fp8 * H * 2);
  uint8_t* wring = ring + wid * SLOTS * STAGE;
  const uint32_t wring_lds = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)wring);
  auto stage_at = [&](int j) {
    const int4 e = s_stage[j];
    return make_int4(__builtin_amdgcn_readfirstlane(e.x), __builtin_amdgcn_readfirstlane(e.y),
                     __builtin_amdgcn_readfirstlane(e.z), __builtin_amdgcn_readfirstlane(e.w));
  };
  const DmaLanes dl = {16u * lane, 4096u + 16u * lane};
  auto issue = [&](int4 e, int slot) {
    if constexpr (APP) {
      // the page of the appended token: its copy waits until the append wave
      // has stored the token (and, for a fresh page, popped its id)
      if (holds && e.w < 0 && e.x == p_new) {
        while (__hip_atomic_load(&s_app, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < 2)
          __builtin_amdgcn_s_sleep(1);
        e = stage_at(n_st - 1);
      }
    }
    const uint32_t dst = wring_lds + slot * STAGE;
    if (e.w >= 0) {
      dma_region<R3>(dst, tq3_l + ((int64_t)e.y * H + h) * R3, dl, lane);
      if (pair) dma_region<R3>(dst + R3, tq3_l + ((int64_t)e.w * H + h) * R3, dl, lane);
    } else {
      dma_fp8_page<D>(dst, fp8_l + ((int64_t)e.y * H + h) * R8, lane);
      if (lane < 2) dma4(4 * lane, scl_l + ((int64_t)e.y * H + h) * 8, dst + R8);
    }
  };
  // Fused decode-step append (APP), run by the two youngest waves of the
  // workgroup that holds the request's new token (K by the older, V by the
  // younger), after the workgroup barrier, while the other waves stream:
  // every such wave reads the whole call (each request's length, the
  // free-list top, the table entries and tags of the
  // pages being appended to) and so reaches the same verdict and the same
  // fresh-page ids as the decode-step append kernel (same validation, ids
  // popped in request order, same arithmetic); it stores K and V of head h
  // for the new token (Alg. 1, Append), then counts itself on an LDS flag; the
  // appended page's stage is released when both have.  Head 0's K wave
  // records the request's fresh id (and request 0's the new free-list top)
  // in the workspace; the merge kernel, which runs after every workgroup of
  // the scan has read the table, writes them into the block table, tags and
  // free-list top.  On any error nothing is written, the error word gets its
  // bits, and the workgroup's partial is marked so that the merge writes
  // zeros for the call.
  auto append_token = [&]() {
    // the append waves are the youngest of their SIMDs: without a raised
    // priority the streaming waves starve them and the appended page's stage,
    // which waits for them, runs last
    STAGE_PRIO(3);
    int bad = 0, n_fresh = 0, rank = 0;
    bool fresh = false;  // this request's page is fresh
    const int top = P.ctrl[CTRL_FP8_TOP];
    for (int b0 = 0; b0 < a.n_req; b0 += 64) {
      const int rr = b0 + lane;
      const bool in = rr < a.n_req;
      const int sr = in ? a.seq_lens[rr] : 0;
      const bool ok = !in || (sr >= 0 && sr < mp * PAGE);
      bool fr = false;
      if (!ok) {
        bad |= MKV_DEVERR_RANGE;
      } else if (in) {
        // a negative table entry opens a fresh page, any other must be a
        // Recent page in range
        const int64_t ix = (int64_t)rr * mp + sr / PAGE;
        const int idr = a.bt[ix];
        fr = idr < 0;
        if (!fr) {
          if (a.tags[ix] != TAG_R) bad |= MKV_DEVERR_NOT_RECENT;
          else if (idr >= P.n_fp8) bad |= MKV_DEVERR_RANGE;
        }
      }
      const uint64_t fm = __ballot(fr);
      if (r >= b0 + 64) rank += __popcll(fm);
      else if (r >= b0) {
        rank += __popcll(fm & ((1ull << (r - b0)) - 1ull));
        fresh = (fm >> (r - b0)) & 1ull;
      }
      n_fresh += __popcll(fm);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) bad |= __shfl_xor(bad, o, 64);
    if (n_fresh > top) bad |= MKV_DEVERR_FP8_EXHAUSTED;
    bad = __builtin_amdgcn_readfirstlane(bad);
    const int id = bad ? -1 : __builtin_amdgcn_readfirstlane(
        fresh ? P.fp8_stack[top - 1 - rank] : a.bt[(int64_t)r * mp + p_new]);
    if (!bad) {
      // the task's code block and table: the wave's second ring slot (its
      // first copy is in flight in the first), or its only slot
      const int kv = wid - (NW - 2);
      uint8_t* own = SLOTS == 2 ? wring + STAGE : wring;
      SmallTask<D> T;
      T.kv = kv;
      T.r = r;
      T.p = p_new;
      T.t0 = s_in % PAGE;
      T.t1 = T.t0 + 1;
      T.row0 = r - T.t0;  // the token's input row is r
      T.layer = a.layer;
      T.li = 0;
      T.h = h;
      small_task_load_x<D>(T, H, a.n_req, a.k_new, a.v_new, lane);
      small_task_load_old<D>(T, P, id, lane);
      small_task_run<D>(T, P, id, reinterpret_cast<uint32_t*>(own), own + PAGE * D, lane);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the token's codes and scale are stored
      if (lane == 0 && kv == 0) s_stage[n_st - 1].y = id;
    } else if (lane == 0) {
      atomicOr(&P.ctrl[CTRL_ERR], bad);
      s_app_bad = 1;
    }
    if (lane == 0) __hip_atomic_fetch_add(&s_app, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    // the record the merge kernel publishes (one writer per request: head 0's
    // K wave)
    if (h == 0 && wid == NW - 2 && lane == 0) {
      a.app_rec[r] = fresh ? id : -1;
      if (r == 0) a.app_rec[a.n_req] = bad ? -1 : top - n_fresh;
    }
  };
  int jc = min(wid, n_st);  // stage this wave processes next
  int jq = n_st;            // two slots: the claimed stage after jc (in flight)
  // the oldest wave of each SIMD copies its first stage now, the others after
  // the barrier: the first copies of a launch queue behind every workgroup's,
  // and each SIMD should get its first stage early
  // (with the fused append, the appended page's stage waits for the append)
  const bool defer0 = APP && holds && jc == n_st - 1;
  if (wid < 4 && jc < n_st && !defer0) issue(stage_of(jc), 0);

  __syncthreads();  // query operands and the stage list visible to every wave
  const float qinv = s_qinv[ln];  // undoes the query-term scale of this lane's column
  if (APP && holds && wid >= NW - 2) {
    // an append wave with two slots copies its first stage before the task
    // (unless that stage is the appended page's), so the copy's latency
    // overlaps it; with one slot the task uses the slot first
    if (SLOTS == 2 && jc < n_st - 1) issue(stage_at(jc), 0);
    append_token();
    if (SLOTS == 1 && jc < n_st - 1) issue(stage_at(jc), 0);
    if (jc == n_st - 1) issue(stage_at(jc), 0);
  } else if ((wid >= 4 || defer0) && jc < n_st) {
    issue(stage_at(jc), 0);
  }
  if (SLOTS == 2 && jc < n_st) {
    jq = claim();
    if (jq < n_st) issue(stage_at(jq), 1);
  }
  // Wait for stage j to land in its slot; with two slots the stage after it
  // may stay in flight (the allowed count is the number of copies it was
  // issued as).
  auto begin_stage = [&](int j) {
    const int nops = (SLOTS > 1 && jq < n_st) ? (stage_at(jq).w >= 0 ? (pair ? 2 : 1) * OPS3 : OPS8) : 0;
    if (nops == 2 * OPS3)
      wait_vmcnt<2 * OPS3>();
    else if (nops == OPS8)
      wait_vmcnt<OPS8>();
    else if (nops == OPS3)
      wait_vmcnt<OPS3>();
    else
      wait_vmcnt<0>();
  };
  // TQ3 stages come first in the list, FP8 stages after them; the two loops
  // share the ring (a copy in flight may belong to either format).
  // Score collector (SCORE instance, Sec. 3.1 Eq. score-partial): after the
  // softmax step a lane's four weights are 2^(s - m_run) of tokens of the
  // page its column scores; their sum over the column's 16 tokens is the
  // page's local mass against m_run, stored with m_run for the collector,
  // which rescales it by the global normalization (Eq. score-global-weight).
  auto record_mass = [&](const float* w, int lp) {
    const float ms = sum4rows((w[0] + w[1]) + (w[2] + w[3]));
    if (lg == 0 && col_valid && lp < (S + PAGE - 1) / PAGE)
      a.page_mass[((int64_t)r * mp + lp) * Hq + h * G + col_head] = make_float2(ms, st.m_run);
  };
  int k_st = 0;  // stages begun by this wave; stage k sits in slot k % SLOTS
  while (jc < st3) {
    const int j = jc;
    const int slot = k_st % SLOTS;
    const int jr = claim();  // stage that refills this slot
    const int4 e = stage_at(j);
    STAGE_PRIO(1);
    begin_stage(j);
    const bool refill = jr < n_st;
    const int4 e2 = refill ? stage_at(jr) : e;
    const uint8_t* ra = wring + slot * STAGE;
    // TQ3 pair (page b absent: same page, every token masked)
    const uint8_t* rb = pair ? ra + R3 : ra;
    const uint8_t* rown = row_b ? rb : ra;
    uint32_t kA[NDW], kB[NDW], vA[NDW], vB[NDW];
    read_chunk<NDW>(kA, ra, 16 * lg + ln);
    read_chunk<NDW>(kB, rb, 16 * lg + ln);
    read_chunk<NDW>(vA, ra + 6 * D, 16 * lg + ln);
    read_chunk<NDW>(vB, rb + 6 * D, 16 * lg + ln);
    const uint2 gw = *reinterpret_cast<const uint2*>((col_b ? rb : ra) + 12 * D + 8 * lg);
    // per-channel V scale and zero of this lane's row page
    half2v sO[CL / 2], zO[CL / 2];
#pragma unroll
    for (int i = 0; i < CL / 2; ++i) {
      sO[i] = reinterpret_cast<const half2v*>(rown + 12 * D + 32 + 2 * CL * ln)[i];
      zO[i] = reinterpret_cast<const half2v*>(rown + 14 * D + 32 + 2 * CL * ln)[i];
    }
    wait_lgkm0();  // the stage is in registers: refill its slot
    if (refill) issue(e2, slot);
    // QK^T: rows = tokens of the page, columns = (page, head), on the
    // 16x16x128 fp8 MFMA: the 3-bit codes become E4M3 codebook bytes (one
    // v_perm per 4 codes) and meet the query's E4M3 terms directly
    float4v sa = zero4, sb = zero4;
#pragma unroll
    for (int S = 0; S < NK8; ++S) {
      v8i Ka, Kb;
#pragma unroll
      for (int w = 0; w < 8; ++w) {
        Ka[w] = (int)__builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kA, 8 * S + w));
        if (pair) Kb[w] = (int)__builtin_amdgcn_perm(KLUT_HI, KLUT_LO, quad_sel<NDW>(kB, 8 * S + w));
      }
#pragma unroll
      for (int t = 0; t < QF8_TERMS; ++t) {
        const v8i qv = *reinterpret_cast<const v8i*>(qf8 + ((t * NK8 + S) * 64 + lane) * 32);
        sa = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(Ka, qv, sa, 0, 0, 0, 0, 0, 0);
        if (pair) sb = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(Kb, qv, sb, 0, 0, 0, 0, 0, 0);
      }
    }
    float sc[4];
    {
      const _Float16* gh = reinterpret_cast<const _Float16*>(&gw);
#pragma unroll
      for (int i = 0; i < 4; ++i) sc[i] = fmaf((col_b ? sb[i] : sa[i]) * qinv, (float)gh[i], col_bias);
      // tokens at or past the end: only in a stage that holds the request's
      // last page or a masked page b
      if ((e.x + 1) * PAGE > S || (pair && (e.z + 1) * PAGE > S)) {
        const int vcnt = S - (col_b ? e.z : e.x) * PAGE;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (4 * lg + i >= vcnt) sc[i] = -INFINITY;
      }
    }
    STAGE_PRIO(2);
    softmax_step<D, NI>(st, sc, lg);
    if constexpr (SCORE) record_mass(sc, col_b ? e.z : e.x);
    STAGE_PRIO(3);
    half8 pT, pTl;
    p_operand(sc, col_b, pT, pTl);
    // PV: the codes enter the MFMA exactly (a code byte read as an E4M3
    // subnormal is c * 2^-9; the converter's power-of-two scale 2^9 makes it
    // c); v = zero + scale * code is applied in fp32 to the MFMA output,
    // the zero term through the rows' weight sums PS (MFMAs against ones)
    const float4v PS = __builtin_amdgcn_mfma_f32_16x16x32_f16(
        pTl, ones8, __builtin_amdgcn_mfma_f32_16x16x32_f16(pT, ones8, zero4, 0, 0, 0), 0, 0, 0);
    auto pv = [&](int m) {
      const uint32_t ua = quad_sel<NDW>(vA, m), ub = quad_sel<NDW>(vB, m);
      const half8 c = h8(cvt_code<false>(ua), cvt_code<true>(ua), cvt_code<false>(ub), cvt_code<true>(ub));
      return __builtin_amdgcn_mfma_f32_16x16x32_f16(
          pTl, c, __builtin_amdgcn_mfma_f32_16x16x32_f16(pT, c, zero4, 0, 0, 0), 0, 0, 0);
    };
    // one tile ahead, so the MFMA of tile m + 1 runs while tile m is scaled
    float4v X = pv(0);
#pragma unroll
    for (int m = 0; m < CL; ++m) {
      float4v Xn = X;
      if (m + 1 < CL) Xn = pv(m + 1);
      const _Float16 sm = sO[m >> 1][m & 1], zm = zO[m >> 1][m & 1];
#pragma unroll
      for (int i = 0; i < NI; ++i)
        st.acc[m][i] = fmaf((float)zm, PS[i], fmaf((float)sm, X[i], st.acc[m][i]));
      X = Xn;
    }
    if (SLOTS == 1) {
      jc = jr;
    } else {
      jc = jq;
      jq = jr;
    }
    ++k_st;
  }
  while (jc < n_st) {
    const int j = jc;
    const int slot = k_st % SLOTS;
    const int jr = claim();  // stage that refills this slot
    const int4 e = stage_at(j);
    STAGE_PRIO(1);
    begin_stage(j);
    const bool refill = jr < n_st;
    const int4 e2 = refill ? stage_at(jr) : e;
    const uint8_t* ra = wring + slot * STAGE;
    // one FP8 page (score columns of page b stay empty)
    constexpr int KW = D / 16;  // dwords of K per lane (D/4 bytes)
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
    wait_lgkm0();  // the stage is in registers: refill its slot
    if (refill) issue(e2, slot);
    float4v sa = zero4;
#pragma unroll
    for (int s = 0; s < NS; ++s)
      sa = __builtin_amdgcn_mfma_f32_16x16x32_f16(
          h8(cvt_lo(kA[2 * s]), cvt_hi(kA[2 * s]), cvt_lo(kA[2 * s + 1]), cvt_hi(kA[2 * s + 1])),
          qpl[s * 64 + lane], sa, 0, 0, 0);
    float sc[4];
    {
      const float kk = ksv.x * smk;
#pragma unroll
      for (int i = 0; i < 4; ++i) sc[i] = fmaf(sa[i], kk, fp8_bias);
      if ((e.x + 1) * PAGE > S) {
        const int vcnt = S - e.x * PAGE;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (4 * lg + i >= vcnt) sc[i] = -INFINITY;
      }
    }
    STAGE_PRIO(2);
    softmax_step<D, NI>(st, sc, lg);
    if constexpr (SCORE) record_mass(sc, col_b ? MASK_LP : e.x);
    STAGE_PRIO(3);
    half8 pT, pTl;
    p_operand(sc, col_b, pT, pTl);
    const half2v z2 = {(_Float16)0.0f, (_Float16)0.0f};
#pragma unroll
    for (int m = 0; m < CL; ++m) {
      const half8 v = h8(cvt_lo(vA[m]), cvt_hi(vA[m]), z2, z2);
      const float4v X = __builtin_amdgcn_mfma_f32_16x16x32_f16(
          pTl, v, __builtin_amdgcn_mfma_f32_16x16x32_f16(pT, v, zero4, 0, 0, 0), 0, 0, 0);
#pragma unroll
      for (int i = 0; i < NI; ++i) st.acc[m][i] = fmaf(ksv.y, X[i], st.acc[m][i]);
    }
    if (SLOTS == 1) {
      jc = jr;
    } else {
      jc = jq;
      jq = jr;
    }
    ++k_st;
  }

  // ---- 4. rows -> heads: fetch each accumulator row's (m, l); merge the two
  // page parities (rows h and h + 8 sit in lanes l and l ^ 32); then merge the
  // waves in LDS into one (m_j, l_j, O_j) partial per chunk
  const float l_col = sum4rows(st.l_run);
  float mrow[4], lrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    mrow[i] = __shfl(st.m_run, 4 * lg + i, 64);
    lrow[i] = __shfl(l_col, 4 * lg + i, 64);
  }
  if (pair) {
    // Merge the two page parities.  Rows of page b sit in lanes l + 32; one
    // permlane32 swap of acc[m] with acc[m + CL/2] puts both parities of
    // acc[m] (channel CL ln + m) in lanes l < 32 and both of acc[m + CL/2]
    // in lanes l + 32, so the merged value of acc[m] lands in the low half of
    // one register and that of acc[m + CL/2] in the high half (the factors
    // of lane l are copied to lane l + 32 first)
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const float m2 = upper_half(mrow[i]), l2 = upper_half(lrow[i]);
      const float M = fmaxf(lrow[i] > 0.0f ? mrow[i] : -INFINITY, l2 > 0.0f ? m2 : -INFINITY);
      const float f1 = lrow[i] > 0.0f ? __builtin_amdgcn_exp2f(mrow[i] - M) : 0.0f;
      const float f2 = l2 > 0.0f ? __builtin_amdgcn_exp2f(m2 - M) : 0.0f;
      lrow[i] = f1 * lrow[i] + f2 * l2;
      mrow[i] = M;
      const float g1 = __uint_as_float(swap32(f1).x), g2 = __uint_as_float(swap32(f2).x);
#pragma unroll
      for (int m = 0; m < CL / 2; ++m) {
        const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(st.acc[m][i]),
                                                        __float_as_uint(st.acc[m + CL / 2][i]), false, false);
        float z = g1 * __uint_as_float(p[0]) + g2 * __uint_as_float(p[1]);
        asm volatile("" : "+v"(z));  // merged here, not sunk past the barriers
        st.acc[m][i] = z;
      }
    }
  }
  // Each wave writes its merged rows into its own ring slot as soon as its
  // scan is done (its copies have all been waited for), so no barrier is
  // needed before the store and the merge work overlaps the other waves'
  // scans.  Row (wave, head) keeps channel c = CL ln + 4 k + t at position
  // (16 k + ln) 4 + t: every lane stores float4s and the 16 lanes of a row
  // store consecutive 16-byte words (no bank conflicts).  With the page-pair
  // layout the lanes l < 32 store k < CL / 8 and the lanes l + 32 the rest.
  float* mm = s_mlf[0];  // [G][NW]
  float* ml = s_mlf[1];  // [G][NW]
  {
    float* macc = reinterpret_cast<float*>(wring);  // [G][D]
    const int rg = pair ? (lg & 1) : lg;             // accumulator row group of this lane's values
    const int k0 = pair ? (lg >> 1) * (CL / 8) : 0;  // first float4 of the row this lane stores
    constexpr int NK = pair ? CL / 8 : CL / 4;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int head = head_of_col<G6>(4 * rg + i);
      if (head >= 0 && head < G) {
        float4* row = reinterpret_cast<float4*>(macc + head * D);
#pragma unroll
        for (int k = 0; k < NK; ++k)
          row[16 * (k0 + k) + ln] = make_float4(st.acc[4 * k][i], st.acc[4 * k + 1][i], st.acc[4 * k + 2][i],
                                                st.acc[4 * k + 3][i]);
        if (ln == 0 && lg == rg) {
          mm[head * NW + wid] = mrow[i];
          ml[head * NW + wid] = lrow[i];
        }
      }
    }
  }
  __syncthreads();  // every wave's rows and (m, l) are in LDS
  // Each thread folds the waves' rows of one head into four channels of the
  // partial, with the head's combine weights f_w = 2^(m_w - M) (M the largest
  // m_w of the rows with l_w > 0; rows with l_w = 0 take no part):
  // O_j = sum_w f_w O_w / L_j, L_j = sum_w f_w l_w.  Every thread of a head
  // computes the same weights, so no further barrier is needed.  Four
  // consecutive positions of a macc row are four consecutive channels.
  for (int it = tid; it < G * D / 4; it += NT) {
    const int n = it / (D / 4), pos = 4 * (it % (D / 4));
    const int c = CL * ((pos >> 2) & 15) + 4 * (pos >> 6);
    const float4* m4 = reinterpret_cast<const float4*>(mm + n * NW);
    const float4* l4 = reinterpret_cast<const float4*>(ml + n * NW);
    float mw[NW], lw[NW];
#pragma unroll
    for (int w4 = 0; w4 < NW / 4; ++w4) {
      const float4 a4 = m4[w4], b4 = l4[w4];
      mw[4 * w4] = a4.x, mw[4 * w4 + 1] = a4.y, mw[4 * w4 + 2] = a4.z, mw[4 * w4 + 3] = a4.w;
      lw[4 * w4] = b4.x, lw[4 * w4 + 1] = b4.y, lw[4 * w4 + 2] = b4.z, lw[4 * w4 + 3] = b4.w;
    }
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, lw[w] > 0.0f ? mw[w] : -INFINITY);
    float L = 0.0f;
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float f = lw[w] > 0.0f ? __builtin_amdgcn_exp2f(mw[w] - M) : 0.0f;
      const float4 x = *reinterpret_cast<const float4*>(ring + w * SLOTS * STAGE + (n * D + pos) * 4);
      L = fmaf(f, lw[w], L);
      o.x = fmaf(f, x.x, o.x);
      o.y = fmaf(f, x.y, o.y);
      o.z = fmaf(f, x.z, o.z);
      o.w = fmaf(f, x.w, o.w);
    }
    const float inv = L > 0.0f ? 1.0f / L : 0.0f;
    o.x *= inv;
    o.y *= inv;
    o.z *= inv;
    o.w *= inv;
    if (pos == 0) {
      part[G * D + n] = M;
      part[G * D + G + n] = (APP && s_app_bad) ? -1.0f : L;  // -1: the merge writes zeros
    }
    *reinterpret_cast<float4*>(part + n * D + c) = o;
  }
}

// Merge stage (Eq. softmax-merge): one single-wave workgroup per (query head
// of the group, KV head, request), one thread per four channels.  The O_j
// rows of up to 32 chunk slots and, in lane j, slot j's (m_j, l_j) are loaded
// together (one memory round trip for the usual grid); the batch maximum and
// the weights 2^(m_j - M) l_j come from wave reductions, and every weight is
// read into a scalar register, so each thread's fold is 32 FMAs per channel.
// Slots with l_j = 0 contribute nothing; a running (M, L, O) is rescaled once
// per batch.
// With the fused append (app_rec non-null) the workgroups of query head 0 and
// KV head 0 also publish their request's fresh page and, for request 0, the
// FP8 free-list top, from the records the scan left.
template <int D>
__global__ __launch_bounds__(D / 4) void decode_merge_kernel(int G, int H, int max_chunks,
                                                            const float* partials, float* out,
                                                            float* lse, const int32_t* app_rec,
                                                            int32_t* bt_w, uint8_t* tags_w,
                                                            int max_pages, const int32_t* seq_lens,
                                                            int32_t* ctrl, int32_t* rc8) {
  constexpr int B = 32;
  static_assert(D / 4 >= B && D / 4 <= 64, "one wave; lane j holds slot j's (m, l)");
  const int n = blockIdx.x, h = blockIdx.y, r = blockIdx.z, c4 = threadIdx.x;
  const int Hq = H * G;
  if (app_rec && n == 0 && h == 0 && c4 == 0) {
    const int id = app_rec[r];
    if (id >= 0) {
      const int64_t ix = (int64_t)r * max_pages + seq_lens[r] / PAGE;
      bt_w[ix] = id;
      tags_w[ix] = TAG_R;
      rc8[id] = 1;  // one request reference
    }
    if (r == 0 && app_rec[gridDim.z] >= 0) ctrl[CTRL_FP8_TOP] = app_rec[gridDim.z];
  }
  const int stride = part_stride(G, D);
  const float* base = partials + ((int64_t)r * H + h) * max_chunks * stride;
  float M = -INFINITY, L = 0.0f;
  float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
  bool poisoned = false;  // a slot with l < 0: a failed fused append, write zeros
  for (int k0 = 0; k0 < max_chunks; k0 += B) {
    float4 ok[B];
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const int k = min(k0 + j, max_chunks - 1);
      ok[j] = reinterpret_cast<const float4*>(base + (int64_t)k * stride + n * D)[c4];
    }
    const bool mine = c4 < B && k0 + c4 < max_chunks;
    const float* pk = base + (int64_t)min(k0 + c4, max_chunks - 1) * stride;
    const float mj = pk[G * D + n];
    const float lj = mine ? pk[G * D + G + n] : 0.0f;
    poisoned |= __any(lj < 0.0f);
    float mb = lj > 0.0f ? mj : -INFINITY;
#pragma unroll
    for (int o = 1; o < D / 4; o <<= 1) mb = fmaxf(mb, __shfl_xor(mb, o, D / 4));
    const float Mb = fmaxf(M, mb);
    if (Mb != -INFINITY) {  // else nothing in this batch, nothing before it (wave-uniform)
      const float f = M == -INFINITY ? 0.0f : exp2f(M - Mb);
      const float wj = lj > 0.0f ? exp2f(mj - Mb) * lj : 0.0f;
      float ws = wj;
#pragma unroll
      for (int o = 1; o < D / 4; o <<= 1) ws += __shfl_xor(ws, o, D / 4);
      L = L * f + ws;
      O.x *= f;
      O.y *= f;
      O.z *= f;
      O.w *= f;
#pragma unroll
      for (int j = 0; j < B; ++j) {
        const float w = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wj), j));
        // an empty slot's O rows were never written (they may hold any bits,
        // NaN included): skip the slot rather than multiply them by 0
        if (w != 0.0f) {
          O.x = fmaf(w, ok[j].x, O.x);
          O.y = fmaf(w, ok[j].y, O.y);
          O.z = fmaf(w, ok[j].z, O.z);
          O.w = fmaf(w, ok[j].w, O.w);
        }
      }
      M = Mb;
    }
  }
  const int64_t row = (int64_t)r * Hq + h * G + n;
  if (poisoned) L = 0.0f;
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  const float4 res = L > 0.0f ? make_float4(O.x * inv, O.y * inv, O.z * inv, O.w * inv)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
  reinterpret_cast<float4*>(out + row * D)[c4] = res;
  if (lse && c4 == 0) lse[row] = L > 0.0f ? (M + log2f(L)) * 0.69314718055994531f : -INFINITY;
}

// Device scratch for callers that cannot allocate (paged_attn_decode_noalloc):
// the split partials live in this fixed array instead of a caller workspace.
// Each device holds its own copy for the life of the process; host code
// never passes the array's name to a kernel (on the host it only names the
// symbol), it uses the device address resolved per device below.
static __device__ __align__(256) uint8_t scratch[MKV_DECODE_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[64];  // per device: the address of `scratch` on it
}  // namespace

hipError_t decode_scratch_init(int dev) {
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev]) return hipSuccess;
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  if (cur != dev) return hipErrorInvalidDevice;  // resolved only with the device current
  void* ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (!ptr) return hipErrorInvalidSymbol;
  g_scratch_ptr[dev] = ptr;
  return hipSuccess;
}

hipError_t decode_scratch(int dev, void** ptr) {
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (g_scratch_ptr[dev]) {
      *ptr = g_scratch_ptr[dev];
      return hipSuccess;
    }
  }
  hipError_t e = decode_scratch_init(dev);  // first call on a device the pool was not created on
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

// dynamic LDS a decode workgroup may use: 160 KiB per CU minus the static arrays
static constexpr size_t lds_limit() {
  // s_stage, s_mlf; s_next and slack
  return 160 * 1024 - sizeof(int4) * MAX_CHUNK_PAGES - 2 * 16 * NW_MAX * sizeof(float) - 256;
}

template <bool APP, bool SCORE = false>
static const void* decode_instance(int d, bool pair, bool g6) {
  if (d == 256)
    return g6 ? (const void*)decode_kernel<256, true, true, APP, SCORE>
                : pair ? (const void*)decode_kernel<256, true, false, APP, SCORE>
                       : (const void*)decode_kernel<256, false, false, APP, SCORE>;
  return g6 ? (const void*)decode_kernel<128, true, true, APP, SCORE>
              : pair ? (const void*)decode_kernel<128, true, false, APP, SCORE>
                     : (const void*)decode_kernel<128, false, false, APP, SCORE>;
}

hipError_t launch_decode(const PoolView& P, int layer, int n_req, const uint16_t* q,
                         const int32_t* bt, const uint8_t* tags, int max_pages,
                         const int32_t* seq_lens, float* out, float* lse, void* ws,
                         hipStream_t s, hipEvent_t* ev, const uint16_t* k_new,
                         const uint16_t* v_new, int32_t* bt_w, uint8_t* tags_w,
                         float2* page_mass) {
  const bool app = k_new != nullptr;
  const bool score = page_mass != nullptr;
  if (app && score) return hipErrorInvalidValue;
  const DecodeShape sh = decode_shape(n_req, max_pages, P.n_kv_heads, P.recent);
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
  a.partials = reinterpret_cast<float*>(ws);
  a.cunits = sh.cunits;
  a.max_chunks = sh.max_chunks;
  a.sm_log2 = 1.4426950408889634f / sqrtf((float)P.d);
  a.k_new = k_new;
  a.v_new = v_new;
  a.bt_w = bt_w;
  a.tags_w = tags_w;
  a.page_mass = page_mass;
  a.app_rec = app ? reinterpret_cast<int32_t*>(reinterpret_cast<uint8_t*>(ws) +
                                              decode_part_bytes(sh, n_req, P.n_kv_heads, P.group, P.d))
                  : nullptr;
  // dynamic LDS: three query operands, then the page ring (reused by the wave merge)
  const bool pair = P.group <= 8;
  const int nw = pair ? DecodeCfg<true>::NW : DecodeCfg<false>::NW;
  const int slots = pair ? DecodeCfg<true>::SLOTS : DecodeCfg<false>::SLOTS;
  const size_t qop_b = (size_t)QF8_TERMS * (P.d / 128) * 64 * 32 + (size_t)(P.d / 32) * 64 * 16;
  const size_t ring_b = (size_t)nw * slots * 2 * tq3_region_bytes(P.d);
  const size_t lds = qop_b + ring_b;  // the epilogue reuses each wave's ring slot
  if (lds > lds_limit()) return hipErrorInvalidValue;
  const bool g6 = pair && P.group <= 6;
  const void* kern = app     ? decode_instance<true>(P.d, pair, g6)
                     : score ? decode_instance<false, true>(P.d, pair, g6)
                             : decode_instance<false>(P.d, pair, g6);
  // the dynamic-LDS limit is raised once per kernel instance and device
  static std::atomic<uint32_t> attr_done[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint32_t bit = 1u << ((app ? 6 : score ? 12 : 0) + (P.d == 256 ? 3 : 0) + (g6 ? 2 : pair ? 1 : 0));
  if (dev < 0 || dev >= 64 || !(attr_done[dev].load() & bit)) {
    e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_limit());
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < 64) attr_done[dev].fetch_or(bit);
  }
  dim3 grid(sh.max_chunks, P.n_kv_heads, n_req);
  dim3 mgrid(P.group, P.n_kv_heads, n_req);
  // with timing on, the events track each kernel's own start and end (the
  // dispatch's timestamps, not markers around the launch)
  void* args[] = {&a};
  e = ev ? hipExtLaunchKernel(kern, grid, dim3(64 * nw), args, lds, s, ev[0], ev[1], 0)
         : hipLaunchKernel(kern, grid, dim3(64 * nw), args, lds, s);
  if (e != hipSuccess) return e;
  int G = P.group, H = P.n_kv_heads, mc = sh.max_chunks, mpg = max_pages;
  const float* pa = a.partials;
  const int32_t* rec = a.app_rec;
  int32_t* ctrl = P.ctrl;
  int32_t* rc8 = P.rc8;
  void* margs[] = {&G, &H, &mc, &pa, &out, &lse, &rec, &bt_w, &tags_w, &mpg, &seq_lens, &ctrl, &rc8};
  const void* mk = P.d == 256 ? (const void*)decode_merge_kernel<256> : (const void*)decode_merge_kernel<128>;
  const dim3 mblock(P.d / 4);
  return ev ? hipExtLaunchKernel(mk, mgrid, mblock, margs, 0, s, ev[2], ev[3], 0)
            : hipLaunchKernel(mk, mgrid, mblock, margs, 0, s);
}

// Attention-score collector (Sec. 3.1, Eqs. score-global-weight and
// attention-score), after a scoring decode of the same call; workgroups over
// blocks of pages and requests.  The globally normalized mass of page p for
// query head hq is its local mass rescaled by the global softmax
// normalization, q = mass * 2^(m_ref - lse / ln 2) (lse of the merge).  The
// collector conditions on page-addressable mass, q / sum_p q; this attention
// has no sink logit and the merge's lse is the log of the very sum of weights
// that the page masses partition, so sum_p q = 1 and q~ = q up to rounding.
// r_p = the mean of q~ over the sampled heads; a_p <- beta a_p + (1 - beta)
// r_p; q~ is written when asked.
// Every load goes out at the start (the length, the block's page masses --
// consecutive terms to consecutive threads, four per thread -- the scores,
// lse and the head mask): one memory round trip.  Each page's sum over the
// sampled heads runs in head order from LDS.
constexpr int SCORE_UP_NT = 256;  // threads per update workgroup
constexpr int SCORE_UP_EPT = 4;   // (page, head) terms per thread
__global__ __launch_bounds__(SCORE_UP_NT) void score_update_kernel(int n_q_heads, int max_pages, int ppb,
                                                                   const int32_t* seq_lens,
                                                                   const float* lse,
                                                                   const float2* page_mass,
                                                                   const uint8_t* head_mask,
                                                                   float beta, float* a_io,
                                                                   float* r_out, float* qn_out) {
  constexpr int MAXH = 256;
  __shared__ float s_l2[MAXH];
  __shared__ bool s_smp[MAXH];
  __shared__ float s_q[SCORE_UP_NT * SCORE_UP_EPT];
  __shared__ int s_ns;
  const int r = blockIdx.y, tid = threadIdx.x;
  const int p0 = blockIdx.x * ppb;
  const int npb = min(ppb, max_pages - p0);  // pages of this block inside the table
  const int64_t e0 = ((int64_t)r * max_pages + p0) * n_q_heads;  // the block's first (page, head) term
  const int ne = npb * n_q_heads;  // at most SCORE_UP_NT * SCORE_UP_EPT
  const int S = seq_lens[r];
  float2 mm[SCORE_UP_EPT];
#pragma unroll
  for (int k = 0; k < SCORE_UP_EPT; ++k) {
    const int e = tid + k * SCORE_UP_NT;
    mm[k] = e < ne ? page_mass[e0 + e] : make_float2(0.0f, 0.0f);
  }
  float a_old = 0.0f;
  if (tid < npb) a_old = a_io[(int64_t)r * max_pages + p0 + tid];
  if (tid == 0) s_ns = 0;
  __syncthreads();
  for (int hq = tid; hq < n_q_heads; hq += SCORE_UP_NT) {
    s_l2[hq] = lse[(int64_t)r * n_q_heads + hq] * 1.4426950408889634f;
    s_smp[hq] = head_mask[hq] != 0;
    if (s_smp[hq]) atomicAdd(&s_ns, 1);
  }
  __syncthreads();
  const int np = S >= 1 ? min((S + PAGE - 1) / PAGE, max_pages) : 0;
#pragma unroll
  for (int k = 0; k < SCORE_UP_EPT; ++k) {
    const int e = tid + k * SCORE_UP_NT;
    if (e >= ne) break;
    const int pl = e / n_q_heads, hq = e - pl * n_q_heads;
    const float qn = mm[k].x * exp2f(mm[k].y - s_l2[hq]);
    const bool live = p0 + pl < np;  // masses past the request's end were never written
    if (qn_out && live) qn_out[e0 + e] = qn;
    s_q[e] = (live && s_smp[hq]) ? qn : 0.0f;
  }
  __syncthreads();
  if (tid >= npb || p0 + tid >= np) return;
  float acc = 0.0f;
  for (int hq = 0; hq < n_q_heads; ++hq) acc += s_q[tid * n_q_heads + hq];
  const int ns = s_ns;
  const float rp = ns ? acc / (float)ns : 0.0f;
  const int64_t pi = (int64_t)r * max_pages + p0 + tid;
  if (r_out) r_out[pi] = rp;
  a_io[pi] = beta * a_old + (1.0f - beta) * rp;
}

hipError_t launch_score_collect(int n_req, int n_q_heads, int max_pages, const int32_t* seq_lens,
                                const float* lse, const float2* page_mass,
                                const uint8_t* head_mask, float beta, float* a_io, float* r_out,
                                float* qn_out, hipStream_t s) {
  if (n_q_heads < 1 || n_q_heads > 256) return hipErrorInvalidValue;
  // pages per workgroup: every thread stages at most SCORE_UP_EPT terms
  const int ppb = max(1, min(SCORE_UP_NT, SCORE_UP_NT * SCORE_UP_EPT / n_q_heads));
  hipLaunchKernelGGL(score_update_kernel, dim3((max_pages + ppb - 1) / ppb, n_req), dim3(SCORE_UP_NT), 0, s,
                     n_q_heads, max_pages, ppb, seq_lens, lse, page_mass, head_mask, beta, a_io, r_out,
                     qn_out);
  return hipGetLastError();
}

}  // namespace mkv
