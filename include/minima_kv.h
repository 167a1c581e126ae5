/*
 * minima_kv.h — C ABI of the MI355X (gfx950) Minima-KV hot path.
 *
 * Minima-KV (arXiv 2608.23834) keeps every logical KV page of a live request
 * in one of two physical formats: FP8 for Recent and Anchor pages and a 3-bit
 * rotated, norm-corrected format ("TQ3") for Stale pages (Sec. 3.1).  Decode
 * attention reads both formats, dequantizes in registers and merges all
 * partial results under one softmax (Sec. 3.3, Eq. softmax-merge), with no
 * cache-sized dense copy (Sec. 4.1).
 *
 * Conventions shared by every call
 *  - All pointers marked "device" are device memory owned by the caller; the
 *    library never allocates device memory that grows with the number of
 *    tokens.  Pointers marked "host" are read during the call only.
 *  - Work is enqueued on the caller's HIP stream and the call returns without
 *    waiting; results are ordered by stream order (the copy-before-publish and
 *    release-after-readers rules of Alg. 1 follow from it on one stream).
 *  - Page size is 16 tokens.  head_dim is 128 or 256.  Query head hq uses KV
 *    head hq / (n_q_heads / n_kv_heads).
 *  - Block table: int32 [n_req][max_pages], entry = physical page id in the
 *    pool named by the tag, -1 = unmapped.  It is shared by all layers (Sec.
 *    4.1: entries are logical blocks, not layers or K/V roles).
 *  - Tags: uint8 [n_req][max_pages]: 0 = Recent (FP8), 1 = Anchor (FP8),
 *    2 = Stale (TQ3), 0xFF = unmapped (Sec. 3.1 tiers z in {R, A, S}).
 *  - bf16 tensors are passed as raw 16-bit patterns (uint16_t).
 *  - Every call checks its host-visible arguments before enqueuing anything,
 *    so a call that returns an error has changed nothing.  Conditions that only
 *    the device can see (a free list running dry, a page in the wrong state)
 *    make the kernels skip all writes of that call and set a bit of the pool's
 *    device error word, read with kv_pool_check_errors().
 */
#ifndef MINIMA_KV_H
#define MINIMA_KV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MKV_OK = 0,
  MKV_EINVAL = 1, /* bad argument (null pointer, negative size, bad geometry) */
  MKV_EUNSUP = 2, /* head_dim, page size or GQA group not compiled */
  MKV_ENOMEM = 3, /* a caller buffer is smaller than the call needs */
  MKV_ERANGE = 4, /* an index or length is out of range */
  MKV_ESTATE = 5, /* the pool is in a state that does not allow the call */
  MKV_EHIP = 6    /* a HIP runtime call or kernel launch failed */
} mkv_status;

/* Device error word bits (sticky until cleared). */
#define MKV_DEVERR_FP8_EXHAUSTED 0x1u /* append: FP8 free list too short */
#define MKV_DEVERR_TQ3_EXHAUSTED 0x2u /* migrate: TQ3 free list too short */
#define MKV_DEVERR_NOT_RECENT 0x4u    /* append: tokens land in a mapped non-Recent page */
#define MKV_DEVERR_RANGE 0x8u         /* a sequence length or page index is out of range */
#define MKV_DEVERR_BAD_TAG 0x10u      /* attention found an unmapped page below seq_len */
#define MKV_DEVERR_REFCOUNT 0x20u     /* acquire of a free page, release beyond its references */

#define MKV_PAGE_SIZE 16
#define MKV_ALL_LAYERS (-1)

typedef struct mkv_pool mkv_pool; /* opaque host handle */

/* Pool geometry and caller-owned storage.  Sizes of the four device buffers
 * come from kv_pool_bytes(). */
typedef struct mkv_pool_desc {
  int32_t n_layers;      /* full-attention layers held by the pool */
  int32_t n_q_heads;     /* query heads; a multiple of n_kv_heads, group <= 16 */
  int32_t n_kv_heads;
  int32_t head_dim;      /* 128 or 256 */
  int32_t page_size;     /* must be 16 */
  int32_t n_fp8_pages;   /* physical FP8 pages (each holds all layers and heads) */
  int32_t n_tq3_pages;   /* physical TQ3 pages */
  int32_t recent_tokens; /* Recent window W >= 1 (Sec. 3.1) */
  const int8_t* rot_signs;  /* host [head_dim], each +1 or -1: R = d^-1/2 H diag(s) */
  const int32_t* fp8_order; /* host [n_fp8_pages] permutation: order in which FP8
                               ids are handed out; NULL = 0, 1, 2, ... */
  const int32_t* tq3_order; /* host [n_tq3_pages] permutation or NULL */
  void* fp8_data;        /* device: [n_layers][n_fp8_pages][n_kv_heads][2*16*d] bytes */
  size_t fp8_data_bytes;
  void* fp8_scales;      /* device: fp32 [n_layers][n_fp8_pages][n_kv_heads][2] (K, V) */
  size_t fp8_scales_bytes;
  void* tq3_data;        /* device: [n_layers][n_tq3_pages][n_kv_heads][16*d+32] bytes */
  size_t tq3_data_bytes;
  void* ctrl;            /* device: free lists, counters, work lists, error word */
  size_t ctrl_bytes;
} mkv_pool_desc;

/* Cheap instrumentation (Sec. 3.3 / Sec. 6.3 route, fallback and dense-shadow
 * counters).  This library has no fallback path and never builds a dense
 * shadow, so those two counters are always zero. */
typedef struct mkv_counters {
  uint64_t decode_routes;     /* paged_attn_decode layer calls served */
  uint64_t chunk_routes;      /* paged_attn_chunk layer calls served */
  uint64_t fallbacks;         /* always 0 */
  uint64_t dense_shadow_bytes;/* always 0 */
  uint64_t fp8_pages_live;    /* FP8 pages currently allocated (synchronizes) */
  uint64_t tq3_pages_live;    /* TQ3 pages currently allocated (synchronizes) */
  uint64_t fp8_bytes_live;    /* physical bytes of live FP8 pages, all layers */
  uint64_t tq3_bytes_live;    /* physical bytes of live TQ3 pages, all layers */
} mkv_counters;

/* Byte sizes of the four caller-owned device buffers for a geometry.
 * Only the geometry fields of desc are read.  Returns MKV_EUNSUP for an
 * uncompiled head_dim/page size/group, MKV_EINVAL for non-positive sizes. */
mkv_status kv_pool_bytes(const mkv_pool_desc* desc, size_t* fp8_data_bytes,
                         size_t* fp8_scales_bytes, size_t* tq3_data_bytes, size_t* ctrl_bytes);

/* Create a pool over caller-owned buffers (Sec. 4.4: separate per-format pools
 * with per-kind free lists).  Initialises the free lists and error word in
 * ctrl synchronously; pool contents are left as they are.  The handle owns
 * only host metadata.  Errors: EINVAL, EUNSUP, ENOMEM (a buffer smaller than
 * kv_pool_bytes() reports), EHIP. */
mkv_status kv_pool_create(const mkv_pool_desc* desc, mkv_pool** out);
mkv_status kv_pool_destroy(mkv_pool* pool);

/* Append(q, p) of Alg. 1 / Recent tier of Sec. 3.1: quantize new bf16 K/V to
 * FP8 E4M3 (round to nearest even, saturating at 448) with one fp32 scale per
 * (layer, page, KV head, K or V), s = amax / 448.
 *  - Request r receives tokens at positions seq_lens_before[r] ..
 *    seq_lens_before[r] + n_r - 1, n_r = cu_new_tokens[r+1] - cu_new_tokens[r];
 *    its rows in k/v are cu_new_tokens[r] .. cu_new_tokens[r+1]-1.
 *  - Every logical page that receives tokens and is unmapped gets a new FP8 id
 *    from the free list (ascending (request, page) order) and tag Recent; the
 *    mapping is written to block_table/tags in place.  A mapped page must be
 *    Recent; a partly filled page keeps its scale unless the new tokens exceed
 *    448 * scale, in which case its scale grows and earlier codes are
 *    re-rounded; unused slots of a new page are zero.
 *  - layer = MKV_ALL_LAYERS writes every layer and k/v are
 *    [n_layers][n_new_total][n_kv_heads][head_dim]; else only that layer and
 *    k/v are [n_new_total][n_kv_heads][head_dim].
 *  - seq_lens_before, cu_new_tokens ([n_req+1], cu[0] = 0, cu[n_req] =
 *    n_new_total) are device int32.  seq_lens are not updated.
 * Device-side failures (free list too short, page not Recent, page index
 * beyond max_pages) set the error word and leave everything unchanged. */
mkv_status kv_append_fp8(mkv_pool* pool, int32_t layer, int32_t n_req, int32_t* block_table,
                         uint8_t* tags, int32_t max_pages, const int32_t* seq_lens_before,
                         const int32_t* cu_new_tokens, int32_t n_new_total, const uint16_t* k,
                         const uint16_t* v, hipStream_t stream);

/* Retier(p, TQ3) of Alg. 1 for every page that has left the Recent window
 * (Sec. 3.1): page p of request r is Recent while (p+1)*16 > seq_len - W.  A
 * Recent page outside the window becomes Anchor (tag only, stays FP8) when
 * anchor_mask[r][p] != 0, else it is encoded FP8 -> TQ3 for all layers and
 * heads ("normalize-rotate-pack", Sec. 4.3) into a newly allocated TQ3 page;
 * only then are (tag Stale, new id) published and the FP8 page released to its
 * free list (Alg. 1 copy-before-publish).  TQ3 ids are handed out and FP8 ids
 * released in ascending (request, page) order.  anchor_mask: device uint8
 * [n_req][max_pages] or NULL; seq_lens: device int32 [n_req].  If the TQ3 free
 * list is too short nothing changes and the error word is set. */
mkv_status kv_migrate_to_tq3(mkv_pool* pool, int32_t n_req, int32_t* block_table, uint8_t* tags,
                             int32_t max_pages, const uint8_t* anchor_mask,
                             const int32_t* seq_lens, hipStream_t stream);

/* Promote(p) of Alg. 1: a Stale page that re-enters the protected budget is
 * materialized back into FP8 (Sec. 3.1 Anchor paragraph).  Every page of
 * request r with tag Stale, promote_mask[r][p] != 0 and p < ceil(seq_lens[r]
 * / 16) is reconstructed for all layers and KV heads -- keys k_c =
 * fp32(gamma * sigma_c * (H mu_code)_c / sqrt(d)), values v_c = fp32(zero_c +
 * scale_c * code), the reconstruction the decode attends to -- and quantized
 * into a newly allocated FP8 page with the rule of a fresh page (s = amax /
 * 448 per page-head and K/V, code = E4M3(x / s)); only then is (tag Anchor,
 * new id) published and the TQ3 page released to its free list (Alg. 1
 * copy-before-publish).  FP8 ids are taken and TQ3 ids released in ascending
 * (request, page) order.  Other pages are left alone.  promote_mask: device
 * uint8 [n_req][max_pages]; seq_lens: device int32 [n_req].  If the FP8 free
 * list is too short, a length is out of range or a Stale page's id is out of
 * range, nothing changes and the error word is set. */
mkv_status kv_promote_to_fp8(mkv_pool* pool, int32_t n_req, int32_t* block_table, uint8_t* tags,
                             int32_t max_pages, const uint8_t* promote_mask,
                             const int32_t* seq_lens, hipStream_t stream);

/* Reference-counted pages and shared prefixes (Alg. 1 SealPrefix and Finish;
 * Sec. 4.4 prefix reuse).  Every mapped page carries a count of the
 * references to it: block-table entries of live requests plus prefix-cache
 * references.  A page appended, migrated or promoted into has one reference
 * (its request's).  A page with more than one reference is shared and
 * immutable: kv_migrate_to_tq3 and kv_promote_to_fp8 leave it as it is (no
 * re-encoding, no retag to Stale) until it is private again; decode reads it
 * in place from every table that maps it.  Only full pages may be shared (the
 * tail page a request still appends to must stay private).
 *  - kv_pages_acquire: one more reference per listed page -- SealPrefix (the
 *    cache's reference on a request's full pages) and attaching a cached
 *    prefix to a new request (the caller writes the (id, tag) entries into
 *    the request's block table, then acquires them).  ids: device int32 [n];
 *    tags: device uint8 [n] (R or A: FP8 pool, S: TQ3 pool).  Every listed
 *    page must be live; otherwise nothing changes and MKV_DEVERR_REFCOUNT is
 *    set.
 *  - kv_pages_release: one reference fewer per listed entry (prefix
 *    eviction); a page whose count reaches zero returns to its free list, at
 *    its last entry, pushes in entry order.  A page listed more often than it
 *    has references, a bad tag or id: nothing changes, MKV_DEVERR_REFCOUNT.
 *  - kv_request_finish: Finish(q) of the requests reqs (device int32
 *    [n_fin], ascending, each < n_req): the mapped entries of their rows are
 *    released as by kv_pages_release in ascending (request, page) order,
 *    then the rows are unmapped (id -1, tag 0xFF).
 *  - kv_pool_read_refcounts: the counts (host int32 [n_fp8_pages] and
 *    [n_tq3_pages], either may be NULL); synchronizes. */
mkv_status kv_pages_acquire(mkv_pool* pool, int32_t n, const int32_t* ids, const uint8_t* tags,
                            hipStream_t stream);
mkv_status kv_pages_release(mkv_pool* pool, int32_t n, const int32_t* ids, const uint8_t* tags,
                            hipStream_t stream);
mkv_status kv_request_finish(mkv_pool* pool, int32_t n_fin, const int32_t* reqs, int32_t n_req,
                             int32_t* block_table, uint8_t* tags, int32_t max_pages,
                             hipStream_t stream);
mkv_status kv_pool_read_refcounts(mkv_pool* pool, int32_t* rc_fp8, int32_t* rc_tq3);

/* Workspace bytes for paged_attn_decode and paged_attn_decode_append
 * (n_q_total = 0; the split partials, then n_req + 1 words the fused append
 * leaves for its merge kernel to publish) or paged_attn_chunk (n_q_total =
 * total chunk queries) at this batch shape. */
mkv_status paged_attn_workspace_bytes(const mkv_pool* pool, int32_t n_req, int32_t max_pages,
                                      int32_t n_q_total, size_t* bytes);

/* Zero a workspace (optional: the attention calls write every workspace word
 * they read, so a workspace needs no initialisation). */
mkv_status paged_attn_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream);

/* Mixed-format decode attention (Sec. 3.3; Sec. 4.1 direct fused decode).
 * The query of request r sits at position seq_lens[r]-1 and attends to every
 * logical token t < seq_lens[r] (1 <= seq_lens[r] <= 16*max_pages), read from
 * its FP8 (Recent/Anchor) and TQ3 (Stale) pages:
 *     out[r][hq] = sum_t softmax_t(q . k_hat_t / sqrt(d)) v_hat_t,
 * k_hat/v_hat being the pages' dequantized values.  Each split of either format
 * produces (m_j, l_j, normalized O_j); all splits are merged by Eq.
 * (softmax-merge).  q: device bf16 [n_req][n_q_heads][d]; out: device fp32
 * [n_req][n_q_heads][d]; lse: device fp32 [n_req][n_q_heads] (natural log of
 * the softmax denominator, scores in units of q.k/sqrt(d)) or NULL.
 * ws: device, >= paged_attn_workspace_bytes(pool, n_req, max_pages, 0); it
 * holds the split partials (O(splits x heads x d) floats).  q, out and ws must
 * be 16-byte aligned (MKV_EINVAL otherwise).  max_pages is at most 262144.  An
 * invalid seq_len sets the error word and gives that request zero outputs; a
 * page below seq_len with an invalid tag or an out-of-range physical id sets
 * the error word and is left out of the softmax.  The waves of a split claim
 * its pages at run time, so the fp32 summation order (and the last bits of
 * out and lse) can differ from call to call. */
mkv_status paged_attn_decode(mkv_pool* pool, int32_t layer, int32_t n_req, const uint16_t* q,
                             const int32_t* block_table, const uint8_t* tags, int32_t max_pages,
                             const int32_t* seq_lens, float* out, float* lse, void* ws,
                             size_t ws_bytes, hipStream_t stream);

/* Decode step with its append fused in (Alg. 1 Append, then the decode above):
 * appends one new token per request to `layer` -- K and V rows k_new, v_new:
 * device bf16 [n_req][n_kv_heads][d], 8-byte aligned -- at position
 * seq_lens_before[r] (opening a fresh FP8 page, popped from the FP8 free list
 * in request order, where the block-table entry of the position's page is
 * negative, as kv_append_fp8 does), then runs the decode
 * attention of paged_attn_decode over seq_lens_before[r] + 1 tokens.  The
 * pool state, block table and tags afterwards, and the outputs, equal those
 * of kv_append_fp8 (one token per request) followed by paged_attn_decode,
 * up to the fp32 summation order of the outputs.  block_table and tags are
 * written (fresh pages).  Same buffer rules as paged_attn_decode.  An append
 * that cannot be done as a whole (a length outside [0, 16*max_pages), a
 * page being appended to that is not Recent or has an out-of-range id, an
 * exhausted FP8 free list) sets the error word, changes no state and gives
 * every request of the call zero outputs. */
mkv_status paged_attn_decode_append(mkv_pool* pool, int32_t layer, int32_t n_req,
                                    const uint16_t* q, const uint16_t* k_new,
                                    const uint16_t* v_new, int32_t* block_table, uint8_t* tags,
                                    int32_t max_pages, const int32_t* seq_lens_before,
                                    float* out, float* lse, void* ws, size_t ws_bytes,
                                    hipStream_t stream);

/* paged_attn_decode for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same attention, with the split partials held in a fixed
 * device array of the library (MKV_DECODE_SCRATCH_BYTES per device, resolved
 * when a pool is created on that device or at the first call there) instead
 * of a caller workspace.  The call allocates nothing.  Returns MKV_ENOMEM
 * when the partials of this shape, paged_attn_workspace_bytes(pool, n_req,
 * max_pages, 0), exceed MKV_DECODE_SCRATCH_BYTES; other arguments and errors
 * as paged_attn_decode.  Every call on a device shares that device's array:
 * calls that overlap in time on one device (different streams, or processes
 * sharing nothing else) race on it and must be serialized by the caller. */
#define MKV_DECODE_SCRATCH_BYTES (32u * 1024u * 1024u)
mkv_status paged_attn_decode_noalloc(mkv_pool* pool, int32_t layer, int32_t n_req,
                                     const uint16_t* q, const int32_t* block_table,
                                     const uint8_t* tags, int32_t max_pages,
                                     const int32_t* seq_lens, float* out, float* lse,
                                     hipStream_t stream);

/* Causal chunked-prefill attention over the same mixed pages.  Request r has
 * n_r = cu_q[r+1]-cu_q[r] queries; query i sits at position
 * seq_lens[r] - n_r + i and attends to keys t <= that position (the chunk's
 * own KV must already be appended as FP8).  q: device bf16
 * [n_q_total][n_q_heads][d]; cu_q: device int32 [n_req+1]; out: device fp32
 * [n_q_total][n_q_heads][d]; ws >= paged_attn_workspace_bytes(..., n_q_total)
 * (it holds the compact per-format page lists).  q, out and ws must be
 * 16-byte aligned (MKV_EINVAL otherwise).  A request whose query range or
 * length is invalid sets the error word and its locatable rows get zeros.
 * Query ranges are expected not to overlap (cu_q nondecreasing); ranges that
 * overlap so much that their 128-row blocks (ceil(n_r * group / 128) per
 * request) exceed ceil(n_q_total * group / 128) + n_req set the error word
 * and the call writes nothing to out.
 * (The paper runs prefill on a generic dense path, Sec. 4.1; this variant
 * keeps the mixed pages and uses MFMA for the dense contraction.) */
mkv_status paged_attn_chunk(mkv_pool* pool, int32_t layer, int32_t n_req, const uint16_t* q,
                            const int32_t* cu_q, int32_t n_q_total, const int32_t* block_table,
                            const uint8_t* tags, int32_t max_pages, const int32_t* seq_lens,
                            float* out, void* ws, size_t ws_bytes, hipStream_t stream);

/* Direct mixed-format attention-score collector (Sec. 3.1, Eqs.
 * score-partial, score-global-weight and attention-score; Sec. 4.2: each
 * split's local page mass is rescaled by its global softmax weight).
 * paged_attn_decode_scores is paged_attn_decode (same arguments and outputs;
 * lse is required) that also writes, for every logical page p <
 * ceil(seq_lens[r] / 16) and query head hq, the page's local softmax mass and
 * the reference exponent it was taken against:
 *   page_mass[r][p][hq] = (sum_{i in p} 2^(s_i - m), m)  (fp32 pairs; s_i =
 *   q.k_i log2(e) / sqrt(d), m the running maximum of the split that read the
 *   page), other entries untouched.  page_mass: device float [n_req][max_pages]
 *   [n_q_heads][2], 8-byte aligned.
 * kv_page_scores_update then, for every request r and page p < ceil(seq_lens
 * [r] / 16), forms the globally normalized mass q_{hq,p} = mass * 2^(m - lse
 * [r][hq] / ln 2) (Eq. score-global-weight), conditions it on page-addressable
 * mass, q~ = q / sum_p q (= q: with no sink logit every token's weight is
 * page mass, and the merge's lse is the log of the sum the masses partition,
 * so sum_p q = 1 up to rounding), averages q~ over the sampled heads (head_mask
 * [hq] != 0; device uint8 [n_q_heads]) into r_p, and updates scores[r][p] =
 * beta * scores[r][p] + (1 - beta) * r_p in place (Eq. attention-score;
 * device fp32 [n_req][max_pages]); r_out (same shape) and qn_out ([n_req]
 * [max_pages][n_q_heads]) receive r and q~ when non-null.  seq_lens, lse
 * and page_mass are those of the scoring decode; n_q_heads <= 256. */
mkv_status paged_attn_decode_scores(mkv_pool* pool, int32_t layer, int32_t n_req,
                                    const uint16_t* q, const int32_t* block_table,
                                    const uint8_t* tags, int32_t max_pages,
                                    const int32_t* seq_lens, float* out, float* lse, void* ws,
                                    size_t ws_bytes, float* page_mass, hipStream_t stream);
mkv_status kv_page_scores_update(const mkv_pool* pool, int32_t n_req, int32_t max_pages,
                                 const int32_t* seq_lens, const float* lse,
                                 const float* page_mass, const uint8_t* head_mask, float beta,
                                 float* scores, float* r_out, float* qn_out, hipStream_t stream);

/* Graph eligibility of a decode step (Sec. 4.1: the graph path is gated on a
 * homogeneous physical-cache cohort; other shapes, prefill or an
 * inconsistent cache state fail closed to the generic path).  A decode step
 * of this library -- paged_attn_decode or paged_attn_decode_append per layer,
 * then kv_migrate_to_tq3 -- launches a fixed set of kernels whose grids and
 * arguments depend only on the pool, n_req and max_pages; everything else it
 * reads (queries, block table, tags, lengths) is read from device memory at
 * run time, and it enqueues no memset and no host synchronization, so a step
 * captured into a HIP graph replays correctly for any contents of the same
 * buffers.  This returns a 64-bit key of everything such a capture bakes in:
 * the pool (identity and geometry, page size, Recent window), n_req,
 * max_pages, the split shape, the decode kernel instance (fused append or
 * not) and the scoring flag (0: no attention scores; scoring runs another
 * instance).  A caller replays a captured step only while the key it computes
 * for the next step equals the captured one and the same device buffers are
 * used, and launches the calls directly otherwise.  Errors: EINVAL;
 * ESTATE when the pool is not a compressed cohort (no TQ3 pool) or kernel
 * timing is on (its events are host objects, not graph nodes). */
mkv_status paged_attn_decode_cohort_key(const mkv_pool* pool, int32_t n_req, int32_t max_pages,
                                        int32_t fused_append, int32_t scoring, uint64_t* key);

/* Compact per-format page lists (Sec. 4.1): the stable partition of logical
 * pages [0, ceil(seq_len/16)) into FP8 (tags R, A) and TQ3 (tag S), logical
 * order kept.  list8/list3: device int32 [n_req][max_pages][2] =
 * (logical page, physical id); counts: device int32 [n_req][2] = (n_fp8,
 * n_tq3).  Entries past the counts are left untouched. */
mkv_status kv_partition_pages(int32_t n_req, const int32_t* block_table, const uint8_t* tags,
                              int32_t max_pages, const int32_t* seq_lens, int32_t* list8,
                              int32_t* list3, int32_t* counts, hipStream_t stream);

/* Free-list state (synchronizes with the device). */
mkv_status kv_pool_free_counts(mkv_pool* pool, int32_t* n_fp8_free, int32_t* n_tq3_free);

/* Copy the free stacks to host memory (synchronizes): ids in [0, top) from the
 * bottom; the next id handed out is the last one. */
mkv_status kv_pool_read_free_lists(mkv_pool* pool, int32_t* fp8_ids, int32_t* n_fp8,
                                   int32_t* tq3_ids, int32_t* n_tq3);

/* Route / fallback / dense-shadow / physical-byte counters (synchronizes). */
mkv_status kv_pool_counters(mkv_pool* pool, mkv_counters* out);

/* Deterministic decode: with enable != 0, paged_attn_decode, its fused-append
 * and scoring forms and paged_attn_decode_noalloc on this pool give every
 * wave of a split a fixed list of stages (wave w: stages w, w + NW, ...)
 * instead of claiming them at run time, so out and lse are bit-identical from
 * call to call for the same inputs (otherwise they can differ in the last
 * bits, by fp32 summation order).  Off by default: the fixed schedule balances
 * the waves of a SIMD less well.  Takes effect for calls enqueued after it;
 * part of the cohort key. */
mkv_status paged_attn_set_deterministic(mkv_pool* pool, int32_t enable);

/* Kernel timing for measurement tools; correct use never needs it.  When
 * enabled, each paged_attn_decode or paged_attn_decode_append call on this
 * pool launches its split-scan and merge kernels with HIP events that track
 * each kernel's own start and end on its stream (hipExtLaunchKernel).
 * paged_attn_last_times waits for the last call's events and returns the
 * durations of the scan and of the merge in microseconds (MKV_ESTATE when
 * timing is off or no call was timed).  Enabling creates the events on the
 * current device; the pool owns them. */
mkv_status paged_attn_set_timing(mkv_pool* pool, int32_t enable);
mkv_status paged_attn_last_times(mkv_pool* pool, float* scan_us, float* merge_us);

/* Streaming-read probe for measurement tools; correct use never needs it.
 * Reads bytes (a multiple of 16; buf 16-byte aligned, device memory) once with
 * 16-byte loads and writes one word per workgroup to sink, which must hold
 * MKV_STREAM_PROBE_WORKGROUPS uint32 values (device memory).  The words fold
 * the data together and have no other meaning: the call exists to time a
 * kernel that reads a buffer once, the bandwidth ceiling of the decode scan.
 * Enqueued on stream; MKV_EINVAL on a null pointer, misalignment or a size
 * that is not a multiple of 16. */
#define MKV_STREAM_PROBE_WORKGROUPS 2048
mkv_status mkv_stream_read(const void* buf, size_t bytes, uint32_t* sink, hipStream_t stream);

/* Dense bf16 control for measurement tools; correct use never needs it.  The
 * fused-decode canary of Sec. 6.3 times the mixed-format route against a
 * dense control on the same KV; these calls hold that KV as bf16 pages and
 * attend to it with a plain paged decode kernel, so the mixed path can be
 * timed against an uncompressed cache of the same shape.
 *  - pages: device, bf16 bits [n_layers][n_pages][n_kv_heads][2*16*head_dim]
 *    (MKV_CONTROL_BF16_PAGE_HEAD_BYTES(head_dim) bytes per page-head: K
 *    token-major, then V in 4-token groups per channel), 16-byte aligned.
 *  - block_table: device int32 [n_req][max_pages] of page ids chosen by the
 *    caller (no allocator, no tags: every page is bf16).
 * mkv_control_bf16_write copies new rows of one layer (k, v: device bf16
 * [n_new_total][n_kv_heads][head_dim]; request r's rows cu_new_tokens[r] ..
 * cu_new_tokens[r+1]-1 land at positions seq_lens_before[r] ..) into their
 * pages; rows whose page is unmapped are skipped.  mkv_control_bf16_decode
 * computes out[r][hq] = sum_t softmax_t(q . k_t / sqrt(d)) v_t over t <
 * seq_lens[r] (fp32 accumulate, lse as in paged_attn_decode), with ws of at
 * least mkv_control_bf16_workspace_bytes().  Both enqueue on stream;
 * EINVAL/EUNSUP/ERANGE/ENOMEM on bad arguments as the calls above. */
#define MKV_CONTROL_BF16_PAGE_HEAD_BYTES(d) ((size_t)4 * 16 * (size_t)(d))
mkv_status mkv_control_bf16_write(uint16_t* pages, int32_t n_pages, int32_t n_layers,
                                  int32_t n_kv_heads, int32_t head_dim, int32_t layer,
                                  int32_t n_req, const int32_t* block_table, int32_t max_pages,
                                  const int32_t* seq_lens_before, const int32_t* cu_new_tokens,
                                  int32_t n_new_total, const uint16_t* k, const uint16_t* v,
                                  hipStream_t stream);
mkv_status mkv_control_bf16_workspace_bytes(int32_t n_req, int32_t max_pages, int32_t n_kv_heads,
                                            int32_t n_q_heads, int32_t head_dim, size_t* bytes);
mkv_status mkv_control_bf16_decode(const uint16_t* pages, int32_t n_pages, int32_t n_layers,
                                   int32_t n_kv_heads, int32_t n_q_heads, int32_t head_dim,
                                   int32_t layer, int32_t n_req, const uint16_t* q,
                                   const int32_t* block_table, int32_t max_pages,
                                   const int32_t* seq_lens, float* out, float* lse, void* ws,
                                   size_t ws_bytes, hipStream_t stream);

/* Arithmetic conformance probe for tests; correct use never needs it.  The
 * bit-exact TQ3 metadata (gamma, V scale and zero; Sec. 4.1 FP16 key-norm
 * correction and scale/zero) relies on the device's fp64 division and square
 * root being correctly rounded and on the library's fp64 -> binary16
 * rounding (nearest-even, saturating at 65504).  This runs exactly that
 * compiled code: quot[i] = a[i] / b[i], root[i] = sqrt(a[i]), half[i] =
 * binary16(a[i]) for i < n.  All five arrays are device memory (8-byte
 * aligned; half 2-byte aligned).  Enqueued on stream; MKV_EINVAL on a null
 * pointer or n < 0. */
mkv_status mkv_fp64_probe(const double* a, const double* b, int64_t n, double* quot, double* root,
                          uint16_t* half, hipStream_t stream);

/* Read (and optionally clear) the device error word; synchronizes. */
mkv_status kv_pool_check_errors(mkv_pool* pool, uint32_t* err_word, int32_t clear);

const char* mkv_status_string(mkv_status s);

#ifdef __cplusplus
}
#endif
#endif /* MINIMA_KV_H */
