// Pool-state kernels: FP8 append (Alg. 1 Append; Sec. 3.1 Recent tier), FP8 ->
// TQ3 migration (Alg. 1 Retier; Sec. 4.3 normalize-rotate-pack), TQ3 -> FP8
// promotion (Alg. 1 Promote), the compact per-format page lists (Sec. 4.1)
// and a zero-fill helper.
//
// Every result that the CPU oracle fixes bit for bit (page ids, tags, free
// lists, FP8 codes and scales, TQ3 codes, gamma, V scale/zero) is produced by
// integer arithmetic or by single IEEE operations in a fixed order; this file
// is compiled with -ffp-contract=off.
#include <hip/hip_runtime.h>

#include "mkv_append.h"
#include "mkv_internal.h"
#include "../../include/minima_kv.h"

namespace mkv {

static int grid_for(int64_t items, int cap) {
  return (int)(items < 1 ? 1 : (items < cap ? items : cap));
}

// ===========================================================================
// Append
// ===========================================================================

// One workgroup: validate the whole call, then hand out FP8 ids in ascending
// (request, page) order and list every page that receives tokens.
__global__ __launch_bounds__(1024) void append_plan_kernel(int n_req, int32_t* bt, uint8_t* tags,
                                                           int max_pages, const int32_t* sb,
                                                           const int32_t* cu, int32_t* ctrl,
                                                           const int32_t* fp8_stack, int32_t* list,
                                                           int n_fp8, int n_new_total, int32_t* rc8) {
  __shared__ int scratch[32];
  __shared__ int s_err, s_need, s_touch;
  const int tid = threadIdx.x;
  if (tid == 0) {
    s_err = 0; s_need = 0; s_touch = 0;
    // rows of request r are cu[r] .. cu[r+1]-1 of an n_new_total-row input
    if (cu[0] != 0 || cu[n_req] != n_new_total) s_err = MKV_DEVERR_RANGE;
  }
  __syncthreads();
  for (int r = 0; r < n_req; ++r) {
    const int n = cu[r + 1] - cu[r], s0 = sb[r];
    if (n < 0 || s0 < 0) {
      if (tid == 0) atomicOr(&s_err, (int)MKV_DEVERR_RANGE);
      continue;
    }
    if (n == 0) continue;
    const int p0 = s0 / PAGE, p1 = (s0 + n - 1) / PAGE;
    if (p1 >= max_pages) {
      if (tid == 0) atomicOr(&s_err, (int)MKV_DEVERR_RANGE);
      continue;
    }
    int need = 0, bad = 0;
    for (int p = p0 + tid; p <= p1; p += blockDim.x) {
      const int64_t i = (int64_t)r * max_pages + p;
      if (bt[i] < 0) need++;
      else if (tags[i] != TAG_R) bad |= MKV_DEVERR_NOT_RECENT;
      else if (bt[i] >= n_fp8) bad |= MKV_DEVERR_RANGE;
    }
    if (need) atomicAdd(&s_need, need);
    if (bad) atomicOr(&s_err, bad);
    if (tid == 0) s_touch += p1 - p0 + 1;
  }
  __syncthreads();
  const int top = ctrl[CTRL_FP8_TOP];
  if (tid == 0) {
    if (s_err == 0 && s_need > top) s_err |= MKV_DEVERR_FP8_EXHAUSTED;
    if (s_err == 0 && s_touch > n_fp8) s_err |= MKV_DEVERR_RANGE;
  }
  __syncthreads();
  if (s_err) {
    if (tid == 0) {
      atomicOr(&ctrl[CTRL_ERR], s_err);
      ctrl[CTRL_ABORT] = 1;
      ctrl[CTRL_NLIST] = 0;
    }
    return;
  }
  int base_alloc = 0, base_list = 0;
  for (int r = 0; r < n_req; ++r) {
    const int n = cu[r + 1] - cu[r], s0 = sb[r];
    if (n <= 0) continue;
    const int p0 = s0 / PAGE, p1 = (s0 + n - 1) / PAGE;
    for (int c0 = p0; c0 <= p1; c0 += blockDim.x) {
      const int p = c0 + tid;
      const bool in = p <= p1;
      const int64_t i = (int64_t)r * max_pages + p;
      const int unm = (in && bt[i] < 0) ? 1 : 0;
      int tot;
      const int rank = block_excl_scan(unm, scratch, &tot);
      if (in) {
        int id;
        if (unm) {
          id = fp8_stack[top - 1 - (base_alloc + rank)];
          bt[i] = id;
          tags[i] = TAG_R;
          rc8[id] = 1;  // one request reference
        } else {
          id = bt[i];
        }
        int32_t* e = list + 4LL * (base_list + (p - p0));
        e[0] = r;
        e[1] = p;
        e[2] = id;
        e[3] = 0;
      }
      base_alloc += tot;
    }
    base_list += p1 - p0 + 1;
  }
  if (tid == 0) {
    ctrl[CTRL_FP8_TOP] = top - base_alloc;
    ctrl[CTRL_NLIST] = base_list;
    ctrl[CTRL_ABORT] = 0;
  }
}


// Quantize one tensor (K or V) of one page-head with one wave.  Slots [0, t0)
// already hold codes with the page's scale; the new fp32 values are rows
// row0 + t (t in [t0, t1)) of src, [row][H][D].  The scale only grows: when the
// new amax exceeds 448 * s_old the old codes are re-rounded to the new scale.
// All loads are issued before any store so that one wave needs about one
// memory round trip (plus one more when old codes are re-rounded).
template <int D>
__device__ void quant_task(uint8_t* reg, float* sc, int kv, const uint16_t* src, int64_t row0,
                           int t0, int t1, int H, int h, int lane) {
  constexpr int CL = D / 16, D4 = D / 4, NC = PAGE * D4 / 64;  // NC uint2 per lane at most
  const uint16_t* srow = src + (row0 * H + h) * D;  // token t at srow[t * H * D + c]
  const int64_t tstride = (int64_t)H * D;
  const float s_old = t0 > 0 ? sc[kv] : 0.0f;
  const int n4 = (t1 - t0) * D4;  // new inputs, 4 channels per item
  uint2 x[NC];
  float amax = 0.0f;
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const int idx = lane + 64 * k;
    x[k] = make_uint2(0u, 0u);
    if (idx < n4) {
      const int t = t0 + idx / D4, c = 4 * (idx % D4);
      x[k] = *reinterpret_cast<const uint2*>(srow + t * tstride + c);
    }
  }
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    amax = fmaxf(amax, fmaxf(fmaxf(fabsf(__uint_as_float(x[k].x << 16)),
                                   fabsf(__uint_as_float(x[k].x & 0xFFFF0000u))),
                             fmaxf(fabsf(__uint_as_float(x[k].y << 16)),
                                   fabsf(__uint_as_float(x[k].y & 0xFFFF0000u)))));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
  float s_new = s_old;
  bool requant = false;
  if (t0 == 0) {
    s_new = amax / 448.0f;
  } else if (!(amax <= 448.0f * s_old)) {
    s_new = amax / 448.0f;
    requant = true;
  }
  uint32_t* rw = reinterpret_cast<uint32_t*>(reg + (kv ? PAGE * D : 0));
  if (requant) {
    // dwords holding old codes: K rows t < t0; V token groups g < ceil(t0/4)
    const int gn = (t0 + 3) / 4;  // V dwords of token groups g < gn: 16 * gn * CL = gn * D
    const int n_old = kv ? gn * D : t0 * D4;
    uint32_t ow[NC];
#pragma unroll
    for (int k = 0; k < NC; ++k) {
      const int w = lane + 64 * k;
      const int wi = kv ? (w / (CL * gn)) * 4 * CL + (w % (CL * gn)) : w;
      ow[k] = w < n_old ? rw[wi] : 0u;
    }
#pragma unroll
    for (int k = 0; k < NC; ++k) {
      const int w = lane + 64 * k;
      if (w < n_old) {
        const int wi = kv ? (w / (CL * gn)) * 4 * CL + (w % (CL * gn)) : w;
        const int g = (wi / CL) % 4;
        uint32_t outw = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int t = kv ? 4 * g + b : wi / D4;
          uint32_t code = (ow[k] >> (8 * b)) & 0xFFu;
          if (t < t0) code = f32_to_e4m3((e4m3_to_f32(code) * s_old) / s_new);
          outw |= code << (8 * b);
        }
        rw[wi] = outw;
      }
    }
    __builtin_amdgcn_s_waitcnt(0);  // re-rounded dwords land before new-code byte stores
  }
  // new codes
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const int idx = lane + 64 * k;
    if (idx < n4) {
      const int t = t0 + idx / D4, c = 4 * (idx % D4);
      uint32_t code[4];
      const uint32_t hv[4] = {x[k].x << 16, x[k].x & 0xFFFF0000u, x[k].y << 16, x[k].y & 0xFFFF0000u};
#pragma unroll
      for (int b = 0; b < 4; ++b)
        code[b] = s_new > 0.0f ? f32_to_e4m3(__uint_as_float(hv[b]) / s_new) : 0u;
      if (!kv) {
        rw[(t * D + c) / 4] = code[0] | (code[1] << 8) | (code[2] << 16) | (code[3] << 24);
      } else {
#pragma unroll
        for (int b = 0; b < 4; ++b) reg[fp8_off<D>(1, t, c + b)] = (uint8_t)code[b];
      }
    }
  }
  // a fresh page: zero every slot past the new tokens
  if (t0 == 0 && t1 < PAGE) {
    if (!kv) {
      for (int w = t1 * D4 + lane; w < PAGE * D4; w += 64) rw[w] = 0u;
    } else {
      for (int w = lane; w < PAGE * D4; w += 64) {
        const int g = (w / CL) % 4;
        if (4 * g >= t1) {
          rw[w] = 0u;
        } else if (4 * g + 4 > t1) {
#pragma unroll
          for (int b = 0; b < 4; ++b)
            if (4 * g + b >= t1) reg[PAGE * D + 4 * w + b] = 0;
        }
      }
    }
  }
  if (lane == 0) sc[kv] = s_new;
}

// One quantisation task = (listed page, layer, head, K or V); one wave each.
template <int D>
__device__ __forceinline__ void run_quant_task(const PoolView& P, int64_t task, int layer_sel,
                                               int n_lcall, const int32_t* sb, const int32_t* cu,
                                               int n_new_total, const uint16_t* k,
                                               const uint16_t* v, const int32_t* lst, int lane) {
  const int H = P.n_kv_heads;
  const int kv = (int)(task & 1);
  const int64_t item = task >> 1;
  const int e = (int)(item / (n_lcall * H));
  const int lh = (int)(item % (n_lcall * H));
  const int li = lh / H, h = lh % H;
  const int r = lst[4 * e], p = lst[4 * e + 1], id = lst[4 * e + 2];
  const int layer = layer_sel < 0 ? li : layer_sel;
  const int s0 = sb[r], n = cu[r + 1] - cu[r];
  const int t0 = max(0, s0 - p * PAGE), t1 = min(PAGE, s0 + n - p * PAGE);
  const int64_t ph = ((int64_t)layer * P.n_fp8 + id) * H + h;
  const int64_t row0 = (int64_t)cu[r] + p * PAGE - s0;  // input row of slot t is row0 + t
  const uint16_t* src = (kv ? v : k) + (int64_t)li * n_new_total * H * D;
  quant_task<D>(P.fp8 + ph * fp8_region_bytes(D), P.fp8_scales + ph * 2, kv, src, row0, t0, t1, H,
                h, lane);
}

// Quantize every listed page-head of every requested layer (grid-stride over
// tasks, one wave per task).
template <int D>
__global__ __launch_bounds__(256) void append_quant_kernel(PoolView P, int layer_sel, int n_lcall,
                                                           const int32_t* sb, const int32_t* cu,
                                                           int n_new_total, const uint16_t* k,
                                                           const uint16_t* v) {
  if (P.ctrl[CTRL_ABORT]) return;
  const int64_t n_tasks = (int64_t)P.ctrl[CTRL_NLIST] * n_lcall * P.n_kv_heads * 2;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  for (int64_t t = (int64_t)blockIdx.x * 4 + wid; t < n_tasks; t += (int64_t)gridDim.x * 4)
    run_quant_task<D>(P, t, layer_sel, n_lcall, sb, cu, n_new_total, k, v, P.list, lane);
}

// Small appends (decode steps: a few tokens per request): one wave per task
// (touched page, layer, head, K or V) and no barrier.  Every wave reads the
// whole call (rows and start positions, block-table entries and tags of the
// touched pages, the head of the FP8 free list) and so reaches the same
// validation and the same fresh-page ids; the wave that arrives last on a
// counter in the control block (by then every other wave has finished its
// reads) records the fresh pages in the block table, pops them off the free
// list and resets the counter.  Three dependent memory round trips: (1) rows,
// starts and the free-list top; (2) table entries, free-list head and the
// task's new rows; (3) the page-head's codes and scale when it already holds
// tokens.  A task assembles the page-head's code block in LDS (old codes,
// re-rounded through a 256-entry table when the scale grows; new codes; zeros
// past the new tokens of a fresh page) and stores it with whole-dword writes.
// Same validation, allocation order and arithmetic as the two-kernel path.
constexpr int STEP_APPEND_MAX_TOKENS = 256;  // also bounds the touched pages
constexpr int STEP_APPEND_MAX_REQ = 256;
constexpr int STEP_APPEND_MAX_WAVES = 4096;


template <int D>
__global__ __launch_bounds__(64) void append_step_kernel(PoolView P, int layer_sel, int n_lcall,
                                                         int n_req, int32_t* bt, uint8_t* tags,
                                                         int max_pages, const int32_t* sb,
                                                         const int32_t* cu, int n_new_total,
                                                         const uint16_t* k, const uint16_t* v) {
  constexpr int RQ = STEP_APPEND_MAX_REQ / 64, EQ = STEP_APPEND_MAX_TOKENS / 64;
  __shared__ int s_base[STEP_APPEND_MAX_REQ + 1];  // first list entry of request r
  __shared__ int s_cu[STEP_APPEND_MAX_REQ], s_n[STEP_APPEND_MAX_REQ], s_s0[STEP_APPEND_MAX_REQ];
  __shared__ __align__(16) uint32_t s_img[PAGE * D / 4];
  __shared__ uint8_t s_lut[256];
  const int lane = threadIdx.x;
  const int H = P.n_kv_heads;
  // ---- round trip 1: rows, starts, free-list top
  const int top = P.ctrl[CTRL_FP8_TOP];
  int bad = (cu[0] != 0 || cu[n_req] != n_new_total) ? (int)MKV_DEVERR_RANGE : 0;
  int run = 0;  // list entries of the requests before this group of 64
#pragma unroll
  for (int i = 0; i < RQ; ++i) {
    const int r = lane + 64 * i;
    int touch = 0;
    if (r < n_req) {
      const int c_r = cu[r], n = cu[r + 1] - c_r, s0 = sb[r];
      // rows outside the input stay unread: inputs are loaded before the call
      // as a whole is known to be valid
      if (n < 0 || s0 < 0 || c_r < 0 || c_r + n > n_new_total) {
        bad |= MKV_DEVERR_RANGE;
      } else if (n > 0) {
        const int p0 = s0 / PAGE, p1 = (s0 + n - 1) / PAGE;
        if (p1 >= max_pages) bad |= MKV_DEVERR_RANGE;
        else touch = p1 - p0 + 1;
      }
      s_cu[r] = c_r;
      s_n[r] = n;
      s_s0[r] = s0;
    }
    const int incl = wave_incl_scan(touch, lane);
    if (r < n_req) s_base[r] = run + incl - touch;
    run += __shfl(incl, 63, 64);
  }
  const int n_ent = run;
  if (lane == 0) s_base[n_req] = n_ent;
  __builtin_amdgcn_wave_barrier();
  // list entry e -> (request, page): the last request whose first entry is <= e
  auto locate = [&](int e, int& r, int& p) {
    int lo = 0, hi = n_req - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_base[mid] <= e) lo = mid;
      else hi = mid - 1;
    }
    r = lo;
    p = s_s0[lo] / PAGE + (e - s_base[lo]);
  };
  // ---- round trip 2: table entries of the list, the free-list head, the
  // task's new rows
  int ent_bt[EQ], ent_tag[EQ];
#pragma unroll
  for (int j = 0; j < EQ; ++j) {
    const int e = lane + 64 * j;
    ent_bt[j] = 0;
    ent_tag[j] = TAG_R;
    if (e < n_ent) {
      int r, p;
      locate(e, r, p);
      const int64_t i = (int64_t)r * max_pages + p;
      ent_bt[j] = bt[i];
      ent_tag[j] = tags[i];
    }
  }
  const int stk = lane < top ? P.fp8_stack[top - 1 - lane] : -1;  // ids handed out first
  const int64_t n_tasks = (int64_t)n_ent * n_lcall * H * 2;
  const int64_t task = blockIdx.x;
  SmallTask<D> T;
  int e_t = 0;
  if (task < n_tasks) {
    T.kv = (int)(task & 1);
    const int64_t item = task >> 1;
    e_t = (int)(item / (n_lcall * H));
    const int lh = (int)(item % (n_lcall * H));
    T.li = lh / H;
    T.h = lh % H;
    T.layer = layer_sel < 0 ? T.li : layer_sel;
    int r, p;
    locate(e_t, r, p);
    T.r = __builtin_amdgcn_readfirstlane(r);
    T.p = __builtin_amdgcn_readfirstlane(p);
    const int c_r = __builtin_amdgcn_readfirstlane(s_cu[T.r]);
    const int s0 = __builtin_amdgcn_readfirstlane(s_s0[T.r]);
    const int n = __builtin_amdgcn_readfirstlane(s_n[T.r]);
    T.row0 = c_r + T.p * PAGE - s0;  // input row of slot t is row0 + t
    T.t0 = max(0, s0 - T.p * PAGE);
    T.t1 = min(PAGE, s0 + n - T.p * PAGE);
    // a listed page belongs to a request whose rows passed the range checks
    small_task_load_x<D>(T, H, n_new_total, k, v, lane);
  }
  // ---- validation and fresh-page ranks (identical in every wave)
  int fresh[EQ], rank[EQ], n_fresh = 0;
#pragma unroll
  for (int j = 0; j < EQ; ++j) {
    const int e = lane + 64 * j;
    fresh[j] = (e < n_ent && ent_bt[j] < 0) ? 1 : 0;
    if (e < n_ent && !fresh[j]) {
      if (ent_tag[j] != TAG_R) bad |= MKV_DEVERR_NOT_RECENT;
      else if (ent_bt[j] >= P.n_fp8) bad |= MKV_DEVERR_RANGE;
    }
    const int incl = wave_incl_scan(fresh[j], lane);
    rank[j] = n_fresh + incl - fresh[j];
    n_fresh += __shfl(incl, 63, 64);
  }
  if (n_fresh > top) bad |= MKV_DEVERR_FP8_EXHAUSTED;
  bad = wave_or(bad);
  // id of each entry: its table entry, or the free-list element of its rank
  int ent_id[EQ];
#pragma unroll
  for (int j = 0; j < EQ; ++j) {
    ent_id[j] = ent_bt[j];
    const int sl = rank[j] < 64 ? __shfl(stk, rank[j] & 63, 64) : -1;
    if (fresh[j] && bad == 0) ent_id[j] = rank[j] < 64 ? sl : P.fp8_stack[top - 1 - rank[j]];
  }
  if (bad == 0 && task < n_tasks) {
    // ---- round trip 3 and the task
    int idv = 0;
#pragma unroll
    for (int j = 0; j < EQ; ++j) idv = (e_t >> 6) == j ? ent_id[j] : idv;
    const int id = __builtin_amdgcn_readfirstlane(__shfl(idv, e_t & 63, 64));
    small_task_load_old<D>(T, P, id, lane);
    small_task_run<D>(T, P, id, s_img, s_lut, lane);
  }
  // ---- nothing to publish (no fresh page; every wave reached the same
  // verdict): the first wave reports an error, no wave waits for the others
  if (n_fresh == 0 || bad) {
    if (bad && blockIdx.x == 0 && lane == 0) atomicOr(&P.ctrl[CTRL_ERR], bad);
    return;
  }
  // ---- arrive; the last wave records the fresh pages.  Only the order of
  // every wave's table reads before the last wave's table writes matters:
  // a wave counts itself once all its loads have returned (no device-scope
  // fence, which would write back this die's L2).  The page codes and the
  // table are published to later kernels by the end of this kernel.
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  int prev = 0;
  if (lane == 0) prev = atomicAdd(&P.ctrl[CTRL_APPEND_ARRIVE], 1);
  prev = __shfl(prev, 0, 64);
  if (prev != (int)gridDim.x - 1) return;
#pragma unroll
  for (int j = 0; j < EQ; ++j) {
    const int e = lane + 64 * j;
    if (e < n_ent && fresh[j]) {
      int r, p;
      locate(e, r, p);
      const int64_t i = (int64_t)r * max_pages + p;
      bt[i] = ent_id[j];
      tags[i] = TAG_R;
      P.rc8[ent_id[j]] = 1;
    }
  }
  if (lane == 0) P.ctrl[CTRL_FP8_TOP] = top - n_fresh;
  if (lane == 0) P.ctrl[CTRL_APPEND_ARRIVE] = 0;
}

// ===========================================================================
// Migrate (Retier to TQ3)
// ===========================================================================

// Plan of a migration, in two launches over nb <= MIG_BLOCKS workgroups; each
// workgroup owns a range of whole batches of the table taken as one run of
// (request, page) entries, MIG_KB consecutive entries per thread with every
// load of a batch in flight together.  The count launch validates its range
// (lengths, candidate ids) and counts the migrating pages; the list launch
// sums the counts of the ranges before its own, checks the whole call
// (errors, free-list room) so that a failing call changes nothing, ranks its
// migrating pages in (request, page) order with one block scan per batch,
// retags Anchors and writes the work list with the TQ3 ids popped in that
// order.  The table entries, Stale tags and FP8 releases are published by the
// publish kernel after the encode kernel has built the TQ3 pages (Alg. 1,
// copy before publish).
constexpr int MIG_KB = 8;
constexpr int MIG_NT = 1024;
constexpr int64_t MIG_BATCH = (int64_t)MIG_NT * MIG_KB;
struct MigBatch {
  uint8_t tg[MIG_KB], an[MIG_KB];
  int32_t id[MIG_KB], sl[MIG_KB], rq[MIG_KB], pg[MIG_KB], rc[MIG_KB];
};
// references of the entries' pages (shared pages are left alone by Retier and
// Promote); 0 where the tag or id names no page
struct RcView {
  const int32_t* rc8;
  const int32_t* rc3;
  int n_fp8, n_tq3;
};
__device__ __forceinline__ void mig_load_rc(MigBatch& m, const RcView& v) {
#pragma unroll
  for (int j = 0; j < MIG_KB; ++j) {
    const bool f8 = m.tg[j] == TAG_R || m.tg[j] == TAG_A, f3 = m.tg[j] == TAG_S;
    const int id = m.id[j];
    const bool ok = m.rq[j] >= 0 && id >= 0 && ((f8 && id < v.n_fp8) || (f3 && id < v.n_tq3));
    m.rc[j] = ok ? (f8 ? v.rc8 : v.rc3)[id] : 0;
  }
}
// entries f0 .. f0 + MIG_KB - 1: (request, page) stepped from one division
__device__ __forceinline__ void mig_load(MigBatch& m, int64_t f0, int64_t N, int max_pages,
                                         const int32_t* bt, const uint8_t* tags,
                                         const uint8_t* anchor, const int32_t* seq_lens) {
  int r = (int)(f0 / max_pages), p = (int)(f0 - (int64_t)r * max_pages);
#pragma unroll
  for (int j = 0; j < MIG_KB; ++j) {
    const bool in = f0 + j < N;
    const int64_t f = in ? f0 + j : 0;
    m.rq[j] = in ? r : -1;
    m.pg[j] = p;
    m.tg[j] = tags[f];
    m.an[j] = anchor ? anchor[f] : 0;
    m.id[j] = bt[f];
    m.sl[j] = seq_lens[in ? r : 0];
    if (++p == max_pages) { p = 0; ++r; }
  }
}
// The reference counts a migration plan needs: only a Recent page that has
// left the window and is not an anchor can migrate, and only then does its
// count decide (a shared page stays FP8); every other entry skips the gather.
__device__ __forceinline__ void mig_load_rc_candidates(MigBatch& m, const RcView& v, int W) {
#pragma unroll
  for (int j = 0; j < MIG_KB; ++j) {
    const int p = m.pg[j], S = m.sl[j], id = m.id[j];
    const bool cand = m.rq[j] >= 0 && m.tg[j] == TAG_R && !m.an[j] && p < (S + PAGE - 1) / PAGE &&
                      (p + 1) * PAGE <= S - W && id >= 0 && id < v.n_fp8;
    m.rc[j] = cand ? v.rc8[id] : 0;
  }
}
// 1: migrating page, 2: Anchor to retag, 0: neither
__device__ __forceinline__ int mig_kind(const MigBatch& m, int j, int W) {
  if (m.rq[j] < 0) return 0;
  const int p = m.pg[j], S = m.sl[j];
  if (m.tg[j] != TAG_R || p >= (S + PAGE - 1) / PAGE || (p + 1) * PAGE > S - W) return 0;
  if (m.an[j]) return 2;
  return m.rc[j] == 1 ? 1 : 0;  // a shared (sealed) page stays until it is private
}

// Count and validate the entries [e0, e1) (the whole workgroup); workgroup 0
// also checks every request's length.  Returns through s_cnt / s_err.
__device__ __forceinline__ void mig_count_range(int b, int n_req, const int32_t* bt,
                                                const uint8_t* tags, int max_pages,
                                                const uint8_t* anchor, const int32_t* seq_lens,
                                                int W, int64_t e0, int64_t e1, int n_fp8,
                                                int* s_cnt, int* s_err, const RcView& rv) {
  const int tid = threadIdx.x;
  int err = 0, cnt = 0;
  if (b == 0) {
    for (int r = tid; r < n_req; r += MIG_NT) {
      const int S = seq_lens[r];
      if (S < 0 || (S + PAGE - 1) / PAGE > max_pages) err |= MKV_DEVERR_RANGE;
    }
  }
  for (int64_t b0 = e0; b0 < e1; b0 += MIG_BATCH) {
    MigBatch m;
    mig_load(m, b0 + (int64_t)tid * MIG_KB, e1, max_pages, bt, tags, anchor, seq_lens);
    mig_load_rc_candidates(m, rv, W);
#pragma unroll
    for (int j = 0; j < MIG_KB; ++j) {
      const int p = m.pg[j], S = m.sl[j];
      const bool old_r = m.rq[j] >= 0 && m.tg[j] == TAG_R && p < (S + PAGE - 1) / PAGE &&
                         (p + 1) * PAGE <= S - W && !m.an[j];
      if (old_r && (m.id[j] < 0 || m.id[j] >= n_fp8)) err |= MKV_DEVERR_RANGE;
      if (mig_kind(m, j, W) == 1) cnt++;
    }
  }
  if (cnt) atomicAdd(s_cnt, cnt);
  if (err) atomicOr(s_err, err);
}

__global__ __launch_bounds__(MIG_NT) void migrate_count_kernel(
    int n_req, const int32_t* bt, const uint8_t* tags, int max_pages, const uint8_t* anchor,
    const int32_t* seq_lens, int W, int32_t* ctrl, int32_t* mig, int64_t per_blk, int n_fp8,
    RcView rv) {
  __shared__ int s_err, s_cnt;
  const int tid = threadIdx.x, b = blockIdx.x;
  if (tid == 0) { s_err = 0; s_cnt = 0; }
  if (b == 0 && tid == 0) mig[2 * MIG_BLOCKS] = ctrl[CTRL_TQ3_TOP];  // read before the list launch moves it
  const int64_t N = (int64_t)n_req * max_pages;
  const int64_t e0 = (int64_t)b * per_blk, e1 = min(N, e0 + per_blk);
  __syncthreads();
  mig_count_range(b, n_req, bt, tags, max_pages, anchor, seq_lens, W, e0, e1, n_fp8, &s_cnt, &s_err,
                  rv);
  __syncthreads();
  if (tid == 0) {
    mig[b] = s_cnt;
    mig[MIG_BLOCKS + b] = s_err;
  }
}

// ONE: a single workgroup owns the whole table (at most one batch): it loads
// the batch once, counts and validates it, and lists it after one scan (one
// launch instead of two, one pass over the table instead of two).
template <bool ONE>
__global__ __launch_bounds__(MIG_NT) void migrate_list_kernel(
    int n_req, const int32_t* bt, uint8_t* tags, int max_pages, const uint8_t* anchor,
    const int32_t* seq_lens, int W, int32_t* ctrl, const int32_t* tq3_stack, int32_t* list,
    const int32_t* mig, int64_t per_blk, int nb, int n_fp8, RcView rv) {
  __shared__ int scratch[32];
  __shared__ int s_err, s_tot, s_pre;
  const int tid = threadIdx.x, b = blockIdx.x;
  if (tid == 0) { s_err = 0; s_tot = 0; s_pre = 0; }
  __syncthreads();
  const int top3 = ONE ? ctrl[CTRL_TQ3_TOP] : mig[2 * MIG_BLOCKS];
  if constexpr (ONE) {
    const int64_t N = (int64_t)n_req * max_pages;  // <= MIG_BATCH
    MigBatch m;
    mig_load(m, (int64_t)tid * MIG_KB, N, max_pages, bt, tags, anchor, seq_lens);
    mig_load_rc_candidates(m, rv, W);
    int err = 0, k[MIG_KB], c = 0;
    for (int r = tid; r < n_req; r += MIG_NT) {
      const int S = seq_lens[r];
      if (S < 0 || (S + PAGE - 1) / PAGE > max_pages) err |= MKV_DEVERR_RANGE;
    }
#pragma unroll
    for (int j = 0; j < MIG_KB; ++j) {
      const int p = m.pg[j], S = m.sl[j];
      const bool old_r = m.rq[j] >= 0 && m.tg[j] == TAG_R && p < (S + PAGE - 1) / PAGE &&
                         (p + 1) * PAGE <= S - W && !m.an[j];
      if (old_r && (m.id[j] < 0 || m.id[j] >= n_fp8)) err |= MKV_DEVERR_RANGE;
      k[j] = mig_kind(m, j, W);
      c += k[j] == 1;
    }
    if (err) atomicOr(&s_err, err);
    int total;
    int e = block_excl_scan(c, scratch, &total);  // its barriers also publish s_err
    err = s_err;
    if (err == 0 && total > top3) err |= MKV_DEVERR_TQ3_EXHAUSTED;
    if (err == 0 && total > n_fp8) err |= MKV_DEVERR_RANGE;
    if (err) {
      if (tid == 0) {
        atomicOr(&ctrl[CTRL_ERR], err);
        ctrl[CTRL_ABORT] = 1;
        ctrl[CTRL_NLIST] = 0;
      }
      return;
    }
    const int64_t f0 = (int64_t)tid * MIG_KB;
#pragma unroll
    for (int j = 0; j < MIG_KB; ++j) {
      if (k[j] == 2) tags[f0 + j] = TAG_A;  // Anchor: tag only, stays FP8
      if (k[j] == 1) {
        int32_t* le = list + 4LL * e;
        le[0] = m.rq[j];
        le[1] = m.pg[j];
        le[2] = m.id[j];
        le[3] = tq3_stack[top3 - 1 - e];
        e++;
      }
    }
    if (tid == 0) {
      ctrl[CTRL_TQ3_TOP] = top3 - total;
      ctrl[CTRL_NLIST] = total;
      ctrl[CTRL_ABORT] = 0;
    }
    return;
  } else if (tid < nb) {
    const int c = mig[tid], e = mig[MIG_BLOCKS + tid];
    if (c) atomicAdd(&s_tot, c);
    if (c && tid < b) atomicAdd(&s_pre, c);
    if (e) atomicOr(&s_err, e);
  }
  __syncthreads();
  int err = s_err;
  const int total = s_tot;
  if (err == 0 && total > top3) err |= MKV_DEVERR_TQ3_EXHAUSTED;
  if (err == 0 && total > n_fp8) err |= MKV_DEVERR_RANGE;
  if (err) {
    if (b == 0 && tid == 0) {
      atomicOr(&ctrl[CTRL_ERR], err);
      ctrl[CTRL_ABORT] = 1;
      ctrl[CTRL_NLIST] = 0;
    }
    return;
  }
  const int64_t N = (int64_t)n_req * max_pages;
  const int64_t e0 = (int64_t)b * per_blk, e1 = min(N, e0 + per_blk);
  int base = s_pre;
  for (int64_t b0 = e0; b0 < e1; b0 += MIG_BATCH) {
    MigBatch m;
    mig_load(m, b0 + (int64_t)tid * MIG_KB, e1, max_pages, bt, tags, anchor, seq_lens);
    mig_load_rc_candidates(m, rv, W);
    int k[MIG_KB], c = 0;
#pragma unroll
    for (int j = 0; j < MIG_KB; ++j) {
      k[j] = mig_kind(m, j, W);
      c += k[j] == 1;
    }
    int tot;
    int e = base + block_excl_scan(c, scratch, &tot);
    const int64_t f0 = b0 + (int64_t)tid * MIG_KB;
#pragma unroll
    for (int j = 0; j < MIG_KB; ++j) {
      if (k[j] == 2) tags[f0 + j] = TAG_A;  // Anchor: tag only, stays FP8
      if (k[j] == 1) {
        int32_t* le = list + 4LL * e;
        le[0] = m.rq[j];
        le[1] = m.pg[j];
        le[2] = m.id[j];
        le[3] = tq3_stack[top3 - 1 - e];
        e++;
      }
    }
    base += tot;
  }
  if (b == 0 && tid == 0) {
    ctrl[CTRL_TQ3_TOP] = top3 - total;
    ctrl[CTRL_NLIST] = total;
    ctrl[CTRL_ABORT] = 0;
  }
}

// TQ3 key code of one rotated coordinate: the codebook level nearest to
// z = y / sqrt(n2) * (normalised coordinate; levels +-{0.25, 0.75, 1.375,
// 2.25}), ties to the lower level.  The decision boundaries are 0 and
// +-{8, 17, 29} / 16, so with u = (16 y)^2 the magnitude class of z is the
// number of boundaries b with u beyond b^2 n2 -- three exact 64-bit integer
// comparisons (u < 2^60 and b^2 n2 < 2^54 for |X_j| <= 448 * 2^9, d <= 256).
// A positive z takes codes 4 + class (strictly beyond a boundary to move up);
// z <= 0 takes 3 - class (at or beyond a boundary to move down, so a tie and
// z = 0 stay on the side of the lower code).
__device__ __forceinline__ int tq3_decide(int32_t y, int64_t n2) {
  const int64_t u = (16LL * y) * (16LL * y);
  const int64_t b1 = 64LL * n2, b2 = 289LL * n2, b3 = 841LL * n2;
  if (y > 0) return 4 + (int)(u > b1) + (int)(u > b2) + (int)(u > b3);
  return 3 - (int)(u >= b1) - (int)(u >= b2) - (int)(u >= b3);
}

// Encode one FP8 page-head into a TQ3 region per work item (grid-stride over
// listed pages x layers x heads).  256 threads.
template <int D>
__global__ __launch_bounds__(256) void migrate_encode_kernel(PoolView P) {
  if (P.ctrl[CTRL_ABORT]) return;
  constexpr int CL = D / 16, NDW = 3 * D / 128, CB = 3 * D / 32;
  __shared__ int32_t y[PAGE * D];
  __shared__ uint8_t kc[PAGE * D];
  __shared__ uint8_t vc[PAGE * D];
  const int H = P.n_kv_heads, L = P.n_layers;
  const int64_t n_items = (int64_t)P.ctrl[CTRL_NLIST] * L * H;
  const int tid = threadIdx.x, tok = tid >> 4, l16 = tid & 15;
  for (int64_t item = blockIdx.x; item < n_items; item += gridDim.x) {
    const int e = (int)(item / (L * H));
    const int lh = (int)(item % (L * H));
    const int layer = lh / H, h = lh % H;
    const int src = P.list[4 * e + 2], dst = P.list[4 * e + 3];
    const int64_t sph = ((int64_t)layer * P.n_fp8 + src) * H + h;
    const uint8_t* f8 = P.fp8 + sph * fp8_region_bytes(D);
    const float sK = P.fp8_scales[sph * 2], sV = P.fp8_scales[sph * 2 + 1];
    uint8_t* reg = P.tq3 + (((int64_t)layer * P.n_tq3 + dst) * H + h) * tq3_region_bytes(D);
    // keys: X = sigma * e4m3 * 2^9 (integers), n2 = |X|^2
    int64_t n2 = 0;
    for (int j = 0; j < D / 16; ++j) {
      const int c = l16 + 16 * j;
      const int32_t X = (int32_t)P.sigma[c] * e4m3_times_512(f8[tok * D + c]);
      y[tok * D + c] = X;
      n2 += (int64_t)X * X;
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) n2 += __shfl_xor(n2, o, 64);
    __syncthreads();
    // Sylvester Walsh-Hadamard transform of each token row (exact in int32)
    for (int s = 1; s < D; s <<= 1) {
      for (int b = l16; b < D / 2; b += 16) {
        const int i = (b / s) * 2 * s + (b % s);
        const int32_t a0 = y[tok * D + i], a1 = y[tok * D + i + s];
        y[tok * D + i] = a0 + a1;
        y[tok * D + i + s] = a0 - a1;
      }
      __syncthreads();
    }
    int M = 0;
    for (int j = 0; j < D / 16; ++j) {
      const int c = l16 + 16 * j;
      const int code = n2 ? tq3_decide(y[tok * D + c], n2) : 3;
      kc[tok * D + c] = (uint8_t)code;
      M += mu2x64(code);
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) M += __shfl_xor(M, o, 64);
    if (l16 == 0) {
      uint16_t g16 = 0;
      if (n2) {
        const double rr = (double)n2 / (double)M;
        const double sq = sqrt(rr);
        const double g = sq * ((double)sK * 0.015625);
        g16 = f64_to_f16_rne_sat(g);
      }
      reinterpret_cast<uint16_t*>(reg + 12 * D)[tok] = g16;
    }
    // values: per channel asymmetric 3-bit over the 16 tokens
    if (tid < D) {
      const int c = tid;
      double lo = INFINITY, hi = -INFINITY;
      for (int t = 0; t < PAGE; ++t) {
        const double vv = (double)sV * (double)e4m3_to_f32(f8[fp8_off<D>(1, t, c)]);
        lo = fmin(lo, vv);
        hi = fmax(hi, vv);
      }
      const uint16_t z16 = f64_to_f16_rne_sat(lo);
      const uint16_t s16 = f64_to_f16_rne_sat((hi - lo) / 7.0);
      reinterpret_cast<uint16_t*>(reg + 12 * D + 32)[c] = s16;
      reinterpret_cast<uint16_t*>(reg + 14 * D + 32)[c] = z16;
      const double z = f16_bits_to_f64(z16), s = f16_bits_to_f64(s16);
      for (int t = 0; t < PAGE; ++t) {
        int code = 0;
        if (s != 0.0) {
          const double vv = (double)sV * (double)e4m3_to_f32(f8[fp8_off<D>(1, t, c)]);
          double u = rint((vv - z) / s);
          u = fmin(fmax(u, 0.0), 7.0);
          code = (int)u;
        }
        vc[t * D + c] = (uint8_t)code;
      }
    }
    __syncthreads();
    // pack: threads 0..63 build K chunks (t, g), threads 64..127 V chunks (r, g)
    if (tid < 128) {
      uint32_t Dw[NDW];
#pragma unroll
      for (int w = 0; w < NDW; ++w) Dw[w] = 0;
      uint8_t* out;
      if (tid < 64) {
        const int t = tid >> 2, g = tid & 3;
        for (int q = 0; q < D / 16; ++q)
          for (int b = 0; b < 4; ++b) quad_put<NDW>(Dw, q, b, kc[t * D + (D / 4) * g + 4 * q + b]);
        out = reg + (g * 16 + t) * CB;
      } else {
        const int rr = (tid - 64) >> 2, g = (tid - 64) & 3;
        for (int q = 0; q < CL; ++q)
          for (int b = 0; b < 4; ++b) quad_put<NDW>(Dw, q, b, vc[(4 * g + b) * D + CL * rr + q]);
        out = reg + 6 * D + (g * 16 + rr) * CB;
      }
#pragma unroll
      for (int w = 0; w < NDW; ++w) reinterpret_cast<uint32_t*>(out)[w] = Dw[w];
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(1024) void migrate_publish_kernel(int32_t* bt, uint8_t* tags,
                                                               int max_pages, int32_t* ctrl,
                                                               int32_t* fp8_stack,
                                                               const int32_t* list, int32_t* rc8,
                                                               int32_t* rc3) {
  if (ctrl[CTRL_ABORT]) return;
  const int n = ctrl[CTRL_NLIST];
  const int top = ctrl[CTRL_FP8_TOP];
  for (int k = threadIdx.x; k < n; k += blockDim.x) {
    const int r = list[4 * k], p = list[4 * k + 1], src = list[4 * k + 2], dst = list[4 * k + 3];
    const int64_t i = (int64_t)r * max_pages + p;
    bt[i] = dst;
    tags[i] = TAG_S;
    rc3[dst] = 1;  // the request's reference moves to the new page
    rc8[src] = 0;
    fp8_stack[top + k] = src;
  }
  __syncthreads();
  if (threadIdx.x == 0) ctrl[CTRL_FP8_TOP] = top + n;
}

// ===========================================================================
// Promote (a Stale page back to FP8)
// ===========================================================================

// Plan of a promotion: one workgroup walks the table twice (count and
// validate, then list in (request, page) order with one block scan per batch).
// A page is promoted when it is Stale, its mask entry is set and it lies below
// the request's length.  A failing call (bad length, out-of-range TQ3 id, FP8
// free list too short) sets the error word and the abort flag and lists
// nothing.  The FP8 ids are popped here; the pages are built by the build
// kernel and published after it (copy before publish).
__device__ __forceinline__ bool pro_hit(const MigBatch& m, int j) {
  if (m.rq[j] < 0 || m.tg[j] != TAG_S || !m.an[j] || m.rc[j] != 1) return false;
  return m.pg[j] < (m.sl[j] + PAGE - 1) / PAGE;
}

__global__ __launch_bounds__(MIG_NT) void promote_plan_kernel(
    int n_req, const int32_t* bt, const uint8_t* tags, int max_pages, const uint8_t* mask,
    const int32_t* seq_lens, int32_t* ctrl, const int32_t* fp8_stack, int32_t* list, int n_tq3,
    RcView rv) {
  __shared__ int scratch[32];
  __shared__ int s_err, s_tot;
  const int tid = threadIdx.x;
  if (tid == 0) { s_err = 0; s_tot = 0; }
  __syncthreads();
  const int64_t N = (int64_t)n_req * max_pages;
  int err = 0, cnt = 0;
  for (int r = tid; r < n_req; r += MIG_NT) {
    const int S = seq_lens[r];
    if (S < 0 || (S + PAGE - 1) / PAGE > max_pages) err |= MKV_DEVERR_RANGE;
  }
  for (int64_t b0 = 0; b0 < N; b0 += MIG_BATCH) {
    MigBatch m;
    mig_load(m, b0 + (int64_t)tid * MIG_KB, N, max_pages, bt, tags, mask, seq_lens);
    mig_load_rc(m, rv);
#pragma unroll
    for (int j = 0; j < MIG_KB; ++j) {
      if (m.rq[j] >= 0 && m.tg[j] == TAG_S && m.an[j] && m.pg[j] < (m.sl[j] + PAGE - 1) / PAGE &&
          (m.id[j] < 0 || m.id[j] >= n_tq3))
        err |= MKV_DEVERR_RANGE;
      if (pro_hit(m, j)) {
        cnt++;
      }
    }
  }
  if (cnt) atomicAdd(&s_tot, cnt);
  if (err) atomicOr(&s_err, err);
  __syncthreads();
  const int total = s_tot;
  const int top8 = ctrl[CTRL_FP8_TOP];
  err = s_err;
  if (err == 0 && total > top8) err |= MKV_DEVERR_FP8_EXHAUSTED;
  if (err) {
    if (tid == 0) {
      atomicOr(&ctrl[CTRL_ERR], err);
      ctrl[CTRL_ABORT] = 1;
      ctrl[CTRL_NLIST] = 0;
    }
    return;
  }
  int base = 0;
  for (int64_t b0 = 0; b0 < N; b0 += MIG_BATCH) {
    MigBatch m;
    const int64_t f0 = b0 + (int64_t)tid * MIG_KB;
    mig_load(m, f0, N, max_pages, bt, tags, mask, seq_lens);
    mig_load_rc(m, rv);
    bool hit[MIG_KB];
    int c = 0;
#pragma unroll
    for (int j = 0; j < MIG_KB; ++j) {
      hit[j] = pro_hit(m, j);
      c += hit[j];
    }
    int tot;
    int e = base + block_excl_scan(c, scratch, &tot);
#pragma unroll
    for (int j = 0; j < MIG_KB; ++j) {
      if (hit[j]) {
        int32_t* le = list + 4LL * e;
        le[0] = m.rq[j];
        le[1] = m.pg[j];
        le[2] = m.id[j];                   // TQ3 source
        le[3] = fp8_stack[top8 - 1 - e];   // FP8 destination
        e++;
      }
    }
    base += tot;
  }
  if (tid == 0) {
    ctrl[CTRL_FP8_TOP] = top8 - total;
    ctrl[CTRL_NLIST] = total;
    ctrl[CTRL_ABORT] = 0;
  }
}

// Rebuild one listed page-head (layer, KV head) from its TQ3 region into its
// new FP8 region; 256 threads, thread (t, l) = (tid / 16, tid % 16) owns token
// t and channels l + 16 j.
//  keys: codes -> 8 * codebook level (integers), the Walsh-Hadamard transform
//        of each token row in int32 (exact), then
//        k = fp32((gamma * sigma_c * (y_c / 8)) / sqrt(D)) -- the products are
//        exact in fp64, the division the only fp64 rounding;
//  values: v = fp32(zero_c + scale_c * code), exact in fp64 before the
//        conversion;
//  FP8: per K and per V, s = amax / 448 over the 16 x D values, code =
//        E4M3(x / s) (0 when s = 0), the page written in the FP8 layout.
template <int D>
__global__ __launch_bounds__(256) void promote_build_kernel(PoolView P) {
  if (P.ctrl[CTRL_ABORT]) return;
  constexpr int NDW = 3 * D / 128, CB = 3 * D / 32, CL = D / 16, NJ = D / 16;
  constexpr int R3W = (int)tq3_region_bytes(D) / 4;
  constexpr int R8W = (int)fp8_region_bytes(D) / 4;
  __shared__ uint32_t src[R3W];
  __shared__ int32_t y[PAGE * D];
  __shared__ uint32_t dst[R8W];
  __shared__ float s_red[2][4];
  const int H = P.n_kv_heads, L = P.n_layers;
  const int64_t n_items = (int64_t)P.ctrl[CTRL_NLIST] * L * H;
  const int tid = threadIdx.x, t = tid >> 4, l16 = tid & 15, lane = tid & 63, wv = tid >> 6;
  // 8 * codebook level of each 3-bit code (levels +-0.25, 0.75, 1.375, 2.25)
  const int lvl8[8] = {-18, -11, -6, -2, 2, 6, 11, 18};
  for (int64_t item = blockIdx.x; item < n_items; item += gridDim.x) {
    const int e = (int)(item / (L * H));
    const int lh = (int)(item % (L * H));
    const int layer = lh / H, h = lh % H;
    const int sid = P.list[4 * e + 2], did = P.list[4 * e + 3];
    const uint32_t* reg3 = reinterpret_cast<const uint32_t*>(
        P.tq3 + (((int64_t)layer * P.n_tq3 + sid) * H + h) * tq3_region_bytes(D));
    for (int w = tid; w < R3W; w += 256) src[w] = reg3[w];
    __syncthreads();
    const uint8_t* sb = reinterpret_cast<const uint8_t*>(src);
    // key codes of token t, channels l16 + 16 j: chunk (t, g), quad q, byte b
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int c = l16 + 16 * j;
      const int g = c / (D / 4), cc = c % (D / 4);
      const uint32_t* ch = reinterpret_cast<const uint32_t*>(sb + (g * 16 + t) * CB);
      uint32_t dw[NDW];
#pragma unroll
      for (int k = 0; k < NDW; ++k) dw[k] = ch[k];
      const uint32_t code = (quad_sel<NDW>(dw, cc >> 2) >> (8 * (cc & 3))) & 7u;
      y[t * D + c] = lvl8[code];
    }
    __syncthreads();
    for (int st = 1; st < D; st <<= 1) {
      for (int b = l16; b < D / 2; b += 16) {
        const int i = (b / st) * 2 * st + (b % st);
        const int32_t a0 = y[t * D + i], a1 = y[t * D + i + st];
        y[t * D + i] = a0 + a1;
        y[t * D + i + st] = a0 - a1;
      }
      __syncthreads();
    }
    const double gam = f16_bits_to_f64(reinterpret_cast<const uint16_t*>(sb + 12 * D)[t]);
    const double rd = sqrt((double)D);
    float kx[NJ], vx[NJ];
    float kmax = 0.0f, vmax = 0.0f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int c = l16 + 16 * j;
      const double hc = (double)y[t * D + c] * 0.125;  // exact
      const double a = (gam * (double)P.sigma[c]) * hc;
      kx[j] = (float)(a / rd);
      kmax = fmaxf(kmax, fabsf(kx[j]));
      // value code of (t, c): V chunk (c / CL, t / 4), quad c % CL, byte t % 4
      const uint32_t* ch = reinterpret_cast<const uint32_t*>(sb + 6 * D + ((t >> 2) * 16 + c / CL) * CB);
      uint32_t dw[NDW];
#pragma unroll
      for (int k = 0; k < NDW; ++k) dw[k] = ch[k];
      const uint32_t vc = (quad_sel<NDW>(dw, c % CL) >> (8 * (t & 3))) & 7u;
      const double sc = f16_bits_to_f64(reinterpret_cast<const uint16_t*>(sb + 12 * D + 32)[c]);
      const double zr = f16_bits_to_f64(reinterpret_cast<const uint16_t*>(sb + 14 * D + 32)[c]);
      vx[j] = (float)(zr + sc * (double)vc);
      vmax = fmaxf(vmax, fabsf(vx[j]));
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      kmax = fmaxf(kmax, __shfl_xor(kmax, o, 64));
      vmax = fmaxf(vmax, __shfl_xor(vmax, o, 64));
    }
    if (lane == 0) {
      s_red[0][wv] = kmax;
      s_red[1][wv] = vmax;
    }
    __syncthreads();
    const float ka = fmaxf(fmaxf(s_red[0][0], s_red[0][1]), fmaxf(s_red[0][2], s_red[0][3]));
    const float va = fmaxf(fmaxf(s_red[1][0], s_red[1][1]), fmaxf(s_red[1][2], s_red[1][3]));
    const float sK = ka / 448.0f, sV = va / 448.0f;
    uint8_t* db = reinterpret_cast<uint8_t*>(dst);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int c = l16 + 16 * j;
      db[fp8_off<D>(0, t, c)] = (uint8_t)(sK > 0.0f ? f32_to_e4m3(kx[j] / sK) : 0u);
      db[fp8_off<D>(1, t, c)] = (uint8_t)(sV > 0.0f ? f32_to_e4m3(vx[j] / sV) : 0u);
    }
    __syncthreads();
    const int64_t ph = ((int64_t)layer * P.n_fp8 + did) * H + h;
    uint32_t* reg8 = reinterpret_cast<uint32_t*>(P.fp8 + ph * fp8_region_bytes(D));
    for (int w = tid; w < R8W; w += 256) reg8[w] = dst[w];
    if (tid == 0) {
      P.fp8_scales[ph * 2] = sK;
      P.fp8_scales[ph * 2 + 1] = sV;
    }
    __syncthreads();
  }
}

// Publish (Anchor, new FP8 id) and release the TQ3 ids, in list order.
__global__ __launch_bounds__(1024) void promote_publish_kernel(int32_t* bt, uint8_t* tags,
                                                               int max_pages, int32_t* ctrl,
                                                               int32_t* tq3_stack,
                                                               const int32_t* list, int32_t* rc8,
                                                               int32_t* rc3) {
  if (ctrl[CTRL_ABORT]) return;
  const int n = ctrl[CTRL_NLIST];
  const int top = ctrl[CTRL_TQ3_TOP];
  for (int k = threadIdx.x; k < n; k += blockDim.x) {
    const int32_t* le = list + 4LL * k;
    const int64_t i = (int64_t)le[0] * max_pages + le[1];
    bt[i] = le[3];
    tags[i] = TAG_A;
    rc8[le[3]] = 1;
    rc3[le[2]] = 0;
    tq3_stack[top + k] = le[2];
  }
  __syncthreads();
  if (threadIdx.x == 0) ctrl[CTRL_TQ3_TOP] = top + n;
}

// ===========================================================================
// Reference counts: SealPrefix / prefix attach (acquire), eviction and Finish
// (release)
// ===========================================================================

// (format, id) of a tagged entry: 0 FP8 (tags R, A), 1 TQ3 (tag S); false when
// the tag names no pool or the id is out of range.
__device__ __forceinline__ bool ref_of(uint8_t tag, int id, int n_fp8, int n_tq3, int& fmt) {
  fmt = tag == TAG_S ? 1 : 0;
  if (tag != TAG_R && tag != TAG_A && tag != TAG_S) return false;
  return id >= 0 && id < (fmt ? n_tq3 : n_fp8);
}

// One workgroup: every listed page must be live (one reference or more);
// otherwise nothing changes.  Then one more reference per entry.
__global__ __launch_bounds__(1024) void pages_acquire_kernel(int n, const int32_t* ids,
                                                             const uint8_t* tags, PoolView P) {
  __shared__ int s_err;
  const int tid = threadIdx.x;
  if (tid == 0) s_err = 0;
  __syncthreads();
  for (int k = tid; k < n; k += blockDim.x) {
    int fmt;
    const int id = ids[k];
    if (!ref_of(tags[k], id, P.n_fp8, P.n_tq3, fmt) || (fmt ? P.rc3 : P.rc8)[id] < 1)
      atomicOr(&s_err, (int)MKV_DEVERR_REFCOUNT);
  }
  __syncthreads();
  if (s_err) {
    if (tid == 0) atomicOr(&P.ctrl[CTRL_ERR], s_err);
    return;
  }
  for (int k = tid; k < n; k += blockDim.x) {
    int fmt;
    const int id = ids[k];
    (void)ref_of(tags[k], id, P.n_fp8, P.n_tq3, fmt);
    atomicAdd(&(fmt ? P.rc3 : P.rc8)[id], 1);
  }
}

// One workgroup.  Entries: an explicit list (reqs == nullptr: ids/tags[n]) or
// the rows of the listed requests (entry j * max_pages + p = row reqs[j], page
// p, mapped entries only).  Each entry drops one reference, in entry order: a
// page whose count reaches zero is pushed onto its free list at its last
// entry.  Pass 1 counts each page's entries and finds its last one (scratch
// occ / last, 0 / -1 at rest); a page with more entries than references, a
// bad tag or id, or a bad request list fails the call (scratch restored,
// nothing else changed).  Pass 2 walks the entries in order, ranks the
// freeing ones with a block scan and applies the counts; table rows are then
// unmapped.
__global__ __launch_bounds__(1024) void pages_release_kernel(int n, const int32_t* ids,
                                                             const uint8_t* tags, int n_fin,
                                                             const int32_t* reqs, int n_req,
                                                             int32_t* bt, uint8_t* bt_tags,
                                                             int max_pages, PoolView P) {
  __shared__ int scratch[32];
  __shared__ int s_err;
  const int tid = threadIdx.x;
  const bool table = reqs != nullptr;
  const int64_t N = table ? (int64_t)n_fin * max_pages : n;
  if (tid == 0) s_err = 0;
  __syncthreads();
  if (table) {
    for (int j = tid; j < n_fin; j += blockDim.x) {
      const int r = reqs[j];
      if (r < 0 || r >= n_req || (j > 0 && reqs[j - 1] >= r)) atomicOr(&s_err, (int)MKV_DEVERR_RANGE);
    }
    __syncthreads();
    if (s_err) {
      if (tid == 0) atomicOr(&P.ctrl[CTRL_ERR], s_err);
      return;
    }
  }
  // entry k -> (mapped, fmt, id); false for an unmapped table entry
  auto entry = [&](int64_t k, int& fmt, int& id, bool& ok) {
    uint8_t tg;
    if (table) {
      const int64_t i = (int64_t)reqs[k / max_pages] * max_pages + k % max_pages;
      id = bt[i];
      tg = bt_tags[i];
      if (id < 0) {
        ok = false;
        return false;
      }
    } else {
      id = ids[k];
      tg = tags[k];
    }
    ok = ref_of(tg, id, P.n_fp8, P.n_tq3, fmt);
    return true;
  };
  for (int64_t k = tid; k < N; k += blockDim.x) {
    int fmt, id;
    bool ok;
    if (!entry(k, fmt, id, ok)) continue;
    if (!ok) {
      atomicOr(&s_err, (int)MKV_DEVERR_REFCOUNT);
      continue;
    }
    atomicAdd(&(fmt ? P.occ3 : P.occ8)[id], 1);
    atomicMax(&(fmt ? P.last3 : P.last8)[id], (int)k);
  }
  __syncthreads();
  for (int64_t k = tid; k < N; k += blockDim.x) {
    int fmt, id;
    bool ok;
    if (!entry(k, fmt, id, ok) || !ok) continue;
    if ((fmt ? P.occ3 : P.occ8)[id] > (fmt ? P.rc3 : P.rc8)[id]) atomicOr(&s_err, (int)MKV_DEVERR_REFCOUNT);
  }
  __syncthreads();
  const int err = s_err;
  if (err) {
    for (int64_t k = tid; k < N; k += blockDim.x) {
      int fmt, id;
      bool ok;
      if (!entry(k, fmt, id, ok) || !ok) continue;
      (fmt ? P.occ3 : P.occ8)[id] = 0;
      (fmt ? P.last3 : P.last8)[id] = -1;
    }
    if (tid == 0) atomicOr(&P.ctrl[CTRL_ERR], err);
    return;
  }
  const int top8 = P.ctrl[CTRL_FP8_TOP], top3 = P.ctrl[CTRL_TQ3_TOP];
  int base8 = 0, base3 = 0;
  for (int64_t b0 = 0; b0 < N; b0 += blockDim.x) {
    const int64_t k = b0 + tid;
    int fmt = 0, id = 0;
    bool ok = false;
    bool last = false, freed = false;
    if (k < N && entry(k, fmt, id, ok) && ok) {
      int32_t* lastv = fmt ? P.last3 : P.last8;
      last = lastv[id] == (int)k;
      if (last) {
        int32_t* rc = fmt ? P.rc3 : P.rc8;
        int32_t* occ = fmt ? P.occ3 : P.occ8;
        const int left = rc[id] - occ[id];
        freed = left == 0;
        rc[id] = left;
        occ[id] = 0;
        lastv[id] = -1;
      }
    }
    // ranks of the freeing entries, FP8 in the low and TQ3 in the high half
    const int v = freed ? (fmt ? (1 << 16) : 1) : 0;
    int tot;
    const int pre = block_excl_scan(v, scratch, &tot);
    if (freed) {
      if (fmt) P.tq3_stack[top3 + base3 + (pre >> 16)] = id;
      else P.fp8_stack[top8 + base8 + (pre & 0xFFFF)] = id;
    }
    base8 += tot & 0xFFFF;
    base3 += tot >> 16;
  }
  __syncthreads();
  if (table)
    for (int64_t k = tid; k < N; k += blockDim.x) {
      const int64_t i = (int64_t)reqs[k / max_pages] * max_pages + k % max_pages;
      bt[i] = -1;
      bt_tags[i] = TAG_NONE;
    }
  if (tid == 0) {
    P.ctrl[CTRL_FP8_TOP] = top8 + base8;
    P.ctrl[CTRL_TQ3_TOP] = top3 + base3;
  }
}

hipError_t launch_pages_acquire(const PoolView& P, int n, const int32_t* ids, const uint8_t* tags,
                                hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(pages_acquire_kernel, dim3(1), dim3(1024), 0, s, n, ids, tags, P);
  return hipGetLastError();
}

hipError_t launch_pages_release(const PoolView& P, int n, const int32_t* ids, const uint8_t* tags,
                                int n_fin, const int32_t* reqs, int n_req, int32_t* bt,
                                uint8_t* bt_tags, int max_pages, hipStream_t s) {
  if ((reqs ? n_fin : n) == 0) return hipSuccess;
  hipLaunchKernelGGL(pages_release_kernel, dim3(1), dim3(1024), 0, s, n, ids, tags, n_fin, reqs,
                     n_req, bt, bt_tags, max_pages, P);
  return hipGetLastError();
}

// ===========================================================================
// Compact per-format page lists
// ===========================================================================
__global__ __launch_bounds__(1024) void partition_kernel(const int32_t* bt, const uint8_t* tags,
                                                         int max_pages, const int32_t* seq_lens,
                                                         int32_t* list8, int32_t* list3,
                                                         int32_t* counts, int32_t* err) {
  __shared__ int scratch[32];
  const int r = blockIdx.x, tid = threadIdx.x;
  const int S = seq_lens[r];
  const int np = (S + PAGE - 1) / PAGE;
  if (S < 1 || np > max_pages) {
    if (tid == 0) {
      counts[2 * r] = 0;
      counts[2 * r + 1] = 0;
      if (err) atomicOr(err, (int)MKV_DEVERR_RANGE);
    }
    return;
  }
  int b8 = 0, b3 = 0, bad = 0;
  for (int c0 = 0; c0 < np; c0 += blockDim.x) {
    const int p = c0 + tid;
    const int64_t i = (int64_t)r * max_pages + p;
    const int tg = p < np ? tags[i] : TAG_NONE;
    const int is8 = (p < np && (tg == TAG_R || tg == TAG_A)) ? 1 : 0;
    const int is3 = (p < np && tg == TAG_S) ? 1 : 0;
    if (p < np && !is8 && !is3) bad = 1;
    int t8, t3;
    const int r8 = block_excl_scan(is8, scratch, &t8);
    const int r3 = block_excl_scan(is3, scratch, &t3);
    if (is8) {
      list8[((int64_t)r * max_pages + b8 + r8) * 2] = p;
      list8[((int64_t)r * max_pages + b8 + r8) * 2 + 1] = bt[i];
    }
    if (is3) {
      list3[((int64_t)r * max_pages + b3 + r3) * 2] = p;
      list3[((int64_t)r * max_pages + b3 + r3) * 2 + 1] = bt[i];
    }
    b8 += t8;
    b3 += t3;
  }
  if (bad && err) atomicOr(err, (int)MKV_DEVERR_BAD_TAG);
  if (tid == 0) {
    counts[2 * r] = b8;
    counts[2 * r + 1] = b3;
  }
}

__global__ void fill_zero_kernel(uint32_t* p, int64_t n_words) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_words;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

// ===========================================================================
// Launchers
// ===========================================================================

hipError_t launch_append(const PoolView& P, int layer, int n_req, int32_t* bt, uint8_t* tags,
                         int max_pages, const int32_t* sb, const int32_t* cu, int n_new_total,
                         const uint16_t* k, const uint16_t* v, hipStream_t s) {
  const int n_lcall = layer < 0 ? P.n_layers : 1;
  // decode-step appends: one wave per task, as many waves as the call can have
  // tasks (every touched page receives at least one token)
  const int64_t step_waves = (int64_t)n_new_total * n_lcall * P.n_kv_heads * 2;
  if (n_new_total <= STEP_APPEND_MAX_TOKENS && n_req <= STEP_APPEND_MAX_REQ &&
      step_waves <= STEP_APPEND_MAX_WAVES) {
    const int grid = step_waves < 1 ? 1 : (int)step_waves;
    if (P.d == 256)
      hipLaunchKernelGGL(append_step_kernel<256>, dim3(grid), dim3(64), 0, s, P, layer, n_lcall,
                         n_req, bt, tags, max_pages, sb, cu, n_new_total, k, v);
    else
      hipLaunchKernelGGL(append_step_kernel<128>, dim3(grid), dim3(64), 0, s, P, layer, n_lcall,
                         n_req, bt, tags, max_pages, sb, cu, n_new_total, k, v);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(append_plan_kernel, dim3(1), dim3(1024), 0, s, n_req, bt, tags, max_pages, sb,
                     cu, P.ctrl, P.fp8_stack, P.list, P.n_fp8, n_new_total, P.rc8);
  // upper bound on listed pages: new tokens / 16 + one partial page per request
  const int64_t pages_bound = (int64_t)n_new_total / PAGE + n_req + 1;
  const int grid = grid_for((pages_bound * n_lcall * P.n_kv_heads * 2 + 3) / 4, 8192);
  if (P.d == 256)
    hipLaunchKernelGGL(append_quant_kernel<256>, dim3(grid), dim3(256), 0, s, P, layer, n_lcall, sb,
                       cu, n_new_total, k, v);
  else
    hipLaunchKernelGGL(append_quant_kernel<128>, dim3(grid), dim3(256), 0, s, P, layer, n_lcall, sb,
                       cu, n_new_total, k, v);
  return hipGetLastError();
}

hipError_t launch_migrate(const PoolView& P, int n_req, int32_t* bt, uint8_t* tags, int max_pages,
                          const uint8_t* anchor, const int32_t* seq_lens, hipStream_t s) {
  // whole batches per workgroup, at most MIG_BLOCKS workgroups
  const int64_t n_ent = (int64_t)n_req * max_pages;
  const int64_t n_bat = (n_ent + MIG_BATCH - 1) / MIG_BATCH;
  const int64_t bat_per = (n_bat + MIG_BLOCKS - 1) / MIG_BLOCKS;
  const int nb = (int)((n_bat + bat_per - 1) / bat_per);
  const int64_t per_blk = bat_per * MIG_BATCH;
  int32_t* mig = P.ctrl + ctrl_layout(P.n_fp8, P.n_tq3, P.d).mig;
  const RcView rv = {P.rc8, P.rc3, P.n_fp8, P.n_tq3};
  if (nb == 1) {
    hipLaunchKernelGGL(migrate_list_kernel<true>, dim3(1), dim3(MIG_NT), 0, s, n_req, bt, tags,
                       max_pages, anchor, seq_lens, P.recent, P.ctrl, P.tq3_stack, P.list, mig,
                       per_blk, nb, P.n_fp8, rv);
  } else {
    hipLaunchKernelGGL(migrate_count_kernel, dim3(nb), dim3(MIG_NT), 0, s, n_req, bt, tags,
                       max_pages, anchor, seq_lens, P.recent, P.ctrl, mig, per_blk, P.n_fp8, rv);
    hipLaunchKernelGGL(migrate_list_kernel<false>, dim3(nb), dim3(MIG_NT), 0, s, n_req, bt, tags,
                       max_pages, anchor, seq_lens, P.recent, P.ctrl, P.tq3_stack, P.list, mig,
                       per_blk, nb, P.n_fp8, rv);
  }
  int64_t bound = (int64_t)n_req * max_pages;
  if (bound > P.n_fp8) bound = P.n_fp8;
  const int grid = grid_for(bound * P.n_layers * P.n_kv_heads, 4096);
  if (P.d == 256)
    hipLaunchKernelGGL(migrate_encode_kernel<256>, dim3(grid), dim3(256), 0, s, P);
  else
    hipLaunchKernelGGL(migrate_encode_kernel<128>, dim3(grid), dim3(256), 0, s, P);
  hipLaunchKernelGGL(migrate_publish_kernel, dim3(1), dim3(1024), 0, s, bt, tags, max_pages, P.ctrl,
                     P.fp8_stack, P.list, P.rc8, P.rc3);
  return hipGetLastError();
}

hipError_t launch_promote(const PoolView& P, int n_req, int32_t* bt, uint8_t* tags, int max_pages,
                          const uint8_t* mask, const int32_t* seq_lens, hipStream_t s) {
  hipLaunchKernelGGL(promote_plan_kernel, dim3(1), dim3(MIG_NT), 0, s, n_req, bt, tags, max_pages,
                     mask, seq_lens, P.ctrl, P.fp8_stack, P.list, P.n_tq3,
                     RcView{P.rc8, P.rc3, P.n_fp8, P.n_tq3});
  int64_t bound = (int64_t)n_req * max_pages;
  if (bound > P.n_fp8) bound = P.n_fp8;
  if (bound > P.n_tq3) bound = P.n_tq3;
  const int grid = grid_for(bound * P.n_layers * P.n_kv_heads, 2048);
  if (P.d == 256)
    hipLaunchKernelGGL(promote_build_kernel<256>, dim3(grid), dim3(256), 0, s, P);
  else
    hipLaunchKernelGGL(promote_build_kernel<128>, dim3(grid), dim3(256), 0, s, P);
  hipLaunchKernelGGL(promote_publish_kernel, dim3(1), dim3(1024), 0, s, bt, tags, max_pages, P.ctrl,
                     P.tq3_stack, P.list, P.rc8, P.rc3);
  return hipGetLastError();
}

// Arithmetic conformance probe: the fp64 division, square root and binary16
// rounding of this translation unit (the ones gamma and the V scale/zero rest
// on), element by element.
__global__ __launch_bounds__(256) void fp64_probe_kernel(const double* a, const double* b, int64_t n,
                                                         double* quot, double* root,
                                                         uint16_t* half) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const double x = a[i], y = b[i];
    quot[i] = x / y;
    root[i] = sqrt(x);
    half[i] = f64_to_f16_rne_sat(x);
  }
}

hipError_t launch_fp64_probe(const double* a, const double* b, int64_t n, double* quot,
                             double* root, uint16_t* half, hipStream_t s) {
  hipLaunchKernelGGL(fp64_probe_kernel, dim3(grid_for((n + 255) / 256, 4096)), dim3(256), 0, s, a, b,
                     n, quot, root, half);
  return hipGetLastError();
}

hipError_t launch_partition(int n_req, const int32_t* bt, const uint8_t* tags, int max_pages,
                            const int32_t* seq_lens, int32_t* list8, int32_t* list3,
                            int32_t* counts, int32_t* err, hipStream_t s) {
  hipLaunchKernelGGL(partition_kernel, dim3(n_req), dim3(1024), 0, s, bt, tags, max_pages, seq_lens,
                     list8, list3, counts, err);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
  const int64_t words = (int64_t)(bytes / 4);
  if (words == 0) return hipSuccess;
  const int grid = grid_for((words + 255) / 256, 1024);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(grid), dim3(256), 0, s, (uint32_t*)p, words);
  return hipGetLastError();
}

}  // namespace mkv
