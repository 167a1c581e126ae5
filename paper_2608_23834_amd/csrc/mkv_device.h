// Device-side helpers shared by the Minima-KV gfx950 kernels: physical page
// layouts, FP8 E4M3 / binary16 conversions, the TQ3 code layout and MFMA
// operand types.  Layout definitions follow the pool description in
// include/minima_kv.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mkv {

constexpr int PAGE = 16;
constexpr int TAG_R = 0, TAG_A = 1, TAG_S = 2, TAG_NONE = 0xFF;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float float4v __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float float16v __attribute__((ext_vector_type(16)));

// ---------------------------------------------------------------------------
// ctrl buffer (int32 words): counters, free stacks, work list, rotation signs.
// ---------------------------------------------------------------------------
enum CtrlSlot {
  CTRL_FP8_TOP = 0,
  CTRL_TQ3_TOP = 1,
  CTRL_ERR = 2,
  CTRL_NLIST = 3,
  CTRL_ABORT = 4,
  CTRL_APPEND_ARRIVE = 5,  // waves of a decode-step append that have finished (reset by the last)
  CTRL_HEADER = 64
};
constexpr int MIG_BLOCKS = 256;  // most workgroups of a migration plan
struct CtrlLayout {
  int64_t fp8_stack, tq3_stack, list, sigma_bytes, mig, rc8, rc3, occ8, occ3, last8, last3,
      total_words;
};
// mig: migration-plan scratch, per-workgroup counts [MIG_BLOCKS], per-workgroup
// error bits [MIG_BLOCKS], the TQ3 free-list top the plan started from.
// rc8 / rc3: references per FP8 / TQ3 page (0: free).  occ* / last*: release
// scratch per page (occurrences in the call, last list index), 0 / -1 at rest.
__host__ __device__ inline CtrlLayout ctrl_layout(int n_fp8, int n_tq3, int d) {
  CtrlLayout c;
  c.fp8_stack = CTRL_HEADER;
  c.tq3_stack = c.fp8_stack + n_fp8;
  c.list = c.tq3_stack + n_tq3;
  c.sigma_bytes = (c.list + 4LL * n_fp8) * 4;  // byte offset of int8 sigma[d]
  c.mig = c.list + 4LL * n_fp8 + (d + 3) / 4;
  c.rc8 = c.mig + 2LL * MIG_BLOCKS + 1;
  c.rc3 = c.rc8 + n_fp8;
  c.occ8 = c.rc3 + n_tq3;
  c.occ3 = c.occ8 + n_fp8;
  c.last8 = c.occ3 + n_tq3;
  c.last3 = c.last8 + n_fp8;
  c.total_words = c.last3 + n_tq3;
  return c;
}

// ---------------------------------------------------------------------------
// Page layouts (per layer, physical page, KV head).
//  FP8 region: 2*16*d bytes.  K at [t*d + c] (token-major).  V in lane-chunk
//  order: with CL = d/16, r = c/CL, m = c%CL, g = t/4, u = t%4 the V byte of
//  (t, c) is at 16*d + ((r*4 + g)*CL + m)*4 + u.
//  TQ3 region: 16*d + 32 bytes: K codes [0, 6d), V codes [6d, 12d), gamma
//  fp16[16] at 12d, V scale fp16[d] at 12d+32, V zero fp16[d] at 14d+32.
//  Codes live in "chunks" of 3d/32 bytes holding d/16 quads of 4 codes:
//   K chunk (t, g) at (g*16+t)*3d/32: quad q, position b = channel d/4*g+4q+b
//   V chunk (r, g) at (g*16+r)*3d/32: quad q = channel CL*r+q, position b =
//   token 4g+b.  Chunks are ordered g-major: the 16 lanes of an MFMA row
//   group read chunks 16g .. 16g+15, contiguous in LDS, without bank conflicts.
//  Within a chunk of n_dw = 3d/128 dwords, quad q < 2*n_dw occupies bits
//  [8b + 3(q%2), +3) of dword q/2; the remaining quads use bits 6-7 of every
//  byte (see quad_sel below).
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int64_t fp8_region_bytes(int d) { return 2LL * PAGE * d; }
__host__ __device__ constexpr int64_t tq3_region_bytes(int d) { return 16LL * d + 32; }
__host__ __device__ constexpr int chunk_bytes(int d) { return 3 * d / 32; }

// Byte selector of the 4 codes of quad q (one code in the low 3 bits of each
// byte) from the chunk's dwords D[].
template <int NDW>
__device__ __forceinline__ uint32_t quad_sel(const uint32_t* D, int q) {
  if (q < 2 * NDW) {
    return (D[q >> 1] >> (3 * (q & 1))) & 0x07070707u;
  }
  int e = q - 2 * NDW, p = e >> 1;
  if ((e & 1) == 0)
    return ((D[3 * p] >> 6) & 0x03030303u) | ((D[3 * p + 1] >> 4) & 0x04040404u);
  return ((D[3 * p + 1] >> 7) & 0x01010101u) | ((D[3 * p + 2] >> 5) & 0x06060606u);
}

// Inverse of quad_sel: OR the 3-bit code into the chunk dwords.
template <int NDW>
__device__ __forceinline__ void quad_put(uint32_t* D, int q, int b, uint32_t code) {
  if (q < 2 * NDW) {
    D[q >> 1] |= code << (8 * b + 3 * (q & 1));
    return;
  }
  int e = q - 2 * NDW, p = e >> 1;
  if ((e & 1) == 0) {
    D[3 * p] |= (code & 3u) << (8 * b + 6);
    D[3 * p + 1] |= ((code >> 2) & 1u) << (8 * b + 6);
  } else {
    D[3 * p + 1] |= (code & 1u) << (8 * b + 7);
    D[3 * p + 2] |= ((code >> 1) & 3u) << (8 * b + 6);
  }
}

// TQ3 codebook levels as E4M3 bytes, code 0..7 ascending:
// -2.25, -1.375, -0.75, -0.25, 0.25, 0.75, 1.375, 2.25
constexpr uint32_t KLUT_LO = 0xA8B4BBC1u, KLUT_HI = 0x413B3428u;
// integers 0..7 as E4M3 bytes (value codes)
constexpr uint32_t VLUT_LO = 0x44403800u, VLUT_HI = 0x4E4C4A48u;
// 64 * level^2 per code
__device__ __forceinline__ int mu2x64(int c) {
  const int t[8] = {324, 121, 36, 4, 4, 36, 121, 324};
  return t[c];
}

// ---------------------------------------------------------------------------
// Scalar conversions
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}
// E4M3 value of a byte (exact).
__device__ __forceinline__ float e4m3_to_f32(uint32_t byte) {
  return __builtin_amdgcn_cvt_f32_fp8((int)byte, 0);
}
// fp32 -> E4M3, nearest-even, saturating at +-448 (the hardware conversion
// does not saturate, so clamp first).
__device__ __forceinline__ uint32_t f32_to_e4m3(float x) {
  x = fminf(fmaxf(x, -448.0f), 448.0f);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(x, 0.0f, 0, false) & 0xFFu;
}
// E4M3 byte times 512 as an exact integer.
__device__ __forceinline__ int32_t e4m3_times_512(uint32_t b) {
  int e = (b >> 3) & 15, m = b & 7;
  int32_t v = e ? ((8 + m) << (e - 1)) : m;
  return (b & 0x80u) ? -v : v;
}

// fp64 -> binary16, round to nearest even, saturating at +-65504 (stored
// metadata stays finite).  Method: pick the binary16 quantum 2^e of |x| (the
// spacing of binary16 numbers in |x|'s binade, never below the subnormal
// quantum 2^-24), scale |x| by 2^-e -- exact, a power of two -- and round that
// once to an integer m with rint (the default mode is ties-to-even).  m is the
// binary16 significand; m = 2048 means the rounding carried into the next
// binade.  One rounding, no intermediate format.
__device__ inline uint16_t f64_to_f16_rne_sat(double x) {
  const uint32_t sign = signbit(x) ? 0x8000u : 0u;
  const double ax = fabs(x);
  if (isnan(x)) return (uint16_t)(sign | 0x7E00u);
  if (ax >= 65504.0) return (uint16_t)(sign | 0x7BFFu);  // largest finite binary16
  if (ax == 0.0) return (uint16_t)sign;
  int bexp;
  (void)frexp(ax, &bexp);            // ax in [2^(bexp-1), 2^bexp)
  const int e = max(bexp - 11, -24);  // quantum: 11 significant bits, subnormals below 2^-14
  double m = rint(ldexp(ax, -e));     // 0 <= m <= 2048
  int ee = e;
  if (m == 2048.0) {  // carried into the next binade
    m = 1024.0;
    ee += 1;
  }
  const uint32_t mi = (uint32_t)m;
  if (mi < 1024u) return (uint16_t)(sign | mi);  // subnormal (ee = -24) or zero
  const uint32_t biased = (uint32_t)(ee + 25);   // value = mi * 2^ee, mi in [1024, 2048)
  return (uint16_t)(sign | (biased << 10) | (mi - 1024u));
}
__device__ __forceinline__ double f16_bits_to_f64(uint16_t h) {
  _Float16 v = __builtin_bit_cast(_Float16, h);
  return (double)v;
}

// ---------------------------------------------------------------------------
// Block-wide helpers (blockDim.x threads, wave64)
// ---------------------------------------------------------------------------
// Exclusive prefix sum of one int per thread; returns the prefix, writes the
// total to *total.  Uses scratch[blockDim.x/64 + 1] ints of LDS.
__device__ inline int block_excl_scan(int v, int* scratch, int* total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) scratch[wid] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int w = 0; w < nw; ++w) {
      int t = scratch[w];
      scratch[w] = acc;
      acc += t;
    }
    scratch[nw] = acc;
  }
  __syncthreads();
  int res = scratch[wid] + x - v;
  *total = scratch[nw];
  __syncthreads();
  return res;
}

__device__ inline int block_sum(int v, int* scratch) {
  int tot;
  block_excl_scan(v, scratch, &tot);
  return tot;
}

}  // namespace mkv
