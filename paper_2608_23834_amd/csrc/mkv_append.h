// FP8 append of a few tokens to one page-head by one wave: the task shared by
// the decode-step append kernel and the decode call that appends its token
// (Alg. 1, Append; FP8 scale and requantization as Sec. 3.1 reads).  Slots
// [0, t0) of the page-head already hold codes with the page's scale; the new
// bf16 rows land in [t0, t1); when their amax exceeds 448 times the scale the
// scale grows and the old codes are re-rounded through a 256-entry table.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mkv_device.h"
#include "mkv_internal.h"

namespace mkv {

// byte offset of (K or V, token t, channel c) in an FP8 page-head region
template <int D>
__device__ __forceinline__ int fp8_off(int kv, int t, int c) {
  if (!kv) return t * D + c;
  constexpr int CL = D / 16;
  const int r = c / CL, m = c % CL, g = t >> 2, u = t & 3;
  return PAGE * D + ((r * 4 + g) * CL + m) * 4 + u;
}

template <int D>
struct SmallTask {
  static constexpr int D4 = D / 4, NC = PAGE * D4 / 64, NV = PAGE * D / (16 * 64);
  int r, p, row0, t0, t1, layer, li, h, kv;
  uint2 x[NC];
  uint4 old[NV];
  float s_old;
  bool have_old;
};

template <int D>
__device__ __forceinline__ void small_task_load_x(SmallTask<D>& T, int H, int n_new_total,
                                                  const uint16_t* k, const uint16_t* v, int lane) {
  constexpr int D4 = SmallTask<D>::D4;
  const uint16_t* src = (T.kv ? v : k) + (int64_t)T.li * n_new_total * H * D;
  const uint16_t* srow = src + ((int64_t)T.row0 * H + T.h) * D;  // token t at srow[t * H * D + c]
  const int64_t tstride = (int64_t)H * D;
  const int n4 = (T.t1 - T.t0) * D4;
#pragma unroll
  for (int j = 0; j < SmallTask<D>::NC; ++j) {
    const int idx = (threadIdx.x & 63) + 64 * j;
    T.x[j] = make_uint2(0u, 0u);
    if (idx < n4) {
      const int t = T.t0 + idx / D4, c = 4 * (idx % D4);
      T.x[j] = *reinterpret_cast<const uint2*>(srow + t * tstride + c);
    }
  }
  (void)lane;
}

// codes and scale of page-head (T.layer, id, T.h), part T.kv; only a page with
// tokens below t0 has any
template <int D>
__device__ __forceinline__ void small_task_load_old(SmallTask<D>& T, const PoolView& P, int id,
                                                    int lane) {
  T.have_old = T.t0 > 0;
  T.s_old = 0.0f;
  if (!T.have_old) return;
  const int64_t ph = ((int64_t)T.layer * P.n_fp8 + id) * P.n_kv_heads + T.h;
  const uint4* reg = reinterpret_cast<const uint4*>(P.fp8 + ph * fp8_region_bytes(D) + T.kv * PAGE * D);
#pragma unroll
  for (int j = 0; j < SmallTask<D>::NV; ++j) T.old[j] = reg[lane + 64 * j];
  T.s_old = P.fp8_scales[ph * 2 + T.kv];
}

template <int D>
__device__ void small_task_run(SmallTask<D>& T, const PoolView& P, int id, uint32_t* img,
                               uint8_t* lut, int lane) {
#pragma clang fp contract(off)  // single IEEE operations in order, as in the oracle
  constexpr int D4 = SmallTask<D>::D4, NC = SmallTask<D>::NC, NV = SmallTask<D>::NV;
  const int t0 = T.t0, t1 = T.t1;
  const int n4 = (t1 - t0) * D4;
  float amax = 0.0f;
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    amax = fmaxf(amax, fmaxf(fmaxf(fabsf(__uint_as_float(T.x[j].x << 16)),
                                   fabsf(__uint_as_float(T.x[j].x & 0xFFFF0000u))),
                             fmaxf(fabsf(__uint_as_float(T.x[j].y << 16)),
                                   fabsf(__uint_as_float(T.x[j].y & 0xFFFF0000u)))));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
  const float s_old = T.s_old;
  float s_new = s_old;
  bool requant = false;
  if (t0 == 0) {
    s_new = amax / 448.0f;
  } else if (!(amax <= 448.0f * s_old)) {
    s_new = amax / 448.0f;
    requant = true;
  }
  // old codes (zeros for a page without tokens below t0), re-rounded through
  // a table when the scale grows, into the LDS block
  uint4 o[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) o[j] = T.have_old ? T.old[j] : make_uint4(0u, 0u, 0u, 0u);
  if (requant) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t c = (uint32_t)(lane + 64 * i);
      lut[c] = (uint8_t)f32_to_e4m3((e4m3_to_f32(c) * s_old) / s_new);
    }
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      uint32_t* ow = reinterpret_cast<uint32_t*>(&o[j]);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int w = 4 * (lane + 64 * j) + q;  // word of the block
        uint32_t outw = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          // token of byte b: K rows are token-major, V words hold tokens 4g .. 4g+3
          const int t = T.kv ? 4 * ((w / (D / 16)) % 4) + b : w / D4;
          const uint32_t code = (ow[q] >> (8 * b)) & 0xFFu;
          const uint32_t nc = lut[code];
          outw |= (t < t0 ? nc : code) << (8 * b);
        }
        ow[q] = outw;
      }
    }
  }
#pragma unroll
  for (int j = 0; j < NV; ++j) reinterpret_cast<uint4*>(img)[lane + 64 * j] = o[j];
  __builtin_amdgcn_wave_barrier();
  // new codes over the block
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int idx = lane + 64 * j;
    if (idx < n4) {
      const int t = t0 + idx / D4, c = 4 * (idx % D4);
      uint32_t code[4];
      const uint32_t hv[4] = {T.x[j].x << 16, T.x[j].x & 0xFFFF0000u, T.x[j].y << 16,
                              T.x[j].y & 0xFFFF0000u};
#pragma unroll
      for (int b = 0; b < 4; ++b)
        code[b] = s_new > 0.0f ? f32_to_e4m3(__uint_as_float(hv[b]) / s_new) : 0u;
      if (!T.kv) {
        img[(t * D + c) / 4] = code[0] | (code[1] << 8) | (code[2] << 16) | (code[3] << 24);
      } else {
        uint8_t* ib = reinterpret_cast<uint8_t*>(img);
#pragma unroll
        for (int b = 0; b < 4; ++b) ib[fp8_off<D>(1, t, c + b) - PAGE * D] = (uint8_t)code[b];
      }
    }
    __builtin_amdgcn_sched_barrier(0);  // one item at a time: bounded register use
  }
  __builtin_amdgcn_wave_barrier();
  const int64_t ph = ((int64_t)T.layer * P.n_fp8 + id) * P.n_kv_heads + T.h;
  uint4* reg = reinterpret_cast<uint4*>(P.fp8 + ph * fp8_region_bytes(D) + T.kv * PAGE * D);
#pragma unroll
  for (int j = 0; j < NV; ++j) reg[lane + 64 * j] = reinterpret_cast<const uint4*>(img)[lane + 64 * j];
  if (lane == 0) P.fp8_scales[ph * 2 + T.kv] = s_new;
  __builtin_amdgcn_wave_barrier();  // the block and table are free for the wave's next task
}

// Inclusive prefix sum over the wave's lanes.
__device__ __forceinline__ int wave_incl_scan(int x, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}
__device__ __forceinline__ int wave_or(int x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x |= __shfl_xor(x, o, 64);
  return x;
}

}  // namespace mkv
