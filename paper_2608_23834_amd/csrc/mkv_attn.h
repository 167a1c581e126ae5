// Device helpers shared by the decode and chunk attention kernels: MFMA
// operand assembly, code conversions, direct HBM -> LDS copies with explicit
// vmcnt gating, and VALU cross-lane exchanges (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mkv_device.h"

namespace mkv {

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
// code bytes 0..7 -> fp16 0..7: each byte read as an E4M3 subnormal (c * 2^-9)
// and scaled by 2^9 in the converter, exactly
template <bool HI>
__device__ __forceinline__ half2v cvt_code(uint32_t w) {
  return __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 512.0f, HI);
}
__device__ __forceinline__ float exp2_safe(float s, float m) {
  return s == -INFINITY ? 0.0f : exp2f(s - m);
}

// Direct HBM -> LDS copies issued by one wave.  dma16<OFF>: lane l copies
// 16 bytes from base + voff_l + OFF to LDS m0 + OFF + 16 l; dma4<OFF>: 4 bytes
// to m0 + OFF + 4 l (the immediate offset applies to both addresses; base and
// m0 are wave-uniform).  They are inline assembly on purpose: the compiler
// then does not order later LDS reads behind them (it cannot tell which ring
// slot a copy fills and would wait for all of them), and the caller gates
// every stage with an explicit vmcnt wait.  The kernel has no other user of m0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"  // m0 is reserved; no compiler code here uses it
template <int OFF>
__device__ __forceinline__ void dma16(uint32_t voff, const uint8_t* base, uint32_t m0) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 offset:%3"
               :
               : "v"(voff), "s"(base), "s"(m0), "n"(OFF)
               : "memory", "m0");
}
__device__ __forceinline__ void dma4(uint32_t voff, const uint8_t* base, uint32_t m0) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1 offset:0"
               :
               : "v"(voff), "s"(base), "s"(m0)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// Per-lane byte offsets of the copies (constant for the kernel).
struct DmaLanes {
  uint32_t lo, hi;  // 16 l and 4096 + 16 l
};
// One region of R bytes (16-byte aligned, R <= 8 KiB + 256): whole KiB blocks
// by 16-byte lanes, the tail by 4-byte lanes.
template <int R>
__device__ __forceinline__ void dma_region(uint32_t dst, const uint8_t* src, const DmaLanes& dl,
                                           int lane) {
  static_assert(R <= 8192 + 256, "region too large for the offset scheme");
#pragma unroll
  for (int i = 0; i < R / 1024 && i < 4; ++i) {
    switch (i) {
      case 0: dma16<0>(dl.lo, src, dst); break;
      case 1: dma16<1024>(dl.lo, src, dst); break;
      case 2: dma16<2048>(dl.lo, src, dst); break;
      default: dma16<3072>(dl.lo, src, dst); break;
    }
  }
#pragma unroll
  for (int i = 4; i < R / 1024; ++i) {
    switch (i) {
      case 4: dma16<0>(dl.hi, src, dst + 4096); break;
      case 5: dma16<1024>(dl.hi, src, dst + 4096); break;
      case 6: dma16<2048>(dl.hi, src, dst + 4096); break;
      default: dma16<3072>(dl.hi, src, dst + 4096); break;
    }
  }
  constexpr int TAIL = R % 1024;
  static_assert(TAIL % 4 == 0 && TAIL <= 256, "tail must fit one 4-byte copy");
  if (TAIL > 0 && lane < TAIL / 4) dma4((R - TAIL) + 4 * lane, src, dst + (R - TAIL));
}
// One FP8 page-head (K then V, 16 d bytes each) into LDS with its 16-byte
// blocks permuted so that the MFMA lanes read it without bank conflicts: LDS
// block 64 w + l of each half holds the w-th 16 bytes of what lane l = 16 lg +
// ln consumes (K: token ln, channels (d/4) lg + 16 w ..; V: the lane-chunk
// (ln, lg), bytes 16 w ..).  2 d / 64 copies; the caller adds the scales.
template <int D>
__device__ __forceinline__ void dma_fp8_page(uint32_t dst, const uint8_t* src, int lane) {
  constexpr int NI = D / 64;  // copies per half (16 d / 1024)
  const int ln = lane & 15, lg = lane >> 4;
  const uint32_t vk = 16u * (uint32_t)(ln * (D / 16) + lg * NI);
  const uint32_t vv = 16u * (uint32_t)((ln * 4 + lg) * NI);
#pragma unroll
  for (int i = 0; i < NI; ++i) dma16<0>(vk, src + 16 * i, dst + 1024 * i);
#pragma unroll
  for (int i = 0; i < NI; ++i) dma16<0>(vv, src + 16 * D + 16 * i, dst + 16 * D + 1024 * i);
}

// The code dwords of chunk idx of a TQ3 code block in LDS (8-byte reads when
// the chunk size allows).
template <int NDW>
__device__ __forceinline__ void read_chunk(uint32_t* dst, const uint8_t* block, int idx) {
  constexpr int CB = 4 * NDW;
  if constexpr (CB % 8 == 0) {
    const uint2* p = reinterpret_cast<const uint2*>(block + idx * CB);
#pragma unroll
    for (int w = 0; w < NDW / 2; ++w) {
      const uint2 x = p[w];
      dst[2 * w] = x.x;
      dst[2 * w + 1] = x.y;
    }
  } else {
    const uint32_t* p = reinterpret_cast<const uint32_t*>(block + idx * CB);
#pragma unroll
    for (int w = 0; w < NDW; ++w) dst[w] = p[w];
  }
}

// vector-memory instructions dma_region<R> issues per wave
template <int R>
constexpr int dma_ops() { return R / 1024 + (R % 1024 ? 1 : 0); }

// Wait until at most N vector-memory operations of this wave are in flight
// (gfx9 s_waitcnt: vmcnt in bits [3:0] and [15:14]; expcnt/lgkmcnt left free).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
  __asm__ __volatile__("" ::: "memory");
}
__device__ __forceinline__ void wait_lgkm0() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0), vmcnt/expcnt free
  __asm__ __volatile__("" ::: "memory");
}

// Cross-lane exchanges on the VALU (gfx950 permlane swaps).  With both operands
// x, v_permlane16_swap yields (rows 0,0,2,2 ; rows 1,1,3,3) of x (a row is 16
// lanes) and v_permlane32_swap yields (low half twice ; high half twice).
__device__ __forceinline__ uint2 swap16(float x) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return make_uint2(p[0], p[1]);
}
__device__ __forceinline__ uint2 swap32(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return make_uint2(p[0], p[1]);
}
// max / sum over the four lanes l, l ^ 16, l ^ 32, l ^ 48
__device__ __forceinline__ float max4rows(float x) {
  uint2 p = swap16(x);
  x = fmaxf(__uint_as_float(p.x), __uint_as_float(p.y));
  p = swap32(x);
  return fmaxf(__uint_as_float(p.x), __uint_as_float(p.y));
}
__device__ __forceinline__ float sum4rows(float x) {
  uint2 p = swap16(x);
  x = __uint_as_float(p.x) + __uint_as_float(p.y);
  p = swap32(x);
  return __uint_as_float(p.x) + __uint_as_float(p.y);
}
// value of lane l ^ M, on the VALU: DPP within rows (quad_perm for 1 and 2,
// half-row mirror then quad reverse for 4, row rotate by 8 for 8) and the
// permlane swaps across rows
template <int M>
__device__ __forceinline__ float lane_xor(float x, int lane) {
  const int xi = __float_as_int(x);
  if constexpr (M == 1) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(xi, 0xB1, 0xF, 0xF, false));
  } else if constexpr (M == 2) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(xi, 0x4E, 0xF, 0xF, false));
  } else if constexpr (M == 4) {
    const int t = __builtin_amdgcn_mov_dpp(xi, 0x141, 0xF, 0xF, false);
    return __int_as_float(__builtin_amdgcn_mov_dpp(t, 0x1B, 0xF, 0xF, false));
  } else if constexpr (M == 8) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(xi, 0x128, 0xF, 0xF, false));
  } else if constexpr (M == 16) {
    const uint2 p = swap16(x);
    return __uint_as_float((lane & 16) ? p.x : p.y);
  } else {
    static_assert(M == 32, "lane_xor: M is a power of two below 64");
    const uint2 p = swap32(x);
    return __uint_as_float((lane & 32) ? p.x : p.y);
  }
}
// value of lane l + 32 (valid in lanes l < 32)
__device__ __forceinline__ float upper_half(float x) { return __uint_as_float(swap32(x).y); }

}  // namespace mkv
