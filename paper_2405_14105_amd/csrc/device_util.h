// Device helpers: bf16 conversion, hi/lo split, MFMA wrappers, fragment
// loads and pack stores.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace dsi {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// fp32 -> bf16 bits, round to nearest even (finite inputs)
__device__ __forceinline__ uint16_t f2bf_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf_bits2f(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// split x into bf16 hi + bf16 lo with x ~= hi + lo (to ~2^-17 relative)
__device__ __forceinline__ void split_bf16(float x, uint16_t& hi, uint16_t& lo) {
  hi = f2bf_bits(x);
  lo = f2bf_bits(x - bf_bits2f(hi));
}

__device__ __forceinline__ f32x4 mfma_bf16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_f32(float a, float b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& v) {
  return __builtin_bit_cast(bf16x8, v);
}

// 8 fp32 values (two 16-byte loads)
struct F8 {
  float4 a, b;
};
__device__ __forceinline__ float f8_get(const F8& v, int e) {
  switch (e) {
    case 0: return v.a.x; case 1: return v.a.y; case 2: return v.a.z; case 3: return v.a.w;
    case 4: return v.b.x; case 5: return v.b.y; case 6: return v.b.z; default: return v.b.w;
  }
}

// store one activation value into a pack at (token m, feature f)
__device__ __forceinline__ size_t pack_index(int Kb, int m, int f) {
  const int mt = m >> 4, kb = f >> 5, grp = (f & 31) >> 3, e = f & 7;
  const int lane = (m & 15) + 16 * grp;
  return (((size_t)mt * Kb + kb) * 64 + lane) * 8 + e;
}
__device__ __forceinline__ void pack_store(const PackRef& p, int wtype, int m, int f, float v) {
  const size_t idx = pack_index(p.Kb, m, f);
  if (wtype == W_BF16) {
    uint16_t hi, lo;
    split_bf16(v, hi, lo);
    ((uint16_t*)p.hi)[idx] = hi;
    ((uint16_t*)p.lo)[idx] = lo;
  } else {
    ((float*)p.hi)[idx] = v;
  }
}

// store 4 consecutive features f0..f0+3 (f0 % 4 == 0) of token m: 8 bytes
// per half for bf16 packs, 16 bytes for fp32 packs
__device__ __forceinline__ void pack_store4(const PackRef& p, int wtype, int m, int f0, const float* v) {
  const size_t idx = pack_index(p.Kb, m, f0);
  if (wtype == W_BF16) {
    uint16_t hi[4], lo[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) split_bf16(v[e], hi[e], lo[e]);
    *(uint2*)((uint16_t*)p.hi + idx) = uint2{(uint32_t)hi[0] | ((uint32_t)hi[1] << 16),
                                             (uint32_t)hi[2] | ((uint32_t)hi[3] << 16)};
    *(uint2*)((uint16_t*)p.lo + idx) = uint2{(uint32_t)lo[0] | ((uint32_t)lo[1] << 16),
                                             (uint32_t)lo[2] | ((uint32_t)lo[3] << 16)};
  } else {
    *(float4*)((float*)p.hi + idx) = float4{v[0], v[1], v[2], v[3]};
  }
}

// store 8 consecutive features f0..f0+7 (f0 % 8 == 0) of token m: one
// 16-byte store per half for bf16 packs, two for fp32 packs
__device__ __forceinline__ void pack_store8(const PackRef& p, int wtype, int m, int f0, const float* v) {
  const size_t idx = pack_index(p.Kb, m, f0);
  if (wtype == W_BF16) {
    uint16_t hi[8], lo[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) split_bf16(v[e], hi[e], lo[e]);
    u32x4 h, l;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      h[e] = (uint32_t)hi[2 * e] | ((uint32_t)hi[2 * e + 1] << 16);
      l[e] = (uint32_t)lo[2 * e] | ((uint32_t)lo[2 * e + 1] << 16);
    }
    *(u32x4*)((uint16_t*)p.hi + idx) = h;
    *(u32x4*)((uint16_t*)p.lo + idx) = l;
  } else {
    float* d = (float*)p.hi + idx;
    *(float4*)d = float4{v[0], v[1], v[2], v[3]};
    *(float4*)(d + 4) = float4{v[4], v[5], v[6], v[7]};
  }
}

// Device-scope (sc1) 16-byte store: written through to the device's
// coherence point, for partial results that another workgroup of the same
// kernel reads with device-scope loads after an arrival counter says they
// are complete (the writer waits for vmcnt(0) before counting).  One wide
// store instead of four device-scope dword stores.
__device__ __forceinline__ void store4_device(float* p, f32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1" ::"v"(p), "v"(v) : "memory");
}

__device__ __forceinline__ float silu_f(float x) { return x / (1.0f + __expf(-x)); }

}  // namespace dsi
