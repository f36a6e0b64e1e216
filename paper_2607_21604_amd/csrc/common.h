// Device helpers shared by the akvs kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/akvs.h"

typedef uint16_t bf16_t;  // bf16 bits as stored in memory
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_t;  // 16-byte load/store unit

namespace akvs {

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// fp32 -> bf16, round to nearest even (NaN stays NaN): the gfx950 packed conversion.
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
__device__ __forceinline__ uint32_t pack_bf2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}
__device__ __forceinline__ bf16_t f2bf(float f) { return (bf16_t)(pack_bf2(f, 0.f) & 0xffffu); }

// ---- 8-element vector access for the two storage types -----------------------------
__device__ __forceinline__ void load8(const float *p, float (&o)[8]) {
  const float4 a = *reinterpret_cast<const float4 *>(p);
  const float4 b = *reinterpret_cast<const float4 *>(p + 4);
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
  o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}
__device__ __forceinline__ void load8(const bf16_t *p, float (&o)[8]) {
  const uint4 v = *reinterpret_cast<const uint4 *>(p);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = __uint_as_float(w[i] << 16);
    o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void store8(float *p, const float (&o)[8]) {
  *reinterpret_cast<float4 *>(p) = make_float4(o[0], o[1], o[2], o[3]);
  *reinterpret_cast<float4 *>(p + 4) = make_float4(o[4], o[5], o[6], o[7]);
}
__device__ __forceinline__ void store8(bf16_t *p, const float (&o)[8]) {
  uint4 v;
  v.x = pack_bf2(o[0], o[1]);
  v.y = pack_bf2(o[2], o[3]);
  v.z = pack_bf2(o[4], o[5]);
  v.w = pack_bf2(o[6], o[7]);
  *reinterpret_cast<uint4 *>(p) = v;
}
__device__ __forceinline__ void store4(float *p, float a, float b, float c, float d) {
  *reinterpret_cast<float4 *>(p) = make_float4(a, b, c, d);
}
__device__ __forceinline__ void store4(bf16_t *p, float a, float b, float c, float d) {
  uint2 v;
  v.x = pack_bf2(a, b);
  v.y = pack_bf2(c, d);
  *reinterpret_cast<uint2 *>(p) = v;
}
__device__ __forceinline__ float load1(const float *p) { return *p; }
__device__ __forceinline__ float load1(const bf16_t *p) { return bf2f(*p); }
__device__ __forceinline__ void store1(float *p, float v) { *p = v; }
__device__ __forceinline__ void store1(bf16_t *p, float v) { *p = f2bf(v); }

// ---- wave64 reductions (fixed butterfly order: deterministic) ------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, 64));
  return v;
}

// ---- unit-cache reader: plain (f32 / bf16) or group-64 quantised ----------------------
// One layer of a cache: rows of [Hkv][hd] per token, token-major.
struct CacheLayer {
  const void *k, *v;
  const _Float16 *k_meta, *v_meta;
  int dtype;  // AKVS_F32 / AKVS_BF16 / AKVS_U4G64 / AKVS_U2G64 / AKVS_E4M3G64
};

// Four E4M3 bytes of w, decoded by the gfx950 conversion (OCP FP8 E4M3), times scale.
__device__ __forceinline__ void e4m3x4(uint32_t w, float scale, float *o) {
  const f32x2_t a = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, false);
  const f32x2_t b = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, true);
  o[0] = a[0] * scale;
  o[1] = a[1] * scale;
  o[2] = b[0] * scale;
  o[3] = b[1] * scale;
}

// 8 consecutive elements e0..e0+7 (e0 % 8 == 0) of row `row` (= token*Hkv + head).
__device__ __forceinline__ void cache_load8(const void *base, const _Float16 *meta, int dtype,
                                            size_t row, int hd, int e0, float (&o)[8]) {
  if (dtype == AKVS_BF16) {
    load8(reinterpret_cast<const bf16_t *>(base) + row * hd + e0, o);
  } else if (dtype == AKVS_F32) {
    load8(reinterpret_cast<const float *>(base) + row * hd + e0, o);
  } else {
    const size_t g = row * (size_t)(hd / 64) + (size_t)(e0 / 64);
    const float scale = (float)meta[2 * g];
    const float zero = (float)meta[2 * g + 1];
    if (dtype == AKVS_E4M3G64) {
      const uint2 w = *reinterpret_cast<const uint2 *>(reinterpret_cast<const uint8_t *>(base) +
                                                       row * hd + e0);
      e4m3x4(w.x, scale, o);
      e4m3x4(w.y, scale, o + 4);
    } else if (dtype == AKVS_U4G64) {
      const uint8_t *c = reinterpret_cast<const uint8_t *>(base) + row * (hd / 2) + e0 / 2;
      const uint32_t w = *reinterpret_cast<const uint32_t *>(c);
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = fmaf(scale, (float)((w >> (4 * i)) & 15u), zero);
    } else {
      const uint8_t *c = reinterpret_cast<const uint8_t *>(base) + row * (hd / 4) + e0 / 4;
      const uint32_t w = *reinterpret_cast<const uint16_t *>(c);
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = fmaf(scale, (float)((w >> (2 * i)) & 3u), zero);
    }
  }
}

__device__ __forceinline__ float cache_load1(const void *base, const _Float16 *meta, int dtype,
                                             size_t row, int hd, int e) {
  if (dtype == AKVS_BF16) return bf2f(reinterpret_cast<const bf16_t *>(base)[row * hd + e]);
  if (dtype == AKVS_F32) return reinterpret_cast<const float *>(base)[row * hd + e];
  const size_t g = row * (size_t)(hd / 64) + (size_t)(e / 64);
  const float scale = (float)meta[2 * g];
  const float zero = (float)meta[2 * g + 1];
  const uint8_t *c = reinterpret_cast<const uint8_t *>(base);
  if (dtype == AKVS_E4M3G64)
    return __builtin_amdgcn_cvt_pk_f32_fp8((int)c[row * hd + e], false)[0] * scale;
  uint32_t code;
  if (dtype == AKVS_U4G64)
    code = (c[row * (hd / 2) + e / 2] >> (4 * (e & 1))) & 15u;
  else
    code = (c[row * (hd / 4) + e / 4] >> (2 * (e & 3))) & 3u;
  return fmaf(scale, (float)code, zero);
}

}  // namespace akvs
