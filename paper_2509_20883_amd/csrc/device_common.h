// Device helpers shared by the kernel files: bf16 conversion, wave / block
// scans, 16-byte row-fragment loads and stores, launch-size arithmetic.
#pragma once

#include "rs_internal.h"

namespace rs {

// ---------------------------------------------------------------------------
// small device helpers
// ---------------------------------------------------------------------------

__device__ inline float bf16_to_f32(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

// Round to nearest, ties to even; NaN -> 0x7FC0.
__device__ inline uint16_t f32_to_bf16(float x) {
  const uint32_t b = __float_as_uint(x);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu) != 0u) return 0x7FC0;
  return static_cast<uint16_t>((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

__device__ inline int wave_incl_scan(int v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int t = __shfl_up(v, d, kWave);
    if (lane >= d) v += t;
  }
  return v;
}

__device__ inline int wave_sum(int v) {
#pragma unroll
  for (int d = kWave / 2; d > 0; d >>= 1) v += __shfl_xor(v, d, kWave);
  return v;
}

// Exclusive block scan of one int per thread; `sh` holds NT/64 + 1 ints.
template <int NT>
__device__ inline int block_excl_scan(int v, int* sh, int& total) {
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  const int inc = wave_incl_scan(v);
  if (lane == kWave - 1) sh[wid] = inc;
  __syncthreads();
  if (wid == 0) {  // one wave scans the per-wave totals
    static_assert(NT / kWave <= kWave, "one wave scans the per-wave totals");
    const int t = lane < NT / kWave ? sh[lane] : 0;
    const int i2 = wave_incl_scan(t);
    if (lane < NT / kWave) sh[lane] = i2 - t;
    if (lane == kWave - 1) sh[NT / kWave] = i2;
  }
  __syncthreads();
  const int ex = sh[wid] + inc - v;
  total = sh[NT / kWave];
  __syncthreads();
  return ex;
}

template <int NT>
__device__ inline int block_sum(int v, int* sh) {
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  v = wave_sum(v);
  if (lane == 0) sh[wid] = v;
  __syncthreads();
  int t = 0;
  if (wid == 0) t = wave_sum(lane < NT / kWave ? sh[lane] : 0);
  return t;  // valid in thread 0
}

// 8 consecutive int32 starting at p[i0] (i0 % 8 == 0), zero past n.
__device__ inline void load8(const int32_t* __restrict__ p, int64_t i0, int64_t n, int (&v)[8]) {
  if (i0 + 8 <= n) {
    const int4 a = *reinterpret_cast<const int4*>(p + i0);
    const int4 b = *reinterpret_cast<const int4*>(p + i0 + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = (i0 + k < n) ? p[i0 + k] : 0;
  }
}

// E fp32 values from a 16-byte-aligned row fragment of type T (f32 or bf16).
template <typename T, int E>
__device__ inline void load_vals(const T* __restrict__ p, float (&v)[E]);

template <>
__device__ inline void load_vals<float, 4>(const float* __restrict__ p, float (&v)[4]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
}
template <>
__device__ inline void load_vals<float, 8>(const float* __restrict__ p, float (&v)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
template <>
__device__ inline void load_vals<uint16_t, 8>(const uint16_t* __restrict__ p, float (&v)[8]) {
  const uint4 a = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[2 * k] = __uint_as_float(w[k] << 16);
    v[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
  }
}
template <>
__device__ inline void load_vals<uint16_t, 4>(const uint16_t* __restrict__ p, float (&v)[4]) {
  const uint2 a = *reinterpret_cast<const uint2*>(p);
  v[0] = __uint_as_float(a.x << 16);
  v[1] = __uint_as_float(a.x & 0xFFFF0000u);
  v[2] = __uint_as_float(a.y << 16);
  v[3] = __uint_as_float(a.y & 0xFFFF0000u);
}

// The 16 bytes of a row fragment as raw bits, and their E fp32 values: a
// batch of loads is issued as raw loads first and widened afterwards, so no
// load waits for the one before it (a widening inside a conditional load
// would make the compiler wait for each load in turn).
__device__ inline uint4 load_raw16(const void* __restrict__ p) { return *reinterpret_cast<const uint4*>(p); }

template <typename T, int E>
__device__ inline void widen16(const uint4& a, float (&v)[E]);

template <>
__device__ inline void widen16<float, 4>(const uint4& a, float (&v)[4]) {
  v[0] = __uint_as_float(a.x);
  v[1] = __uint_as_float(a.y);
  v[2] = __uint_as_float(a.z);
  v[3] = __uint_as_float(a.w);
}
template <>
__device__ inline void widen16<uint16_t, 8>(const uint4& a, float (&v)[8]) {
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[2 * k] = __uint_as_float(w[k] << 16);
    v[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
  }
}

template <typename T, int E>
__device__ inline void store_vals(T* __restrict__ p, const float (&v)[E]);

template <>
__device__ inline void store_vals<float, 4>(float* __restrict__ p, const float (&v)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
template <>
__device__ inline void store_vals<float, 8>(float* __restrict__ p, const float (&v)[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
template <>
__device__ inline void store_vals<uint16_t, 8>(uint16_t* __restrict__ p, const float (&v)[8]) {
  uint4 a;
  a.x = static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
  a.y = static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
  a.z = static_cast<uint32_t>(f32_to_bf16(v[4])) | (static_cast<uint32_t>(f32_to_bf16(v[5])) << 16);
  a.w = static_cast<uint32_t>(f32_to_bf16(v[6])) | (static_cast<uint32_t>(f32_to_bf16(v[7])) << 16);
  *reinterpret_cast<uint4*>(p) = a;
}
template <>
__device__ inline void store_vals<uint16_t, 4>(uint16_t* __restrict__ p, const float (&v)[4]) {
  uint2 a;
  a.x = static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
  a.y = static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
  *reinterpret_cast<uint2*>(p) = a;
}

// The same stores, non-temporal, for rows and optimizer state written by an
// update: nothing reads them again in the step, and the lines leave the
// caches at once instead of being written back under the next kernel.
typedef float nt_f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t nt_u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t nt_u32x2 __attribute__((ext_vector_type(2)));

template <typename T, int E>
__device__ inline void store_vals_nt(T* __restrict__ p, const float (&v)[E]);

template <>
__device__ inline void store_vals_nt<float, 4>(float* __restrict__ p, const float (&v)[4]) {
  const nt_f32x4 a = {v[0], v[1], v[2], v[3]};
  __builtin_nontemporal_store(a, reinterpret_cast<nt_f32x4*>(p));
}
template <>
__device__ inline void store_vals_nt<float, 8>(float* __restrict__ p, const float (&v)[8]) {
  const nt_f32x4 a = {v[0], v[1], v[2], v[3]};
  const nt_f32x4 b = {v[4], v[5], v[6], v[7]};
  __builtin_nontemporal_store(a, reinterpret_cast<nt_f32x4*>(p));
  __builtin_nontemporal_store(b, reinterpret_cast<nt_f32x4*>(p + 4));
}
template <>
__device__ inline void store_vals_nt<uint16_t, 8>(uint16_t* __restrict__ p, const float (&v)[8]) {
  nt_u32x4 a;
#pragma unroll
  for (int k = 0; k < 4; ++k)
    a[k] = static_cast<uint32_t>(f32_to_bf16(v[2 * k])) | (static_cast<uint32_t>(f32_to_bf16(v[2 * k + 1])) << 16);
  __builtin_nontemporal_store(a, reinterpret_cast<nt_u32x4*>(p));
}
template <>
__device__ inline void store_vals_nt<uint16_t, 4>(uint16_t* __restrict__ p, const float (&v)[4]) {
  nt_u32x2 a;
#pragma unroll
  for (int k = 0; k < 2; ++k)
    a[k] = static_cast<uint32_t>(f32_to_bf16(v[2 * k])) | (static_cast<uint32_t>(f32_to_bf16(v[2 * k + 1])) << 16);
  __builtin_nontemporal_store(a, reinterpret_cast<nt_u32x2*>(p));
}

// Four int32 to a 16-byte-aligned p in one non-temporal store (per-id
// results that no kernel reads soon).
__device__ inline void store4_nt(int32_t* p, int a, int b, int c, int d) {
  const nt_u32x4 v = {static_cast<uint32_t>(a), static_cast<uint32_t>(b), static_cast<uint32_t>(c),
                      static_cast<uint32_t>(d)};
  __builtin_nontemporal_store(v, reinterpret_cast<nt_u32x4*>(p));
}

inline unsigned grid_for(int64_t work_items, int64_t per_block, int64_t cap = 1 << 20) {
  int64_t g = (work_items + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return static_cast<unsigned>(g);
}


}  // namespace rs
