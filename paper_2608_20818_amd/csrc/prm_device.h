// Device helpers shared by the libprm kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "prm_internal.h"

namespace prm {

// ---- bf16 <-> fp32 ---------------------------------------------------------
__device__ __forceinline__ float bf2f(uint32_t h) { return __uint_as_float(h << 16); }

// fp32 -> bf16, round to nearest with ties to even (gfx950 v_cvt_pk_bf16_f32).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  bf16x2_t h = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, h);
}

__device__ __forceinline__ uint32_t f2bf(float f) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f);
}

// ---- global-memory addressing ------------------------------------------------
// Every buffer the helpers below touch (caller tensors, workspace) is global
// memory.  Addressing it through address space 1 lets the compiler emit
// global_* instructions (scalar base + vector offset, vmcnt only) instead of
// flat_* ones, which also count against lgkmcnt and must be assumed to alias
// LDS.
#define PRM_GLOBAL __attribute__((address_space(1)))
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
template <typename T>
__device__ __forceinline__ PRM_GLOBAL T* gptr(T* p) { return (PRM_GLOBAL T*)p; }
template <typename T>
__device__ __forceinline__ const PRM_GLOBAL T* gptr(const T* p) { return (const PRM_GLOBAL T*)p; }

// ---- typed loads / stores of 4 or 8 consecutive elements --------------------
// Element storage type T is either float or uint16_t (bf16 bits).
template <typename T> struct Vec;

template <> struct Vec<float> {
  __device__ __forceinline__ static void load4(const float* p, float v[4]) {
    const f32x4_t x = *gptr(reinterpret_cast<const f32x4_t*>(p));
    v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
  }
  __device__ __forceinline__ static void store4(float* p, const float v[4]) {
    const f32x4_t x = {v[0], v[1], v[2], v[3]};
    *gptr(reinterpret_cast<f32x4_t*>(p)) = x;
  }
  __device__ __forceinline__ static void load8(const float* p, float v[8]) {
    load4(p, v);
    load4(p + 4, v + 4);
  }
  __device__ __forceinline__ static void store8(float* p, const float v[8]) {
    store4(p, v);
    store4(p + 4, v + 4);
  }
  __device__ __forceinline__ static float load1(const float* p) { return *gptr(p); }
  __device__ __forceinline__ static void store1(float* p, float v) { *gptr(p) = v; }
};

template <> struct Vec<uint16_t> {
  __device__ __forceinline__ static void load4(const uint16_t* p, float v[4]) {
    const u32x2_t x = *gptr(reinterpret_cast<const u32x2_t*>(p));
    v[0] = bf2f(x[0] & 0xffffu); v[1] = bf2f(x[0] >> 16);
    v[2] = bf2f(x[1] & 0xffffu); v[3] = bf2f(x[1] >> 16);
  }
  __device__ __forceinline__ static void store4(uint16_t* p, const float v[4]) {
    const u32x2_t x = {pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3])};
    *gptr(reinterpret_cast<u32x2_t*>(p)) = x;
  }
  __device__ __forceinline__ static void load8(const uint16_t* p, float v[8]) {
    const u32x4_t x = *gptr(reinterpret_cast<const u32x4_t*>(p));
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      v[2 * k] = bf2f(x[k] & 0xffffu);
      v[2 * k + 1] = bf2f(x[k] >> 16);
    }
  }
  __device__ __forceinline__ static void store8(uint16_t* p, const float v[8]) {
    const u32x4_t x = {pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]),
                       pack_bf2(v[6], v[7])};
    *gptr(reinterpret_cast<u32x4_t*>(p)) = x;
  }
  __device__ __forceinline__ static float load1(const uint16_t* p) { return bf2f(*gptr(p)); }
  __device__ __forceinline__ static void store1(uint16_t* p, float v) { *gptr(p) = (uint16_t)f2bf(v); }
};

// ---- streaming (nontemporal) variants for data touched once per step ---------
// Same interface as Vec; the loads and stores carry the nontemporal hint so that
// the single pass over G, M and W does not displace cached operands.

template <typename T> struct VecNT;

template <> struct VecNT<float> {
  __device__ __forceinline__ static void load4(const float* p, float v[4]) {
    const f32x4_t x = __builtin_nontemporal_load(gptr(reinterpret_cast<const f32x4_t*>(p)));
    v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
  }
  __device__ __forceinline__ static void store4(float* p, const float v[4]) {
    const f32x4_t x = {v[0], v[1], v[2], v[3]};
    __builtin_nontemporal_store(x, gptr(reinterpret_cast<f32x4_t*>(p)));
  }
  __device__ __forceinline__ static void load8(const float* p, float v[8]) {
    load4(p, v);
    load4(p + 4, v + 4);
  }
  __device__ __forceinline__ static void store8(float* p, const float v[8]) {
    store4(p, v);
    store4(p + 4, v + 4);
  }
  __device__ __forceinline__ static float load1(const float* p) { return __builtin_nontemporal_load(gptr(p)); }
  __device__ __forceinline__ static void store1(float* p, float v) { __builtin_nontemporal_store(v, gptr(p)); }
};

template <> struct VecNT<uint16_t> {
  __device__ __forceinline__ static void load4(const uint16_t* p, float v[4]) {
    const u32x2_t x = __builtin_nontemporal_load(gptr(reinterpret_cast<const u32x2_t*>(p)));
    v[0] = bf2f(x[0] & 0xffffu); v[1] = bf2f(x[0] >> 16);
    v[2] = bf2f(x[1] & 0xffffu); v[3] = bf2f(x[1] >> 16);
  }
  __device__ __forceinline__ static void store4(uint16_t* p, const float v[4]) {
    const u32x2_t x = {pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3])};
    __builtin_nontemporal_store(x, gptr(reinterpret_cast<u32x2_t*>(p)));
  }
  __device__ __forceinline__ static void load8(const uint16_t* p, float v[8]) {
    const u32x4_t x = __builtin_nontemporal_load(gptr(reinterpret_cast<const u32x4_t*>(p)));
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      v[2 * k] = bf2f(x[k] & 0xffffu);
      v[2 * k + 1] = bf2f(x[k] >> 16);
    }
  }
  __device__ __forceinline__ static void store8(uint16_t* p, const float v[8]) {
    const u32x4_t x = {pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]),
                       pack_bf2(v[6], v[7])};
    __builtin_nontemporal_store(x, gptr(reinterpret_cast<u32x4_t*>(p)));
  }
  __device__ __forceinline__ static float load1(const uint16_t* p) {
    return bf2f(__builtin_nontemporal_load(gptr(p)));
  }
  __device__ __forceinline__ static void store1(uint16_t* p, float v) {
    __builtin_nontemporal_store((uint16_t)f2bf(v), gptr(p));
  }
};

// ---- reductions (fixed order: deterministic run to run) ---------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Sum over a whole workgroup of NT threads (NT a multiple of 64, <= 1024).
// `red` must hold NT/64 floats.  Every thread gets the total.
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  if constexpr (NT == 64) {
    return v;
  } else {
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < NT / 64; ++i) t += red[i];
    return t;
  }
}

// Binary search: index of the last segment whose start <= b.
__device__ __forceinline__ int find_segment(const int32_t* start, int n, int b) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (start[mid] <= b) lo = mid; else hi = mid - 1;
  }
  return lo;
}

}  // namespace prm
