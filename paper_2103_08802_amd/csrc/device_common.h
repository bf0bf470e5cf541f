// Device-side helpers for gfx950: storage-type traits, bf16 rounding, MFMA wrappers and the
// grouped-launch problem lookup.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pnn_internal.h"

namespace pnn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// bf16 <-> f32.  f32 -> bf16 rounds to nearest even (gfx950 v_cvt_pk_bf16_f32).
__device__ __forceinline__ float bf2f(uint16_t u) { return __uint_as_float((uint32_t)u << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) {
  __bf16 b = (__bf16)f;
  return __builtin_bit_cast(uint16_t, b);
}

// Storage traits: T is the in-memory element (float or uint16_t holding bf16 bits).
template <typename T> struct St;
template <> struct St<float> {
  static constexpr int VE = 4;  // elements per 16-byte chunk
  __device__ static __forceinline__ float ld(const void* p, long i) { return ((const float*)p)[i]; }
  __device__ static __forceinline__ void st(void* p, long i, float v) { ((float*)p)[i] = v; }
  __device__ static __forceinline__ float rnd(float v) { return v; }   // value as stored
};
template <> struct St<uint16_t> {
  static constexpr int VE = 8;
  __device__ static __forceinline__ float ld(const void* p, long i) { return bf2f(((const uint16_t*)p)[i]); }
  __device__ static __forceinline__ void st(void* p, long i, float v) { ((uint16_t*)p)[i] = f2bf(v); }
  __device__ static __forceinline__ float rnd(float v) { return bf2f(f2bf(v)); }
};

// One 16-byte operand chunk per lane, unpacked to floats.
template <typename T>
struct Chunk {
  float v[St<T>::VE];
};

template <typename T>
__device__ __forceinline__ void unpack_chunk(uint4 u, Chunk<T>& c) {
  if constexpr (sizeof(T) == 4) {
    c.v[0] = __uint_as_float(u.x);
    c.v[1] = __uint_as_float(u.y);
    c.v[2] = __uint_as_float(u.z);
    c.v[3] = __uint_as_float(u.w);
  } else {
    uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      c.v[2 * e] = __uint_as_float(w[e] << 16);
      c.v[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
  }
}

template <typename T>
__device__ __forceinline__ void load_chunk(const void* base, long idx, Chunk<T>& c) {
  unpack_chunk<T>(*(const uint4*)((const T*)base + idx), c);
}

template <typename T>
__device__ __forceinline__ void store_chunk(void* base, long idx, const float* v) {
  if constexpr (sizeof(T) == 4) {
    *(float4*)((float*)base + idx) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    uint4 u;
    u.x = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
    u.y = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
    u.z = (uint32_t)f2bf(v[4]) | ((uint32_t)f2bf(v[5]) << 16);
    u.w = (uint32_t)f2bf(v[6]) | ((uint32_t)f2bf(v[7]) << 16);
    *(uint4*)((uint16_t*)base + idx) = u;
  }
}

// MFMA fragment: the lane's 16 bytes of an A or B operand.
template <typename T> struct Frag;
template <> struct Frag<uint16_t> {
  bf16x8 v;
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (__bf16)0.0f;
  }
  __device__ __forceinline__ void from_raw(uint4 u) { v = __builtin_bit_cast(bf16x8, u); }
  __device__ __forceinline__ void from_chunk(const Chunk<uint16_t>& c) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (__bf16)c.v[e];
  }
};
template <> struct Frag<float> {
  float v[4];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = 0.0f;
  }
  __device__ __forceinline__ void from_raw(uint4 u) {
    v[0] = __uint_as_float(u.x);
    v[1] = __uint_as_float(u.y);
    v[2] = __uint_as_float(u.z);
    v[3] = __uint_as_float(u.w);
  }
  __device__ __forceinline__ void from_chunk(const Chunk<float>& c) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = c.v[e];
  }
};

// acc += A(16 x KS) * B(KS x 16) for one K step of the lane-chunk layout: lane l supplies row / col
// (l & 15) and the K elements [VE*(l>>4), VE*(l>>4)+VE) of the step.  bf16: one
// v_mfma_f32_16x16x32_bf16 (KS = 32).  f32: four v_mfma_f32_16x16x4f32 (KS = 16); MFMA e takes
// element e of every lane's chunk, so each MFMA sums a different interleaved quarter of K.
__device__ __forceinline__ void mma(const Frag<uint16_t>& a, const Frag<uint16_t>& b, f32x4& acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(const Frag<float>& a, const Frag<float>& b, f32x4& acc) {
#pragma unroll
  for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[e], b.v[e], acc, 0, 0, 0);
}

// Problem of this workgroup in a grouped launch: the last p whose first workgroup is <= blockIdx.x,
// by binary search.  With the table, the search reads one line of it (16 problems per 64 bytes)
// where a search over the problem records misses the scalar cache at every step.
template <typename Launch>
__device__ __forceinline__ int find_group(const Launch& L) {
  const int t = blockIdx.x;
  if constexpr (HasTb<Launch>::value) {
    int lo = 0, hi = L.tb[0] - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (L.tb[mid] <= t) lo = mid;
      else hi = mid - 1;
    }
    return lo;
  } else {
    int lo = 0, hi = L.n - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (L.p[mid].tile_begin <= t) lo = mid;
      else hi = mid - 1;
    }
    return lo;
  }
}

// x / d and x % d for a divisor given with log2(d) (>= 0) or as a plain value (lg < 0)
__device__ __forceinline__ int div_l2(int x, int d, int lg) { return lg >= 0 ? (x >> lg) : x / d; }

// q = x / d, r = x % d for 0 <= x < 2^22 and 0 < d < 2^22, with rd = 1.0f / d: the float quotient
// is within one of the true one and the remainder check corrects it.
__device__ __forceinline__ void divmod_small(int x, int d, float rd, int& q, int& r) {
  q = (int)((float)x * rd);
  r = x - q * d;
  if (r < 0) { --q; r += d; }
  else if (r >= d) { ++q; r -= d; }
}

// (r, s) of tap t of a k x k filter, k in {1, 3}
__device__ __forceinline__ void tap_rs(int t, int k, int& r, int& s) {
  r = (k == 3) ? ((t * 11) >> 5) : 0;
  s = t - r * k;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Device-coherent 8-byte accesses for data that workgroups of one launch exchange (BN partial rows,
// their folds): agent-scope relaxed atomics, i.e. plain loads / stores with the coherence bit, so
// every XCD sees them without the writeback and invalidate of its whole L2 that a device-scope
// fence costs.  Ordering: the writer's waves wait for their own stores (wait_mem) before the
// barrier and counter update that publish them; the readers load after observing the counter.
__device__ __forceinline__ void st_coherent(float2* p, float2 v) {
  __hip_atomic_store((unsigned long long*)p, __builtin_bit_cast(unsigned long long, v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_coherent(const float2* p) {
  return __builtin_bit_cast(float2, __hip_atomic_load((unsigned long long*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ void st_coherent(double* p, double v) {
  __hip_atomic_store((unsigned long long*)p, __builtin_bit_cast(unsigned long long, v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double ld_coherent(const double* p) {
  return __builtin_bit_cast(double, __hip_atomic_load((unsigned long long*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
// the wave's memory operations complete (its coherent stores have reached the device-wide level)
__device__ __forceinline__ void wait_mem() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}


}  // namespace pnn
