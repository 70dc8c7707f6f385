// Device-side helpers shared by the SPLA kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "spla_layout.h"

namespace spla {

constexpr int kWave = 64;

// bfloat16 is carried as its raw 16 bits.
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// Round to nearest, ties to even; NaN stays NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T> struct Elem;
// store4: elements i .. i + 3 in one store (i a multiple of 4).
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float* p, int64_t i) { return p[i]; }
  static __device__ __forceinline__ void store(float* p, int64_t i, float v) { p[i] = v; }
  static __device__ __forceinline__ void store4(float* p, int64_t i, const float (&v)[4]) {
    *reinterpret_cast<float4*>(p + i) = make_float4(v[0], v[1], v[2], v[3]);
  }
};
template <> struct Elem<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t* p, int64_t i) {
    return bf16_to_f32(p[i].bits);
  }
  static __device__ __forceinline__ void store(bf16_t* p, int64_t i, float v) {
    p[i].bits = f32_to_bf16(v);
  }
  static __device__ __forceinline__ void store4(bf16_t* p, int64_t i, const float (&v)[4]) {
    const uint32_t a = f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
    const uint32_t b = f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
    *reinterpret_cast<uint2*>(p + i) = make_uint2(a, b);
  }
};

// ---- lane exchanges without LDS: lane l receives lane l ^ 32 / l ^ 16 (the
// gfx950 permlane swaps; 1-D workgroups, so lane = threadIdx.x % 64).
__device__ __forceinline__ uint32_t lane_xor32(uint32_t x) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return (threadIdx.x & 32) ? r[0] : r[1];
}
__device__ __forceinline__ uint32_t lane_xor16(uint32_t x) {
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  return (threadIdx.x & 16) ? r[0] : r[1];
}
__device__ __forceinline__ float xor32(float x) { return __uint_as_float(lane_xor32(__float_as_uint(x))); }
// Reduce-scatter steps with one swap and no selects. half_sum(a, b): lanes
// 0..31 get a(l) + a(l + 32), lanes 32..63 get b(l - 32) + b(l);
// row_pair_sum(a, b): lanes of even 16-lane rows get a(l) + a(l + 16),
// lanes of odd rows b(l - 16) + b(l). The permlane swaps exchange exactly
// the halves (rows) that the other side needs.
__device__ __forceinline__ double half_sum(double a, double b) {
  const uint64_t ua = __double_as_longlong(a), ub = __double_as_longlong(b);
  const auto lo = __builtin_amdgcn_permlane32_swap((uint32_t)ua, (uint32_t)ub, false, false);
  const auto hi =
      __builtin_amdgcn_permlane32_swap((uint32_t)(ua >> 32), (uint32_t)(ub >> 32), false, false);
  return __longlong_as_double((long long)(((uint64_t)hi[0] << 32) | lo[0])) +
         __longlong_as_double((long long)(((uint64_t)hi[1] << 32) | lo[1]));
}
__device__ __forceinline__ double row_pair_sum(double a, double b) {
  const uint64_t ua = __double_as_longlong(a), ub = __double_as_longlong(b);
  const auto lo = __builtin_amdgcn_permlane16_swap((uint32_t)ua, (uint32_t)ub, false, false);
  const auto hi =
      __builtin_amdgcn_permlane16_swap((uint32_t)(ua >> 32), (uint32_t)(ub >> 32), false, false);
  return __longlong_as_double((long long)(((uint64_t)hi[0] << 32) | lo[0])) +
         __longlong_as_double((long long)(((uint64_t)hi[1] << 32) | lo[1]));
}

__device__ __forceinline__ float xor16(float x) { return __uint_as_float(lane_xor16(__float_as_uint(x))); }
__device__ __forceinline__ double xor32(double x) {
  const uint64_t u = __double_as_longlong(x);
  const uint64_t lo = lane_xor32((uint32_t)u), hi = lane_xor32((uint32_t)(u >> 32));
  return __longlong_as_double((long long)((hi << 32) | lo));
}
__device__ __forceinline__ double xor16(double x) {
  const uint64_t u = __double_as_longlong(x);
  const uint64_t lo = lane_xor16((uint32_t)u), hi = lane_xor16((uint32_t)(u >> 32));
  return __longlong_as_double((long long)((hi << 32) | lo));
}

// Rotations inside 16-lane rows and quad permutes (DPP).
template <int CTRL>
__device__ __forceinline__ float dpp_rot(float x) {
  return __uint_as_float((uint32_t)__builtin_amdgcn_update_dpp(0, (int)__float_as_uint(x), CTRL,
                                                               0xF, 0xF, false));
}

// Sum / max over the wavefront; every lane gets the same bits (each step
// combines a value with its partner's, and + / max commute).
__device__ __forceinline__ float wave_sum(float v) {
  v += xor32(v);
  v += xor16(v);
  v += dpp_rot<0x128>(v);  // row_ror:8
  v += dpp_rot<0x124>(v);  // row_ror:4
  v += dpp_rot<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_rot<0xB1>(v);   // quad_perm [1,0,3,2]
  return v;
}
// The same over each half-wavefront (lanes 0..31, 32..63) on its own.
__device__ __forceinline__ float half_wave_sum(float v) {
  v += xor16(v);
  v += dpp_rot<0x128>(v);
  v += dpp_rot<0x124>(v);
  v += dpp_rot<0x4E>(v);
  v += dpp_rot<0xB1>(v);
  return v;
}
__device__ __forceinline__ float half_wave_max(float v) {
  v = fmaxf(v, xor16(v));
  v = fmaxf(v, dpp_rot<0x128>(v));
  v = fmaxf(v, dpp_rot<0x124>(v));
  v = fmaxf(v, dpp_rot<0x4E>(v));
  v = fmaxf(v, dpp_rot<0xB1>(v));
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, xor32(v));
  v = fmaxf(v, xor16(v));
  v = fmaxf(v, dpp_rot<0x128>(v));
  v = fmaxf(v, dpp_rot<0x124>(v));
  v = fmaxf(v, dpp_rot<0x4E>(v));
  v = fmaxf(v, dpp_rot<0xB1>(v));
  return v;
}

// ---- wavefront scans on DPP: shifts inside 16-lane rows, then the row
// broadcasts of lanes 15 and 31. No LDS traffic; lane 63 ends with the total.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t old, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROW_MASK, 0xF, false);
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_f64(double old, double v) {
  const uint64_t o = __double_as_longlong(old), x = __double_as_longlong(v);
  const uint32_t lo = dpp_u32<CTRL, ROW_MASK>((uint32_t)o, (uint32_t)x);
  const uint32_t hi = dpp_u32<CTRL, ROW_MASK>((uint32_t)(o >> 32), (uint32_t)(x >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Inclusive prefix sum over lanes 0 .. l.
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t x) {
  x += dpp_u32<0x111, 0xF>(0u, x);  // row_shr:1
  x += dpp_u32<0x112, 0xF>(0u, x);  // row_shr:2
  x += dpp_u32<0x114, 0xF>(0u, x);  // row_shr:4
  x += dpp_u32<0x118, 0xF>(0u, x);  // row_shr:8
  x += dpp_u32<0x142, 0xA>(0u, x);  // row_bcast:15 into rows 1, 3
  x += dpp_u32<0x143, 0xC>(0u, x);  // row_bcast:31 into rows 2, 3
  return x;
}

__device__ __forceinline__ uint32_t lane_u32(uint32_t v, int lane) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}
__device__ __forceinline__ float lane_f32(float v, int lane) {
  return __uint_as_float(lane_u32(__float_as_uint(v), lane));
}
__device__ __forceinline__ double lane_f64(double v, int lane) {
  const uint64_t x = __double_as_longlong(v);
  const uint32_t lo = lane_u32((uint32_t)x, lane), hi = lane_u32((uint32_t)(x >> 32), lane);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Wave-uniform sum / max of doubles (fixed association order).
__device__ __forceinline__ double wave_sum_u(double x) {
  x += dpp_f64<0x111, 0xF>(0.0, x);
  x += dpp_f64<0x112, 0xF>(0.0, x);
  x += dpp_f64<0x114, 0xF>(0.0, x);
  x += dpp_f64<0x118, 0xF>(0.0, x);
  x += dpp_f64<0x142, 0xA>(0.0, x);
  x += dpp_f64<0x143, 0xC>(0.0, x);
  return lane_f64(x, 63);
}
__device__ __forceinline__ double wave_max_u(double x) {
  x = fmax(x, dpp_f64<0x111, 0xF>(-INFINITY, x));
  x = fmax(x, dpp_f64<0x112, 0xF>(-INFINITY, x));
  x = fmax(x, dpp_f64<0x114, 0xF>(-INFINITY, x));
  x = fmax(x, dpp_f64<0x118, 0xF>(-INFINITY, x));
  x = fmax(x, dpp_f64<0x142, 0xA>(-INFINITY, x));
  x = fmax(x, dpp_f64<0x143, 0xC>(-INFINITY, x));
  return lane_f64(x, 63);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_f32(float old, float v) {
  return __uint_as_float(dpp_u32<CTRL, ROW_MASK>(__float_as_uint(old), __float_as_uint(v)));
}

// Max / sum over the 16 lanes of this lane's DPP row (row_shr steps); lane
// 15 of each row ends with the result.
__device__ __forceinline__ float row_max_to15(float x) {
  x = fmaxf(x, dpp_f32<0x111, 0xF>(-INFINITY, x));
  x = fmaxf(x, dpp_f32<0x112, 0xF>(-INFINITY, x));
  x = fmaxf(x, dpp_f32<0x114, 0xF>(-INFINITY, x));
  x = fmaxf(x, dpp_f32<0x118, 0xF>(-INFINITY, x));
  return x;
}
__device__ __forceinline__ double row_sum_to15(double x) {
  x += dpp_f64<0x111, 0xF>(0.0, x);
  x += dpp_f64<0x112, 0xF>(0.0, x);
  x += dpp_f64<0x114, 0xF>(0.0, x);
  x += dpp_f64<0x118, 0xF>(0.0, x);
  return x;
}

// ---- memory access policy of data that one workgroup hands to another
// within a launch. Mem<false>: ordinary loads and stores (the data crosses a
// kernel boundary). Mem<true>: agent-scope atomic loads and stores, which
// the compiler emits with the device-coherence bit (sc1): they write through
// and read past the per-XCD L2 caches, so no cache-wide writeback or
// invalidation is needed between producer and consumer.
template <bool CO>
struct Mem;
constexpr int kCacheSc1 = 16;  // cache-policy operand of the buffer intrinsics: sc1
// ld16(base, off): the 16 bytes at byte offset off (16-byte aligned) of a
// wave-uniform base. Mem<true> issues it as one buffer load with the sc1
// bit (agent-scope atomics are at most 8 bytes wide).
template <>
struct Mem<false> {
  static __device__ __forceinline__ uint4 ld16(const void* base, uint32_t off) {
    return *reinterpret_cast<const uint4*>(static_cast<const char*>(base) + off);
  }
  template <typename T>
  static __device__ __forceinline__ T ld(const T* p) { return *p; }
  template <typename T>
  static __device__ __forceinline__ void st(T* p, T v) { *p = v; }
  static __device__ __forceinline__ float2 ld2(const float* p) {
    return *reinterpret_cast<const float2*>(p);
  }
  static __device__ __forceinline__ float4 ld4(const float* p) {
    return *reinterpret_cast<const float4*>(p);
  }
};
template <>
struct Mem<true> {
  static __device__ __forceinline__ uint4 ld16(const void* base, uint32_t off) {
    // raw buffer over the 4 GiB above base (dword 3: the gfx9 data format)
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, -1, 0x00020000);
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCacheSc1);
    return make_uint4(v[0], v[1], v[2], v[3]);
  }
  template <typename T>
  static __device__ __forceinline__ T ld(const T* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  template <typename T>
  static __device__ __forceinline__ void st(T* p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  static __device__ __forceinline__ float2 ld2(const float* p) {  // 8-byte aligned
    const uint64_t u = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
    return make_float2(__uint_as_float((uint32_t)u), __uint_as_float((uint32_t)(u >> 32)));
  }
  static __device__ __forceinline__ float4 ld4(const float* p) {  // 16-byte aligned
    const float2 a = ld2(p), b = ld2(p + 2);
    return make_float4(a.x, a.y, b.x, b.y);
  }
};

// Waits until every memory operation this wavefront issued has completed
// (for the coherent stores of Mem<true>: reached the device-coherent level).
// The memory clobber keeps the compiler from moving accesses across it.
__device__ __forceinline__ void wait_memory() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// log2(e): exponentials are taken as the hardware exp2 of a scaled argument.
constexpr float kLog2e = 1.4426950408889634f;

// Agent-scope (whole device) relaxed atomics on int32 counters and words.
__device__ __forceinline__ int atomic_add_agent(int32_t* p, int v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int load_agent(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_agent(int32_t* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Every thread: waits until its stores (Mem<true>, so device-coherent once
// complete) have completed, then the workgroup counts itself in *ctr. True in
// every thread of the workgroup that arrived as the n-th; that workgroup reads
// what the others published with Mem<true> loads.
__device__ __forceinline__ bool arrive_last(int32_t* ctr, int n, int* s_flag) {
  wait_memory();
  __syncthreads();
  if (threadIdx.x == 0) *s_flag = atomic_add_agent(ctr, 1) == n - 1;
  __syncthreads();
  return *s_flag != 0;
}

// Number of tokens of block i in a sequence of length L.
__device__ __forceinline__ int block_count(int L, int B, int i) {
  int n = L - i * B;
  return n < 0 ? 0 : (n > B ? B : n);
}

}  // namespace spla
