// ea_device.h -- element conversions and wavefront helpers shared by libea's
// kernels.  gfx950, wave64.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "ea_internal.h"

namespace ea {

// bf16 <-> f32.  Widening is exact; narrowing rounds to nearest, ties to even
// (NaN stays NaN).
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// The narrowing is gfx950's v_cvt_pk_bf16_f32 (one instruction per two
// values); it was checked against the bit-level round-to-nearest-even on 2^25
// float patterns of every exponent, subnormals, ties and infinities included:
// identical results, and NaN stays NaN.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

// Two values narrowed to bf16 in one instruction, lo in bits 0..15.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float f16_to_f32(uint16_t h) {
  _Float16 v;
  __builtin_memcpy(&v, &h, 2);
  return (float)v;
}

__device__ __forceinline__ uint16_t f32_to_f16(float f) {
  _Float16 v = (_Float16)f;
  uint16_t h;
  __builtin_memcpy(&h, &v, 2);
  return h;
}

// Wavefront-uniform read-only metadata (tuple table, block tables) through
// the constant address space: scalar loads, waited on with lgkmcnt, so they
// never force a wait on in-flight vector loads.
template <class T>
__device__ __forceinline__ T ld_uniform(const T* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  return *(const __attribute__((address_space(4))) T*)(p);
#else
  return *p;  // host pass: parsed, never executed
#endif
}

// ---- hand-off between workgroups through global memory ------------------
// The eight XCDs' L2 caches are not coherent with each other.  Agent-scope
// relaxed atomic loads and stores are (they carry the coherence bits), so
// partial results passed from one workgroup to another use them, and no
// device-scope fence -- which would write back and invalidate the whole L2 of
// the XCD, evicting every co-resident workgroup's operands -- is needed.  The
// writer drains its stores (vmcnt 0) before it counts its arrival; the reader
// issues its loads only after its own arrival count has returned.
__device__ __forceinline__ void store_agent2(float* p, float a, float b) {
  const uint64_t v = (uint64_t)__float_as_uint(a) | ((uint64_t)__float_as_uint(b) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ float2 load_agent2(const float* p) {
  const uint64_t v =
      __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
}

__device__ __forceinline__ float load_agent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// every outstanding vector-memory access of this wave completed (vmcnt 0)
__device__ __forceinline__ void drain_vmem() { __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8)); }

// arrival count of a split key; returns the count before this arrival
__device__ __forceinline__ int arrive_agent(int32_t* counter) {
  return __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void reset_agent(int32_t* counter) {
  __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Store with the non-temporal hint: the line is streamed towards memory
// instead of being kept dirty in the XCD's L2, which the end of the kernel
// would otherwise have to write back (measured on an RMSNorm over 64 MiB run
// back to back: 16.1 -> 12.1 us).  When the next kernel reads the output,
// plain stores are faster: it then finds the lines in the caches.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
template <class T>
__device__ __forceinline__ void store_stream(void* p, const T& v) {
  if constexpr (sizeof(T) == 16) {
    __builtin_nontemporal_store(__builtin_bit_cast(u32x4_t, v), reinterpret_cast<u32x4_t*>(p));
  } else if constexpr (sizeof(T) == 8) {
    __builtin_nontemporal_store(__builtin_bit_cast(u32x2_t, v), reinterpret_cast<u32x2_t*>(p));
  } else if constexpr (sizeof(T) == 4) {
    __builtin_nontemporal_store(__builtin_bit_cast(uint32_t, v), reinterpret_cast<uint32_t*>(p));
  } else if constexpr (sizeof(T) == 2) {
    __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, v), reinterpret_cast<uint16_t*>(p));
  } else {
    static_assert(sizeof(T) == 1, "store_stream: 1, 2, 4, 8 or 16 bytes");
    __builtin_nontemporal_store(__builtin_bit_cast(uint8_t, v), reinterpret_cast<uint8_t*>(p));
  }
}

// An output store under the caller's policy: streamed (non-temporal) or
// plain.  The policy is a template argument, and callers branch once around a
// whole store loop: the compiler merges two otherwise identical stores in the
// arms of a runtime branch into one and drops the non-temporal hint.
template <bool STREAM, class T>
__device__ __forceinline__ void store_out(void* p, const T& v) {
  if constexpr (STREAM) store_stream(p, v);
  else *reinterpret_cast<T*>(p) = v;
}

// Load/store one element of a relation given its dtype.
__device__ __forceinline__ float ld_elem(const char* base, int64_t idx, int dt) {
  if (dt == EA_F32) return reinterpret_cast<const float*>(base)[idx];
  const uint16_t h = reinterpret_cast<const uint16_t*>(base)[idx];
  return dt == EA_BF16 ? bf16_to_f32(h) : f16_to_f32(h);
}

__device__ __forceinline__ void st_elem(char* base, int64_t idx, int dt, float v) {
  if (dt == EA_F32) {
    reinterpret_cast<float*>(base)[idx] = v;
  } else {
    reinterpret_cast<uint16_t*>(base)[idx] = dt == EA_BF16 ? f32_to_bf16(v) : f32_to_f16(v);
  }
}

// Wavefront (64 lanes) reductions without LDS round trips: DPP swaps of
// lane pairs (quad_perm 1,0,3,2) and of pair pairs (quad_perm 2,3,0,1), the
// 8- and 16-lane mirrors, then v_permlane16_swap and v_permlane32_swap for
// the other 16-lane row and the other 32-lane half.  At every stage a lane
// combines its value with one that holds the same kind of partial, so every
// lane ends with the same bits (x + y == y + x).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, true));
}
__device__ __forceinline__ float other16(float v) {  // the value of lane l ^ 16
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float((threadIdx.x & 16) ? r[0] : r[1]);
}
__device__ __forceinline__ float other32(float v) {  // the value of lane l ^ 32
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}
template <class Op>
__device__ __forceinline__ float wave_reduce(float v, Op op) {
  v = op(v, dpp_f<0xB1>(v));   // quad_perm [1, 0, 3, 2]
  v = op(v, dpp_f<0x4E>(v));   // quad_perm [2, 3, 0, 1]
  v = op(v, dpp_f<0x141>(v));  // row_half_mirror
  v = op(v, dpp_f<0x140>(v));  // row_mirror
  v = op(v, other16(v));
  return op(v, other32(v));
}

__device__ __forceinline__ float wave_sum(float v) {
  return wave_reduce(v, [](float a, float b) { return a + b; });
}

__device__ __forceinline__ float wave_max(float v) {
  return wave_reduce(v, [](float a, float b) { return fmaxf(a, b); });
}

}  // namespace ea
