// Shared device types and small helpers for the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ u32x4 ld_u32x4(const uint16_t* p) { return *(const u32x4*)p; }
__device__ __forceinline__ bf16x8 ld_bf16x8(const uint16_t* p) { return *(const bf16x8*)p; }
__device__ __forceinline__ void st_u32x4(uint16_t* p, u32x4 v) { *(u32x4*)p = v; }

// Load through the constant address space: for a wave-uniform address this is
// a scalar (s_load) read.  Only for data no kernel writes while it runs.
template <typename T>
__device__ __forceinline__ T ld_uniform(const T* p) {
  static_assert(sizeof(T) % 4 == 0, "word-sized types only");
  typedef const __attribute__((address_space(4))) uint32_t cu32;
  cu32* q = (cu32*)p;
  uint32_t w[sizeof(T) / 4];
#pragma unroll
  for (unsigned i = 0; i < sizeof(T) / 4; ++i) w[i] = q[i];
  T out;
  __builtin_memcpy(&out, w, sizeof(T));
  return out;
}

// Workgroup barrier that orders LDS accesses only.  __syncthreads() also
// waits for every outstanding global access (vmcnt(0)), which would drain
// the direct-to-LDS tile loads a kernel deliberately keeps in flight across
// the barrier; their completion is awaited explicitly where it is needed.
// The empty asm statements keep the compiler from moving memory accesses
// across the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): my LDS accesses are done
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// 16-byte global -> LDS copy through a buffer resource covering
// [base, base + nbytes): lane i of the wave fills dst + 16 i with the 16 bytes
// at base + voff (zeros if voff is outside the range).  The buffer form keeps
// the compiler's LDS wait counting exact while the copy is in flight (the
// global-segment form makes it wait for every outstanding LDS access).
__device__ __forceinline__ void lds_dma16(const void* base, uint32_t nbytes, uint32_t voff,
                                          __attribute__((address_space(3))) void* dst) {
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)nbytes, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, 0, 0, 0);
}

// max that propagates NaN instead of quieting it: lowers to v_maximum3_f32
// without the canonicalising v_max x, x that fmaxf needs for MFMA results
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// v_exp_f32: 2^x (exp2(-inf) = 0).
__device__ __forceinline__ float exp2f_fast(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
  __bf16 b = (__bf16)x;
  return __builtin_bit_cast(uint16_t, b);
}

// Four floats -> four bf16 (round to nearest even), one 8-byte store.
__device__ __forceinline__ void st_bf16x4(uint16_t* p, float a, float b, float c, float d) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
  *(bf16x4*)p = v;
}

}  // namespace sa
