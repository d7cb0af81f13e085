// Buffer-descriptor access for gfx950, shared by the kernels of the library.
//
// A raw buffer descriptor covers [base, base + bytes); the hardware range check
// returns zeros for loads and drops stores at byte offsets outside it, so tile
// tails need no branches: an out-of-range element is addressed at kOOB.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace resbm {

typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef int v2i __attribute__((ext_vector_type(2)));
typedef int v4i __attribute__((ext_vector_type(4)));

constexpr uint32_t kOOB = 0xFFFFFFF0u;        // a byte offset outside every descriptor
constexpr int64_t kMaxRange = 0xFFFFF000ll;   // descriptor ranges are clamped below kOOB

// Raw buffer descriptor over [base, base + bytes): gfx9-family dword 3, no stride.
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const uint32_t nb = bytes <= 0 ? 0u : (bytes > kMaxRange ? (uint32_t)kMaxRange : (uint32_t)bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, nb, 0x00020000);
}

// Loads and stores at a byte offset; POL is the cache-policy operand.
template <int POL = 0>
__device__ __forceinline__ uint4 bld16(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, POL));
}
template <int POL = 0>
__device__ __forceinline__ uint2 bld8(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, POL));
}
template <int POL = 0>
__device__ __forceinline__ void bst16(rsrc_t r, uint32_t off, uint4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i, v), r, off, 0, POL);
}
template <int POL = 0>
__device__ __forceinline__ void bst8(rsrc_t r, uint32_t off, uint2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(v2i, v), r, off, 0, POL);
}

}  // namespace resbm
