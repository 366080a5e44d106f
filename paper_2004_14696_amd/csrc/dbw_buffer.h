// Buffer-resource loads for gfx950.
//
// A raw buffer resource covers [base, base + bytes); a load whose byte offset
// falls outside that range returns 0 without touching memory.  Predicated
// loads ("value or 0") therefore need no branch: the predicate selects an
// out-of-range offset instead.  Plain "cond ? p[i] : 0" code is compiled into
// one branch and one full memory wait per load, which serialises streams.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace dbw {

// Word 3 of a raw (stride 0) buffer resource on gfx9-family parts.
constexpr int kBufferWord3 = 0x00020000;
// An offset no resource built here covers (resources are < 2^31 bytes).
constexpr uint32_t kOutOfRange = 0x80000000u;
// Largest array a single resource may cover.
constexpr int64_t kMaxBufferBytes = (int64_t{1} << 31) - 256;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), kBufferWord3);
}

__device__ __forceinline__ float buf_f32(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0));
}

__device__ __forceinline__ float4 buf_f32x4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0));
}

// The same with a wave-uniform byte offset soff added in the scalar operand
// (no vector arithmetic per load; an out-of-range voff stays out of range).
__device__ __forceinline__ float4 buf_f32x4_s(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, static_cast<int>(soff), 0));
}

__device__ __forceinline__ int32_t buf_i32(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return static_cast<int32_t>(__builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0));
}

}  // namespace dbw
