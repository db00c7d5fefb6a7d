// Device helpers shared by the forward kernels (bf16 storage, MFMA types).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sb {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

// Buffer resource word 3 for gfx9-family raw buffers, and the cache-policy
// bit that marks a load non-temporal on gfx94x/gfx950.
constexpr int kBufferDword3 = 0x00020000;
constexpr int kNonTemporal = 2;

// A pointer the compiler is told is the same in every lane (kept in scalar
// registers, so a buffer descriptor built from it needs no per-lane loop).
__device__ __forceinline__ void *uniform_ptr(const void *p) {
  const unsigned long long v = (unsigned long long)p;
  const unsigned lo = (unsigned)__builtin_amdgcn_readfirstlane((int)(unsigned)v);
  const unsigned hi = (unsigned)__builtin_amdgcn_readfirstlane((int)(unsigned)(v >> 32));
  return (void *)(((unsigned long long)hi << 32) | lo);
}

// Buffer descriptor of `bytes` bytes at p, both wave-uniform: loads through
// it at offsets >= bytes read zero (branch-free bounds).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t uniform_rsrc(const void *p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(uniform_ptr(p), 0, __builtin_amdgcn_readfirstlane(bytes),
                                           kBufferDword3);
}

// 16-byte streaming load (data read once: weights)
__device__ __forceinline__ uint4 load_stream(const uint4 *p) {
  u32x4 v = __builtin_nontemporal_load((const u32x4 *)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// float -> bfloat16 bits, round to nearest even (inputs are finite here;
// NaN keeps a quiet NaN pattern)
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Index of element (row t, column k) in the "packed operand" layout of the
// bf16 activations the matrix-core GEMMs read: [t/16][k/32][t%16][k%32],
// 1 KB per (16-row tile, k-step) in which each row's 32 values are
// contiguous.  Lane l of the GEMM's operand fragment (row l % 16, columns
// 8 (l / 16) .. + 7 of the k-step) reads 16 bytes at (l % 16) * 64 +
// (l / 16) * 16, so a tile with a single valid row costs one 64-byte
// sector per k-step.  ksteps = K/32.
__device__ __forceinline__ size_t packed_index(int t, int k, int ksteps) {
  const int tt = t >> 4, s = k >> 5;
  return (((size_t)tt * ksteps + s) * 16 + (t & 15)) * 32 + (k & 31);
}

}  // namespace sb
