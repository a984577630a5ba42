// Device-side helpers shared by the gfx950 kernels of the VLA library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vla {

typedef uint16_t bf16_t;  // raw bf16 storage
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// fp32 -> bf16, round to nearest even (hardware conversion on gfx950).
__device__ __forceinline__ bf16_t f2bf(float f) {
  __bf16 b = (__bf16)f;
  return __builtin_bit_cast(bf16_t, b);
}

__device__ __forceinline__ uint32_t pack2bf(float lo, float hi) {
  return uint32_t(f2bf(lo)) | (uint32_t(f2bf(hi)) << 16);
}

// 8 bf16 held in a uint4 <-> 8 floats
__device__ __forceinline__ void unpack8(const uint4& v, float* f) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Sum / max over the 16 lanes that share (lane / 16).
__device__ __forceinline__ float group16_sum(float v) {
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float group16_max(float v) {
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8, v); }

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Fragment-major ("frag") layout of a bf16 matrix X[R][K], K % 32 == 0: 16 x 32
// blocks of 1 KB.  The blocks of 16-row block r / 16 are consecutive, K block
// k / 32 at element ((r/16) * frag_kb(K) + k/32) * 512, and one spare block
// ends each 16-row block so that equal K blocks of consecutive 16-row blocks
// are not a power-of-two distance apart (they would share memory channels).
// Inside a block, the 16 bytes that lane l of an MFMA 16x16x32 operand holds
// (row l % 16, K elements 8 (l / 16) .. + 8) are at 16 l bytes.  One 64-lane
// 16-byte load of a block reads 1 KB of contiguous memory and leaves every
// lane holding its fragment.  Storage: frag_elems(R, K) elements.
__host__ __device__ __forceinline__ int frag_kb(int K) { return (K >> 5) + 1; }
__host__ __device__ __forceinline__ size_t frag_elems(size_t R, int K) {
  return ((R + 15) >> 4) * (size_t)frag_kb(K) * 512;
}
__host__ __device__ __forceinline__ size_t frag_index(int r, int k, int K) {
  return ((((size_t)(r >> 4) * frag_kb(K) + (k >> 5)) << 6) + (r & 15) + (((k & 31) >> 3) << 4)) * 8 + (k & 7);
}

typedef __attribute__((address_space(3))) void lds_ptr_t;

// s_waitcnt with vmcnt <= n (n < 64) and the other counters unconstrained.
#define WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt((((n) >> 4) << 14) | (0xF << 8) | (0x7 << 4) | ((n) & 15))

// 16 bytes per lane from a buffer straight into LDS (buffer_load_dwordx4 ... lds):
// lane i writes bytes [16 i, 16 i + 16) after the wave-uniform LDS byte address
// m0.  Issued through inline assembly so that the compiler does not treat it
// as an LDS store (it would wait for every copy in flight before any later LDS
// read); the kernel waits for the copies it consumes itself.
__device__ __forceinline__ void lds_dma16(uint32_t m0, uint32_t voff, __amdgpu_buffer_rsrc_t rsrc, int soff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(m0), "v"(voff), "s"(rsrc), "s"(soff)
               : "memory");
}

}  // namespace vla
