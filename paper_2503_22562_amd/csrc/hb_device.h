// Device-side helpers shared by the gfx950 kernels: bf16 conversions, vector
// types for 16-byte loads and the MFMA operand types.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hb {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16, round to nearest even (the hardware conversion of gfx950)
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
// 16-byte load of data read once (the decode path's K/V stream): the
// non-temporal hint keeps it from displacing reused lines in the caches.
__device__ __forceinline__ u32x4 ld16_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ u32x2 ld8(const void* p) { return *reinterpret_cast<const u32x2*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ void st8(void* p, u32x2 v) { *reinterpret_cast<u32x2*>(p) = v; }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Element offset of (key slot s, dimension d) in one K block of one kv head.
// The block is stored as [2][hd / 8][8][8]: slots 0-3 and 8-11 form group 0,
// slots 4-7 and 12-15 group 1, and within a group each 8-dimension chunk
// holds its 8 slots x 8 dimensions (128 bytes). One score MFMA of an
// attention step takes exactly one group's keys, so its 16-byte lane loads
// read whole 128-byte lines.
__host__ __device__ __forceinline__ int k_block_offset(int s, int d, int hd) {
  const int g = (s >> 2) & 1, j = ((s >> 3) << 2) | (s & 3);
  return ((g * (hd >> 3) + (d >> 3)) * 8 + j) * 8 + (d & 7);
}

// D(16x16) += A(16x32) * B(32x16), bf16 in, fp32 accumulate.
// Operand registers: lane l holds row (A) / column (B) l % 16 and eight
// consecutive k values of k-group l / 16; the result holds column l % 16 and
// rows 4 * (l / 16) + i, i = 0..3.
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Reductions over the four 16-lane rows of a wave (lanes l, l^16, l^32, l^48),
// with the gfx950 row-swap instructions: VALU only, no LDS round trip. Each
// swap returns the pair (x of this lane, x of the partner lane) in some order.
__device__ __forceinline__ float rows_max(float v) {
  const uint32_t x = __float_as_uint(v);
  const auto a = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  const uint32_t y = __float_as_uint(fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1])));
  const auto b = __builtin_amdgcn_permlane16_swap(y, y, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows_sum(float v) {
  const uint32_t x = __float_as_uint(v);
  const auto a = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  const uint32_t y = __float_as_uint(__uint_as_float(a[0]) + __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(y, y, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Load from memory that no kernel of the launch writes (the per-iteration
// metadata): read through the constant address space so that wave-uniform
// addresses become scalar loads, which do not wait on outstanding vector
// memory traffic.
template <typename T>
__device__ __forceinline__ T const_load(const T* p) {
  static_assert(sizeof(T) % 4 == 0, "whole 32-bit words");
  struct Words {
    int32_t w[sizeof(T) / 4];
  } b;
  const __attribute__((address_space(4))) int32_t* q =
      reinterpret_cast<const __attribute__((address_space(4))) int32_t*>(reinterpret_cast<uintptr_t>(p));
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) b.w[i] = q[i];
  return __builtin_bit_cast(T, b);
}

// Sum over all 64 lanes, on the vector ALUs: lane swaps within quads, within
// 8- and 16-lane rows (DPP mirrors), then across rows.
__device__ __forceinline__ float wave_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xF, 0xF, false));  // row_half_mirror
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xF, 0xF, false));  // row_mirror
  return rows_sum(v);
}

// Index of the calling wave in its workgroup, as a wave-uniform value (so
// loads addressed by it become scalar loads).
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

}  // namespace hb
