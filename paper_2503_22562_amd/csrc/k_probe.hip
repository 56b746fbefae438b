// Sustained-rate probes of the device, so that the kernels' roofline fractions
// can be read against what this GPU delivers on the same access patterns:
// reads of random 4-KB chunks (one pool block of one kv head, the paged
// attention pattern), a sequential streaming read, and a loop of 16x16x32
// bf16 MFMAs with no memory traffic.
#include "hb_device.h"
#include "hb_kernels.h"

namespace hb {
namespace probe_detail {

// Chunk index of wave w's iteration i (a 32-bit integer hash).
__device__ __forceinline__ uint32_t chunk_hash(uint32_t w, uint32_t i) {
  uint32_t h = w * 0x9E3779B1u ^ (i + 0x7F4A7C15u + (w << 6) + (w >> 2));
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  return h ^ (h >> 16);
}

// Every wave reads `iters` 4-KB chunks at hashed places of buf[0, 4096 n_chunks)
// as four 1-KB loads. The XOR of the data keeps the loads; it is written to
// sink only in the (never expected) case that it equals a marker.
__global__ __launch_bounds__(256) void random_read_kernel(const uint8_t* __restrict__ buf, uint32_t n_chunks,
                                                          int iters, uint32_t* sink) {
  const int lane = threadIdx.x & 63;
  const uint32_t w = blockIdx.x * 4 + (threadIdx.x >> 6);
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (int it = 0; it < iters; ++it) {
    const uint8_t* c = buf + (size_t)(chunk_hash(w, (uint32_t)it) % n_chunks) * 4096 + lane * 16;
    u32x4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = ld16(c + j * 1024);
#pragma unroll
    for (int j = 0; j < 4; ++j) acc ^= v[j];
  }
  if ((acc[0] ^ acc[1] ^ acc[2] ^ acc[3]) == 0x5EED5EEDu) sink[0] = acc[0];
}

// Grid-stride read of buf[0, 16 n), four 16-byte loads in flight per thread.
__global__ __launch_bounds__(256) void stream_read_kernel(const uint8_t* __restrict__ buf, size_t n, uint32_t* sink) {
  u32x4 acc = {0u, 0u, 0u, 0u};
  const size_t stride = (size_t)gridDim.x * 256 * 4;
  for (size_t i = (size_t)blockIdx.x * 256 * 4 + threadIdx.x; i < n; i += stride) {
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = (i + u * 256 < n) ? ld16(buf + (i + u * 256) * 16) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int u = 0; u < 4; ++u) acc ^= v[u];
  }
  if ((acc[0] ^ acc[1] ^ acc[2] ^ acc[3]) == 0x5EED5EEDu) sink[0] = acc[0];
}

// Eight independent accumulator chains of 16x16x32 bf16 MFMAs, 16 per
// iteration, operands in registers. The operands are pseudo-random values in
// [-1, 1) (the matrix cores draw more power, and run slower, on varied data
// than on constant operands, so constant operands would overstate the rate
// a GEMM on real data can reach).
__global__ __launch_bounds__(256) void mfma_kernel(int iters, uint32_t* sink) {
  f32x4 acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 a, b;
  const uint32_t t = blockIdx.x * 256 + threadIdx.x;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    a[j] = (__bf16)((float)(chunk_hash(t, j) >> 8) * (2.0f / 16777216.0f) - 1.0f);
    b[j] = (__bf16)((float)(chunk_hash(t, 8 + j) >> 8) * (2.0f / 16777216.0f) - 1.0f);
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j & 7] = mfma16x16x32(a, b, acc[j & 7]);
  }
  float r = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) r += acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3];
  if (r == 1234.5f) sink[0] = __float_as_uint(r);
}

}  // namespace probe_detail

void launch_probe_random_read(hipStream_t s, const void* buf, uint32_t n_chunks, int blocks, int iters,
                              uint32_t* sink) {
  probe_detail::random_read_kernel<<<blocks, 256, 0, s>>>(static_cast<const uint8_t*>(buf), n_chunks, iters, sink);
}

void launch_probe_stream_read(hipStream_t s, const void* buf, int64_t bytes, int blocks, uint32_t* sink) {
  probe_detail::stream_read_kernel<<<blocks, 256, 0, s>>>(static_cast<const uint8_t*>(buf), (size_t)bytes / 16, sink);
}

void launch_probe_mfma(hipStream_t s, int blocks, int iters, uint32_t* sink) {
  probe_detail::mfma_kernel<<<blocks, 256, 0, s>>>(iters, sink);
}

}  // namespace hb
