// bf16 MFMA GEMMs of the layer (QKV, O + residual, gate/up + SwiGLU,
// down + residual): C[M][N] = A[M][K] B[N][K]^T, both operands K-contiguous
// (activations row-major, weights row-major [out][in]), fp32 accumulation.
//
// Tiling: 256 threads = 4 wavefronts in a 2 x 2 arrangement over a
// 128 x 128 output tile; each wave owns 64 x 64 = 4 x 4 MFMA 16x16 tiles.
// K advances in steps of 64 through LDS (rows padded by 16 bytes so the
// 16-byte fragment reads of eight consecutive rows hit distinct banks); the
// next K step is fetched into registers while the current one is multiplied.
// Each MFMA computes a transposed 16x16 block (weights as the A operand), so a
// lane ends up with four consecutive output columns of one row and the
// epilogue stores 8- or 16-byte vectors.
#include "hb_device.h"
#include "hb_kernels.h"

namespace hb {

namespace {
constexpr int BM = 128, BN = 128, BK = 64, LDSW = BK + 8;  // LDS row width in bf16

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + __expf(-z)); }

template <int EPI>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t As[BM * LDSW];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * LDSW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BM;
  const int nb = blockIdx.x;
  const int M = a.M, N = a.N, K = a.K;

  // global -> register staging: 4 x 16 B of A and of B per thread
  u32x4 ra[4], rb[4];
  const u32x4 zero = {0u, 0u, 0u, 0u};
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = tid + 256 * i, row = v >> 3, kk = k0 + ((v & 7) << 3);
      const int gm = m0 + row;
      ra[i] = (gm < M && kk < K) ? ld16(a.A + (size_t)gm * a.lda + kk) : zero;
      int brow;
      bool ok;
      if (EPI == GEMM_SWIGLU) {
        const int c = nb * 64 + (row & 63);
        ok = c < N;
        brow = (row < 64) ? c : N + c;
      } else {
        brow = nb * BN + row;
        ok = brow < N;
      }
      rb[i] = (ok && kk < K) ? ld16(a.B + (size_t)brow * a.ldb + kk) : zero;
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = tid + 256 * i, row = v >> 3, kk = (v & 7) << 3;
      *reinterpret_cast<u32x4*>(&As[row * LDSW + kk]) = ra[i];
      *reinterpret_cast<u32x4*>(&Bs[row * LDSW + kk]) = rb[i];
    }
  };
  // LDS row of the wave's B fragment ni
  auto brow_lds = [&](int ni) -> int {
    if (EPI == GEMM_SWIGLU) return (ni >> 1) * 64 + wn * 32 + 16 * (ni & 1);
    return wn * 64 + 16 * ni;
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = (K + BK - 1) / BK;
  gload(0);
  sstore();
  __syncthreads();
  const int fr = lane & 15, fk = (lane >> 4) << 3;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
    for (int kc = 0; kc < BK; kc += 32) {
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
        af[mi] = as_bf16x8(*reinterpret_cast<const u32x4*>(&As[(wm * 64 + 16 * mi + fr) * LDSW + kc + fk]));
#pragma unroll
      for (int ni = 0; ni < 4; ++ni)
        bfr[ni] = as_bf16x8(*reinterpret_cast<const u32x4*>(&Bs[(brow_lds(ni) + fr) * LDSW + kc + fk]));
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = mfma16x16x32(bfr[ni], af[mi], acc[mi][ni]);
    }
    __syncthreads();
    if (kt + 1 < nk) {
      sstore();
      __syncthreads();
    }
  }

  // epilogue: acc[mi][ni][r] = C[m][n + r], m = row of lane, n = 4 consecutive columns
  const int cq = (lane >> 4) << 2;
#pragma unroll
  for (int mi = 0; mi < 4; ++mi) {
    const int m = m0 + wm * 64 + 16 * mi + fr;
    if (m >= M) continue;
    if (EPI == GEMM_SWIGLU) {
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int n = nb * 64 + wn * 32 + 16 * ni + cq;
        if (n >= N) continue;
        const f32x4 gt = acc[mi][ni], up = acc[mi][ni + 2];
        u32x2 o;
        o[0] = pack_bf16x2(silu_f(gt[0]) * up[0], silu_f(gt[1]) * up[1]);
        o[1] = pack_bf16x2(silu_f(gt[2]) * up[2], silu_f(gt[3]) * up[3]);
        st8(reinterpret_cast<uint16_t*>(a.C) + (size_t)m * a.ldc + n, o);
      }
    } else {
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const int n = nb * BN + wn * 64 + 16 * ni + cq;
        if (n >= N) continue;
        f32x4 c = acc[mi][ni];
        if (EPI == GEMM_RESIDUAL) {
          if (a.r_f32) {
            const u32x4 r = ld16(reinterpret_cast<const float*>(a.R) + (size_t)m * a.ldr + n);
            for (int j = 0; j < 4; ++j) c[j] += __uint_as_float(r[j]);
          } else {
            const u32x2 r = ld8(reinterpret_cast<const uint16_t*>(a.R) + (size_t)m * a.ldr + n);
            c[0] += bf16_lo(r[0]); c[1] += bf16_hi(r[0]);
            c[2] += bf16_lo(r[1]); c[3] += bf16_hi(r[1]);
          }
        }
        if (EPI == GEMM_RESIDUAL && a.c_f32) {
          u32x4 o = {__float_as_uint(c[0]), __float_as_uint(c[1]), __float_as_uint(c[2]), __float_as_uint(c[3])};
          st16(reinterpret_cast<float*>(a.C) + (size_t)m * a.ldc + n, o);
        } else {
          u32x2 o = {pack_bf16x2(c[0], c[1]), pack_bf16x2(c[2], c[3])};
          st8(reinterpret_cast<uint16_t*>(a.C) + (size_t)m * a.ldc + n, o);
        }
      }
    }
  }
}
}  // namespace

void launch_gemm(hipStream_t s, const GemmArgs& a) {
  if (a.M <= 0 || a.N <= 0) return;
  const int ncols = (a.epi == GEMM_SWIGLU) ? 64 : BN;
  dim3 grid((a.N + ncols - 1) / ncols, (a.M + BM - 1) / BM);
  switch (a.epi) {
    case GEMM_STORE_BF16: gemm_kernel<GEMM_STORE_BF16><<<grid, 256, 0, s>>>(a); break;
    case GEMM_RESIDUAL: gemm_kernel<GEMM_RESIDUAL><<<grid, 256, 0, s>>>(a); break;
    default: gemm_kernel<GEMM_SWIGLU><<<grid, 256, 0, s>>>(a); break;
  }
}

}  // namespace hb
