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
#include <algorithm>

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

static void launch_gemm_regstaged(hipStream_t s, const GemmArgs& a) {
  const int ncols = (a.epi == GEMM_SWIGLU) ? 64 : BN;
  dim3 grid((a.N + ncols - 1) / ncols, (a.M + BM - 1) / BM);
  switch (a.epi) {
    case GEMM_STORE_BF16: gemm_kernel<GEMM_STORE_BF16><<<grid, 256, 0, s>>>(a); break;
    case GEMM_RESIDUAL: gemm_kernel<GEMM_RESIDUAL><<<grid, 256, 0, s>>>(a); break;
    default: gemm_kernel<GEMM_SWIGLU><<<grid, 256, 0, s>>>(a); break;
  }
}


// ---------------------------------------------------------------------------
// LDS-pipelined GEMM for K % 64 == 0.
//
// The K loop runs over a ring of STAGES LDS buffers that global memory fills
// directly (16-byte global-to-LDS loads, no register staging), so up to
// STAGES-1 K steps are in flight while one is multiplied. A 1-KB load
// instruction of a wave fills eight 128-byte rows of a tile; inside a row the
// eight 16-byte chunks are XOR-swizzled with the row index, so that the MFMA
// fragment reads of eight consecutive rows fall into eight different chunk
// positions. 4 waves in a 2 x 2 arrangement each own a (BM/2) x (BN/2) block
// of 16x16 MFMA tiles. Workgroups are numbered so that the ones sharing a
// weight tile run on the same XCD (one L2), and K can be split over several
// workgroups whose fp32 partials a second kernel sums in a fixed order.
// ---------------------------------------------------------------------------
namespace gemm_detail {

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// One K step (64 columns) of the A and B tiles: each wave issues A_LOADS +
// B_LOADS 1-KB global-to-LDS loads; lane L of a load lands at byte 16 L.
template <int A_LOADS, int B_LOADS>
__device__ __forceinline__ void issue_stage(uint8_t* base, int a_bytes, const uint16_t* Abase, const uint16_t* Bbase,
                                            const uint32_t* aoff, const uint32_t* boff, int wave, int koff) {
#pragma unroll
  for (int j = 0; j < A_LOADS; ++j)
    __builtin_amdgcn_global_load_lds(Abase + aoff[j] + koff, base + (wave * A_LOADS + j) * 1024, 16, 0, 0);
#pragma unroll
  for (int j = 0; j < B_LOADS; ++j)
    __builtin_amdgcn_global_load_lds(Bbase + boff[j] + koff, base + a_bytes + (wave * B_LOADS + j) * 1024, 16, 0, 0);
}

template <int BM, int BN, int STAGES, int EPI>
__global__ __launch_bounds__(256, 1) void gemm_lds_kernel(GemmArgs a, int tiles_m, int tiles_n, int ksplit,
                                                           int kchunk, float* __restrict__ partial) {
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int A_BYTES = BM * 128, STAGE_BYTES = (BM + BN) * 128;
  constexpr int A_LOADS = BM / 32, B_LOADS = BN / 32, LOADS = A_LOADS + B_LOADS;
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];

  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int wm = wave >> 1, wn = wave & 1;
  // XCD-aware tile order: workgroup g runs on XCD g % 8; give each XCD a
  // contiguous run of tiles, M fastest, so tiles sharing weights share an L2.
  const int total = tiles_m * tiles_n * ksplit;
  const int xcd = blockIdx.x & 7, loc = blockIdx.x >> 3, q = total >> 3, r = total & 7;
  const int t = (xcd < r) ? xcd * (q + 1) + loc : r * (q + 1) + (xcd - r) * q + loc;
  const int mt = t % tiles_m;
  const int ks = (t / tiles_m) % ksplit;
  const int nt = t / (tiles_m * ksplit);
  const int m0 = mt * BM;
  const int M = a.M, N = a.N;
  const int k_begin = ks * kchunk;
  const int k_end = min(a.K, k_begin + kchunk);
  const int nk = (k_end - k_begin) >> 6;

  // per-lane source offsets (elements) of this wave's load instructions,
  // rows clamped in range: rows past M or N only feed outputs never stored
  const int lrow = lane >> 3;
  const int lchunk = (lane & 7) ^ lrow;
  uint32_t aoff[A_LOADS], boff[B_LOADS];
#pragma unroll
  for (int j = 0; j < A_LOADS; ++j) {
    const int row = 8 * (wave * A_LOADS + j) + lrow;
    aoff[j] = (uint32_t)min(m0 + row, M - 1) * (uint32_t)a.lda + 8 * lchunk;
  }
#pragma unroll
  for (int j = 0; j < B_LOADS; ++j) {
    const int row = 8 * (wave * B_LOADS + j) + lrow;
    int brow;
    if (EPI == GEMM_SWIGLU) {
      const int c = min(nt * (BN / 2) + (row % (BN / 2)), N - 1);
      brow = (row < BN / 2) ? c : N + c;
    } else {
      brow = min(nt * BN + row, N - 1);
    }
    boff[j] = (uint32_t)brow * (uint32_t)a.ldb + 8 * lchunk;
  }
  const uint16_t* Abase = a.A + k_begin;
  const uint16_t* Bbase = a.B + k_begin;

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Fragment rows of a wave differ by multiples of 8, so the chunk swizzle
  // (row & 7) is that of the lane's own row: every fragment address is one
  // per-lane base plus a compile-time offset. k-half kc flips chunk bit 2.
  const int fr = lane & 15, fg = lane >> 4;
  const int swz = ((fg ^ (fr & 7)) << 4);
  const int a_lane = (wm * WM + fr) * 128 + swz;
  const int b_lane = (EPI == GEMM_SWIGLU ? wn * (BN / 4) : wn * WN) * 128 + fr * 128 + swz;

#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nk) issue_stage<A_LOADS, B_LOADS>(smem + s * STAGE_BYTES, A_BYTES, Abase, Bbase, aoff, boff, wave, s * 64);
  for (int kt = 0; kt < nk; ++kt) {
    // loads of step kt are complete once at most the later steps' are pending
    const int ahead = min(STAGES - 2, nk - 1 - kt);
    if (STAGES >= 4 && ahead >= 2) wait_vmcnt<(STAGES >= 4 ? 2 * LOADS : 0)>();
    else if (STAGES >= 3 && ahead >= 1) wait_vmcnt<(STAGES >= 3 ? LOADS : 0)>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    if (kt + STAGES - 1 < nk)
      issue_stage<A_LOADS, B_LOADS>(smem + ((kt + STAGES - 1) % STAGES) * STAGE_BYTES, A_BYTES, Abase, Bbase, aoff, boff,
                                    wave, (kt + STAGES - 1) * 64);
    const uint8_t* As = smem + (kt % STAGES) * STAGE_BYTES;
    const uint8_t* Bs = As + A_BYTES;
    // all fragment reads of the step first, so LDS latency overlaps the MFMAs
    // (the compiler then waits on partial counts instead of after every read)
    bf16x8 af[2][TM], bfr[2][TN];
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      const uint8_t* ap = As + (a_lane ^ (kc << 6));
      const uint8_t* bp = Bs + (b_lane ^ (kc << 6));
#pragma unroll
      for (int mi = 0; mi < TM; ++mi) af[kc][mi] = as_bf16x8(*reinterpret_cast<const u32x4*>(ap + mi * 2048));
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) {
        const int roff = (EPI == GEMM_SWIGLU) ? ((ni < TN / 2) ? 16 * ni : BN / 2 + 16 * (ni - TN / 2)) : 16 * ni;
        bfr[kc][ni] = as_bf16x8(*reinterpret_cast<const u32x4*>(bp + roff * 128));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
#pragma unroll
      for (int mi = 0; mi < TM; ++mi)
#pragma unroll
        for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = mfma16x16x32(bfr[kc][ni], af[kc][mi], acc[mi][ni]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // epilogue: acc[mi][ni][i] = C[m][n + i]
  const int cq = fg << 2;
#pragma unroll
  for (int mi = 0; mi < TM; ++mi) {
    // keep the residual loads of one fragment row at a time in flight
    __builtin_amdgcn_sched_barrier(0);
    const int m = m0 + wm * WM + 16 * mi + fr;
    if (m >= M) continue;
    if (EPI == GEMM_SWIGLU) {
#pragma unroll
      for (int ni = 0; ni < TN / 2; ++ni) {
        const int n = nt * (BN / 2) + wn * (BN / 4) + 16 * ni + cq;
        if (n >= N) continue;
        const f32x4 gt = acc[mi][ni], up = acc[mi][ni + TN / 2];
        u32x2 o;
        o[0] = pack_bf16x2(silu_f(gt[0]) * up[0], silu_f(gt[1]) * up[1]);
        o[1] = pack_bf16x2(silu_f(gt[2]) * up[2], silu_f(gt[3]) * up[3]);
        st8(reinterpret_cast<uint16_t*>(a.C) + (size_t)m * a.ldc + n, o);
      }
    } else {
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) {
        const int n = nt * BN + wn * WN + 16 * ni + cq;
        if (n >= N) continue;
        f32x4 c = acc[mi][ni];
        if (ksplit > 1) {
          u32x4 o = {__float_as_uint(c[0]), __float_as_uint(c[1]), __float_as_uint(c[2]), __float_as_uint(c[3])};
          st16(partial + ((size_t)ks * M + m) * N + n, o);
          continue;
        }
        if (EPI == GEMM_RESIDUAL) {
          if (a.r_f32) {
            const u32x4 rr = ld16(reinterpret_cast<const float*>(a.R) + (size_t)m * a.ldr + n);
            for (int j = 0; j < 4; ++j) c[j] += __uint_as_float(rr[j]);
          } else {
            const u32x2 rr = ld8(reinterpret_cast<const uint16_t*>(a.R) + (size_t)m * a.ldr + n);
            c[0] += bf16_lo(rr[0]); c[1] += bf16_hi(rr[0]);
            c[2] += bf16_lo(rr[1]); c[3] += bf16_hi(rr[1]);
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

// Sum of the split-K partials in split order, then the epilogue.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs a, int ksplit, const float* __restrict__ partial) {
  const int64_t nvec = (int64_t)a.M * a.N / 4;
  for (int64_t v = blockIdx.x * 256ll + threadIdx.x; v < nvec; v += (int64_t)gridDim.x * 256) {
    const int64_t e = v * 4;
    const int m = (int)(e / a.N), n = (int)(e - (int64_t)m * a.N);
    f32x4 c = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < ksplit; ++s) {
      const u32x4 p = ld16(partial + ((size_t)s * a.M + m) * a.N + n);
      for (int j = 0; j < 4; ++j) c[j] += __uint_as_float(p[j]);
    }
    if (a.epi == GEMM_RESIDUAL) {
      if (a.r_f32) {
        const u32x4 rr = ld16(reinterpret_cast<const float*>(a.R) + (size_t)m * a.ldr + n);
        for (int j = 0; j < 4; ++j) c[j] += __uint_as_float(rr[j]);
      } else {
        const u32x2 rr = ld8(reinterpret_cast<const uint16_t*>(a.R) + (size_t)m * a.ldr + n);
        c[0] += bf16_lo(rr[0]); c[1] += bf16_hi(rr[0]);
        c[2] += bf16_lo(rr[1]); c[3] += bf16_hi(rr[1]);
      }
    }
    if (a.epi == GEMM_RESIDUAL && a.c_f32) {
      u32x4 o = {__float_as_uint(c[0]), __float_as_uint(c[1]), __float_as_uint(c[2]), __float_as_uint(c[3])};
      st16(reinterpret_cast<float*>(a.C) + (size_t)m * a.ldc + n, o);
    } else {
      u32x2 o = {pack_bf16x2(c[0], c[1]), pack_bf16x2(c[2], c[3])};
      st8(reinterpret_cast<uint16_t*>(a.C) + (size_t)m * a.ldc + n, o);
    }
  }
}


}  // namespace gemm_detail

namespace {
using namespace gemm_detail;

struct TileCfg {
  int bm, bn, stages;
  float eff;  // relative MFMA efficiency of the tile shape
};
constexpr TileCfg kTiles[] = {
    {256, 256, 2, 1.00f}, {256, 128, 3, 0.90f}, {128, 256, 3, 0.90f}, {128, 128, 4, 0.75f}, {64, 256, 3, 0.70f},
};

template <int BM, int BN, int ST, int EPI>
void launch_tile(hipStream_t s, const GemmArgs& a, int tiles_m, int tiles_n, int ksplit, int kchunk, float* partial) {
  constexpr int lds = ST * (BM + BN) * 128;
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_lds_kernel<BM, BN, ST, EPI>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    attr = true;
  }
  gemm_lds_kernel<BM, BN, ST, EPI><<<tiles_m * tiles_n * ksplit, 256, lds, s>>>(a, tiles_m, tiles_n, ksplit, kchunk,
                                                                                  partial);
}

template <int EPI>
void launch_cfg(int idx, hipStream_t s, const GemmArgs& a, int tm, int tn, int ks, int kchunk, float* part) {
  switch (idx) {
    case 0: launch_tile<256, 256, 2, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 1: launch_tile<256, 128, 3, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 2: launch_tile<128, 256, 3, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 3: launch_tile<128, 128, 4, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    default: launch_tile<64, 256, 3, EPI>(s, a, tm, tn, ks, kchunk, part); break;
  }
}
}  // namespace

GemmPlan plan_gemm(const GemmArgs& a, int cu_count, int force_cfg, int force_ksplit) {
  GemmPlan best{-1, 0, 0, 1, 0};
  if (a.K % 64 != 0) return best;
  double best_cost = 1e300;
  const int ksteps = a.K / 64;
  for (int i = 0; i < (int)(sizeof(kTiles) / sizeof(kTiles[0])); ++i) {
    if (force_cfg >= 0 && i != force_cfg) continue;
    const TileCfg& c = kTiles[i];
    const int ncols = (a.epi == GEMM_SWIGLU) ? c.bn / 2 : c.bn;
    const int tm = (a.M + c.bm - 1) / c.bm, tn = (a.N + ncols - 1) / ncols;
    for (int ks = 1; ks <= 8; ks *= 2) {
      if (ks > 1 && (a.epi == GEMM_SWIGLU || ksteps < 4 * ks)) break;
      if (force_ksplit > 0 && ks != force_ksplit && !(a.epi == GEMM_SWIGLU && ks == 1)) continue;
      const int kchunk = ((ksteps + ks - 1) / ks) * 64;
      const int nwg = tm * tn * ks;
      const int rounds = (nwg + cu_count - 1) / cu_count;
      double cost = (double)rounds * c.bm * c.bn * kchunk / c.eff;
      if (ks > 1) cost += (double)a.M * a.N * (ks + 2) * 4.0 / (8e12 / 2.5e15) / 2 / cu_count;  // reduce pass
      if (cost < best_cost * 0.999) {
        best_cost = cost;
        best = GemmPlan{i, tm, tn, ks, kchunk};
      }
    }
  }
  return best;
}

void launch_gemm(hipStream_t s, const GemmArgs& a, const GemmPlan& p, float* partial) {
  if (a.M <= 0 || a.N <= 0) return;
  if (p.cfg < 0) {
    launch_gemm_regstaged(s, a);
    return;
  }
  switch (a.epi) {
    case GEMM_STORE_BF16: launch_cfg<GEMM_STORE_BF16>(p.cfg, s, a, p.tiles_m, p.tiles_n, p.ksplit, p.kchunk, partial); break;
    case GEMM_RESIDUAL: launch_cfg<GEMM_RESIDUAL>(p.cfg, s, a, p.tiles_m, p.tiles_n, p.ksplit, p.kchunk, partial); break;
    default: launch_cfg<GEMM_SWIGLU>(p.cfg, s, a, p.tiles_m, p.tiles_n, p.ksplit, p.kchunk, partial); break;
  }
  if (p.ksplit > 1) {
    const int64_t nvec = (int64_t)a.M * a.N / 4;
    const int grid = (int)std::min<int64_t>((nvec + 255) / 256, 8192);
    splitk_reduce_kernel<<<grid, 256, 0, s>>>(a, p.ksplit, partial);
  }
}

}  // namespace hb
