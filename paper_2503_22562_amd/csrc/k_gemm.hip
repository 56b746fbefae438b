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
        if (EPI == GEMM_RESIDUAL && a.R) {
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
// Tile BM x BN = 16 TM WR x 16 TN WC: WR x WC waves (2 x 2, 2 x 4 or 4 x 2)
// each own TM x TN 16x16 MFMA blocks (accumulators in VGPRs: the kernels are
// built with the MFMA VGPR form, so no copies between register files). K advances
// in stages of 64 through a ring of S LDS buffers that global memory fills
// directly (16-byte global-to-LDS loads, no register staging). A 1-KB load
// instruction of a wave fills eight 128-byte rows; inside a row the eight
// 16-byte chunks are XOR-swizzled with the row index, so the fragment reads
// of eight consecutive rows fall into eight different chunk positions.
//
// Software pipeline: a stage is consumed in two K halves of 32 whose MFMA
// operands live in two register sets. While the MFMAs of one half run, the
// fragment reads of the next half are issued between them (the scheduler is
// told the interleave), so LDS latency and bandwidth hide under the matrix
// cores. One barrier per stage, between the halves: after it, the buffer just
// read is refilled with the stage S ahead and the next stage's first half is
// read. Workgroups are numbered so that those sharing a weight tile run on the
// same XCD (one L2); K can be split over workgroups whose fp32 partials a
// second kernel sums in a fixed order.
// ---------------------------------------------------------------------------
namespace gemm_detail {

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void wait_lgkm0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// One K stage (64 columns) of the A and B tiles: LA (LB) 1-KB loads fill the
// A (B) tile, 8 rows each; wave w issues loads w, w + NW, w + 2 NW, ...
// (NA / NB slots, the last possibly empty); lane L of a load lands at byte
// 16 L. The loads are buffer loads straight into LDS: the wave-uniform byte
// offset of each slot's 8-row group (ao / bo, plus the stage's K offset) is a
// scalar operand, and the lane's offset inside the group (la / lb) the only
// vector one, so no per-load address registers are needed.
template <int NW, int LA, int LB, int NA, int NB>
__device__ __forceinline__ void issue_stage(uint8_t* base, int a_bytes, __amdgpu_buffer_rsrc_t ra,
                                            __amdgpu_buffer_rsrc_t rb, const uint32_t (&ao)[NA],
                                            const uint32_t (&bo)[NB], uint32_t la, uint32_t lb, int wave,
                                            uint32_t kbytes) {
  typedef __attribute__((address_space(3))) void* lds_ptr;
#pragma unroll
  for (int j = 0; j < NA; ++j)
    if (LA % NW == 0 || j * NW + wave < LA) {
      uint8_t* p = base + (j * NW + wave) * 1024;
      const uint32_t so = ao[j] + kbytes;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr)p, 16, la, so, 0, 0);
    }
#pragma unroll
  for (int j = 0; j < NB; ++j)
    if (LB % NW == 0 || j * NW + wave < LB) {
      uint8_t* p = base + a_bytes + (j * NW + wave) * 1024;
      const uint32_t so = bo[j] + kbytes;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr)p, 16, lb, so, 0, 0);
    }
}

// Buffer resource over [p, p + bytes) for raw (unstrided) loads.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// Fragment reads of one K half: TM A fragments (16-row blocks 2 KB apart)
// and TN B fragments at the given per-fragment row offsets.
template <int TM, int TN>
__device__ __forceinline__ void read_frags(bf16x8 (&fa)[TM], bf16x8 (&fb)[TN], const uint8_t* ap, const uint8_t* bp,
                                           const int (&broff)[TN]) {
#pragma unroll
  for (int mi = 0; mi < TM; ++mi) fa[mi] = as_bf16x8(*reinterpret_cast<const u32x4*>(ap + mi * 2048));
#pragma unroll
  for (int ni = 0; ni < TN; ++ni) fb[ni] = as_bf16x8(*reinterpret_cast<const u32x4*>(bp + broff[ni]));
}

template <int TM, int TN>
__device__ __forceinline__ void mfma_block(f32x4 (&acc)[TM][TN], const bf16x8 (&fa)[TM], const bf16x8 (&fb)[TN]) {
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = mfma16x16x32(fb[ni], fa[mi], acc[mi][ni]);
}

// Scheduling directive for the region just emitted: NMFMA MFMAs with NREAD
// LDS reads spread evenly between them, an MFMA first (its operands were read
// one K half earlier, so the new reads never delay it).
template <int NREAD, int NMFMA>
__device__ __forceinline__ void interleave_reads() {
  constexpr int per = NMFMA / NREAD > 0 ? NMFMA / NREAD : 1;
  constexpr int groups = NMFMA / per < NREAD ? NMFMA / per : NREAD;
  constexpr int extra = NMFMA - per * groups;
#pragma unroll
  for (int i = 0; i + 1 < groups; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, per, 0);  // `per` MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);    // then one LDS read
  }
  __builtin_amdgcn_sched_group_barrier(0x008, per, 0);
  __builtin_amdgcn_sched_group_barrier(0x100, NREAD - groups + 1, 0);
  if (extra > 0) __builtin_amdgcn_sched_group_barrier(0x008, extra, 0);
}

// Scheduling directive for the second K half: after the barrier, NLOAD
// global-to-LDS loads (the stage S ahead) and NREAD LDS reads (the next
// stage's first half) each follow an MFMA of this half, loads first, so the
// MFMA pipe keeps running while they issue.
template <int NLOAD, int NREAD, int NMFMA>
__device__ __forceinline__ void interleave_loads_reads() {
  constexpr int ops = NLOAD + NREAD;
  constexpr int per_op = (ops + NMFMA - 1) / NMFMA;  // ops after each MFMA
  constexpr int slots = (ops + per_op - 1) / per_op;
  int loads = NLOAD, reads = NREAD;
#pragma unroll
  for (int i = 0; i < slots; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
#pragma unroll
    for (int j = 0; j < per_op; ++j) {
      if (loads > 0) {
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        --loads;
      } else if (reads > 0) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        --reads;
      }
    }
  }
  if (NMFMA > slots) __builtin_amdgcn_sched_group_barrier(0x008, NMFMA > slots ? NMFMA - slots : 1, 0);
}

// Whether a tile (TM x TN blocks per wave, NW waves) applies RoPE in its own
// epilogue for head size hd: each wave row must span whole heads (rotation
// partners in one lane), and 8-wave tiles (256 VGPRs per wave) must keep
// their accumulators within 128 VGPRs to leave room for the rotation.
constexpr bool rope_in_tile(int tm, int tn, int nw, int hd) {
  return (16 * tn) % hd == 0 && (nw == 4 || tm * tn <= 32);
}

// QKV epilogue of one accumulator row (TN fragments of 4 columns, starting at
// a head boundary nbase): q and k heads are rotated pairwise (column j with
// j + hd/2, PAIR = hd/32 fragments apart, both in this lane) with the row's
// cos/sin; q is stored to C, k and v to the token's pool slot.
template <int TN, int PAIR>
__device__ __forceinline__ void qkv_rope_row(const GemmArgs& a, const f32x4 (&acc)[TN], int m, int nbase, int cq) {
  constexpr int HD = 32 * PAIR, HALF = HD / 2;
  const int qk_end = (a.nq + a.nkv) * HD;
  const int slotm = a.tok_slot[m];
  const int blk = slotm >> 4, slot = slotm & 15;
  const float* csr = a.rope_cs + (size_t)m * HD;
#pragma unroll
  for (int ni = 0; ni < TN; ++ni) {
    const int n = nbase + 16 * ni + cq;
    if (n >= a.N) continue;
    if (n < qk_end) {
      if ((ni % (2 * PAIR)) >= PAIR) continue;  // upper half: done with its partner
      const f32x4 lo = acc[ni], hi = acc[ni + PAIR < TN ? ni + PAIR : TN - 1];
      const int j = n % HD;
      const u32x4 c4 = ld16(csr + j), s4 = ld16(csr + HALF + j);
      float rl[4], rh[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float c = __uint_as_float(c4[e]), sn = __uint_as_float(s4[e]);
        rl[e] = lo[e] * c - hi[e] * sn;
        rh[e] = hi[e] * c + lo[e] * sn;
      }
      const u32x2 wl = {pack_bf16x2(rl[0], rl[1]), pack_bf16x2(rl[2], rl[3])};
      const u32x2 wh = {pack_bf16x2(rh[0], rh[1]), pack_bf16x2(rh[2], rh[3])};
      if (n < a.nq * HD) {
        uint16_t* dst = reinterpret_cast<uint16_t*>(a.C) + (size_t)m * a.ldc + (n - j);
        st8(dst + j, wl);
        st8(dst + HALF + j, wh);
      } else {
        const int g = (n - a.nq * HD) / HD;
        uint16_t* kb = a.k_pool + ((size_t)blk * a.nkv + g) * 16 * HD;
        st8(kb + k_block_offset(slot, j, HD), wl);
        st8(kb + k_block_offset(slot, HALF + j, HD), wh);
      }
    } else {
      const int g = (n - qk_end) / HD, d = n % HD;
      uint16_t* vp = a.v_pool + ((size_t)blk * a.nkv + g) * 16 * HD + ((slot >> 3) * HD + d) * 8 + (slot & 7);
#pragma unroll
      for (int e = 0; e < 4; ++e) vp[8 * e] = (uint16_t)f32_to_bf16(acc[ni][e]);
    }
  }
}

// One accumulator row of a plain or residual epilogue: 4 columns per
// fragment, TN fragments 16 columns apart from column nbase. RK: residual
// none (0), bf16 (1) or fp32 (2); CF: fp32 (else bf16) output. All residual
// loads are issued before the first add.
template <int TN, int RK, bool CF>
__device__ __forceinline__ void residual_row(const GemmArgs& a, const f32x4 (&acc)[TN], int m, int nbase) {
  f32x4 r[TN];
#pragma unroll
  for (int ni = 0; ni < TN; ++ni) {
    const int n = min(nbase + 16 * ni, a.N - 4);
    if (RK == 2) {
      const u32x4 rr = ld16(reinterpret_cast<const float*>(a.R) + (size_t)m * a.ldr + n);
      r[ni] = f32x4{__uint_as_float(rr[0]), __uint_as_float(rr[1]), __uint_as_float(rr[2]), __uint_as_float(rr[3])};
    } else if (RK == 1) {
      const u32x2 rr = ld8(reinterpret_cast<const uint16_t*>(a.R) + (size_t)m * a.ldr + n);
      r[ni] = f32x4{bf16_lo(rr[0]), bf16_hi(rr[0]), bf16_lo(rr[1]), bf16_hi(rr[1])};
    } else {
      r[ni] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
#pragma unroll
  for (int ni = 0; ni < TN; ++ni) {
    const int n = nbase + 16 * ni;
    if (n >= a.N) continue;
    const f32x4 c = acc[ni] + r[ni];
    if (CF) {
      const u32x4 o = {__float_as_uint(c[0]), __float_as_uint(c[1]), __float_as_uint(c[2]), __float_as_uint(c[3])};
      st16(reinterpret_cast<float*>(a.C) + (size_t)m * a.ldc + n, o);
    } else {
      const u32x2 o = {pack_bf16x2(c[0], c[1]), pack_bf16x2(c[2], c[3])};
      st8(reinterpret_cast<uint16_t*>(a.C) + (size_t)m * a.ldc + n, o);
    }
  }
}

template <int TM, int TN, int WR, int WC, int S, int EPI>
__global__ __launch_bounds__(64 * WR * WC) void gemm_pipe_kernel(GemmArgs a, int tiles_m, int tiles_n, int ksplit,
                                                                  int kchunk, float* __restrict__ partial) {
  constexpr int NW = WR * WC;
  constexpr int WM = 16 * TM, WN = 16 * TN, BM = WM * WR, BN = WN * WC;
  constexpr int A_BYTES = BM * 128, STAGE_BYTES = (BM + BN) * 128;
  constexpr int LA = BM / 8, LB = BN / 8;                      // 1-KB loads per stage
  constexpr int NA = (LA + NW - 1) / NW, NB = (LB + NW - 1) / NW;  // load slots per wave
  constexpr int LOADS = LA / NW + LB / NW;                     // fewest loads any wave issues
  static_assert(S >= 2 && (S - 2) * LOADS < 64, "stage count");
  static_assert(EPI != GEMM_SWIGLU || (TN % 2 == 0), "gate/up pairs");
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int wm = wave / WC, wn = wave % WC;
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

  // Load offsets (bytes): the first row of each of this wave's 8-row groups
  // is wave-uniform; a lane adds row lrow and its swizzled 16-byte chunk.
  // A rows past M read the caller's padding rows (they only feed outputs that
  // are never stored); B row groups past N are clamped whole (N % 8 == 0).
  const int lrow = lane >> 3;
  const int lchunk = (lane & 7) ^ lrow;
  const uint32_t la = 2u * (uint32_t)(lrow * a.lda + 8 * lchunk), lb = 2u * (uint32_t)(lrow * a.ldb + 8 * lchunk);
  uint32_t ao[NA], bo[NB];
#pragma unroll
  for (int j = 0; j < NA; ++j) ao[j] = 2u * (uint32_t)(m0 + min(8 * (j * NW + wave), BM - 8)) * (uint32_t)a.lda;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int r8 = min(8 * (j * NW + wave), BN - 8);
    int brow;
    if (EPI == GEMM_SWIGLU) {
      const int c = min(nt * (BN / 2) + (r8 % (BN / 2)), N - 8);
      brow = (r8 < BN / 2) ? c : N + c;
    } else {
      brow = min(nt * BN + r8, N - 8);
    }
    bo[j] = 2u * (uint32_t)brow * (uint32_t)a.ldb;
  }
  const __amdgpu_buffer_rsrc_t ra = buffer_rsrc(a.A + k_begin, (uint32_t)kOperandWindow);
  const __amdgpu_buffer_rsrc_t rb = buffer_rsrc(a.B + k_begin, (uint32_t)kOperandWindow);

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Fragment rows of a wave differ by multiples of 8, so the chunk swizzle
  // (row & 7) is that of the lane's own row: every fragment address is one
  // per-lane base plus a compile-time offset. K half kc flips chunk bit 2.
  const int fr = lane & 15, fg = lane >> 4;
  const int swz = ((fg ^ (fr & 7)) << 4);
  const int a_lane = (wm * WM + fr) * 128 + swz;
  const int b_lane = A_BYTES + (EPI == GEMM_SWIGLU ? wn * (WN / 2) : wn * WN) * 128 + fr * 128 + swz;
  int broff[TN];
#pragma unroll
  for (int ni = 0; ni < TN; ++ni)
    broff[ni] = 128 * ((EPI == GEMM_SWIGLU) ? ((ni < TN / 2) ? 16 * ni : BN / 2 + 16 * (ni - TN / 2)) : 16 * ni);

  bf16x8 fa0[TM], fb0[TN], fa1[TM], fb1[TN];

#pragma unroll
  for (int s = 0; s < S; ++s)
    if (s < nk) issue_stage<NW, LA, LB, NA, NB>(smem + s * STAGE_BYTES, A_BYTES, ra, rb, ao, bo, la, lb, wave, s * 128);
  // stage 0 complete: the later prologue stages may stay in flight
  {
    const int pend = min(S, nk) - 1;
    if (S >= 4 && pend >= 3) wait_vmcnt<(S >= 4 ? 3 * LOADS : 0)>();
    else if (S >= 3 && pend >= 2) wait_vmcnt<(S >= 3 ? 2 * LOADS : 0)>();
    else if (pend >= 1) wait_vmcnt<LOADS>();
    else wait_vmcnt<0>();
  }
  __builtin_amdgcn_s_barrier();
  read_frags<TM, TN>(fa0, fb0, smem + a_lane, smem + b_lane, broff);
  __builtin_amdgcn_sched_barrier(0);

  // (the last stage is peeled so that every loop body is one straight block
  // in which reads and MFMAs can be interleaved)
  const int pend = min(S, nk) - 2;
  for (int kt = 0; kt < nk - 1; ++kt) {
    const int buf = kt % S;
    const uint8_t* st = smem + buf * STAGE_BYTES;
    // first K half: read the second half's fragments under the MFMAs
    read_frags<TM, TN>(fa1, fb1, st + (a_lane ^ 64), st + (b_lane ^ 64), broff);
    mfma_block<TM, TN>(acc, fa0, fb0);
    interleave_reads<TM + TN, TM * TN>();
    __builtin_amdgcn_sched_barrier(0);
    // this buffer is fully read (second-half fragments are in registers);
    // the next stage must be complete, the later ones may stay in flight
    wait_lgkm0();
    // the prologue issued min(S, nk) stages and every iteration one more
    // (past the end: the last stage again, into a buffer no later stage
    // reads), so min(S, nk) - 2 stages may stay in flight
    if (pend >= S - 2) wait_vmcnt<(S - 2) * LOADS>();
    else if (S >= 4 && pend >= 2) wait_vmcnt<(S >= 4 ? 2 * LOADS : 0)>();
    else if (S >= 3 && pend >= 1) wait_vmcnt<(S >= 3 ? LOADS : 0)>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    // second K half: refill this buffer with the stage S ahead and read the
    // next stage's first half, both under this half's MFMAs
    issue_stage<NW, LA, LB, NA, NB>(smem + buf * STAGE_BYTES, A_BYTES, ra, rb, ao, bo, la, lb, wave,
                                    min(kt + S, nk - 1) * 128);
    const uint8_t* nx = smem + ((kt + 1) % S) * STAGE_BYTES;
    read_frags<TM, TN>(fa0, fb0, nx + a_lane, nx + b_lane, broff);
    mfma_block<TM, TN>(acc, fa1, fb1);
    interleave_loads_reads<NA + NB, TM + TN, TM * TN>();
    __builtin_amdgcn_sched_barrier(0);
  }
  if (nk > 0) {
    const uint8_t* st = smem + ((nk - 1) % S) * STAGE_BYTES;
    read_frags<TM, TN>(fa1, fb1, st + (a_lane ^ 64), st + (b_lane ^ 64), broff);
    mfma_block<TM, TN>(acc, fa0, fb0);
    interleave_reads<TM + TN, TM * TN>();
    __builtin_amdgcn_sched_barrier(0);
    mfma_block<TM, TN>(acc, fa1, fb1);
  }
  // the loads issued past the end land in LDS before the workgroup ends
  wait_vmcnt<0>();

  // epilogue: acc[mi][ni][i] = C[m][n + i]. Fragment rows go in groups of
  // EPB, whose loads (residual, or cos/sin and pool slots) are in flight
  // together: one memory round trip per group, about 16 TN registers per
  // group. The K loop's fragment registers cover that in 4-wave tiles; the
  // 8-wave tiles (two waves per SIMD) would spill, and take one row at a time.
  constexpr int EPB = (NW == 4 && 16 / TN > 1) ? 16 / TN : 1;
  const int cq = fg << 2;
#pragma unroll
  for (int mi = 0; mi < TM; ++mi) {
    if (mi % EPB == 0) __builtin_amdgcn_sched_barrier(0);
    const int m = m0 + wm * WM + 16 * mi + fr;
    if (m >= M) continue;
    if (ksplit > 1) {
      // fp32 partial sums, rows of partial_width(N) columns: the reduce
      // kernel applies the epilogue (SwiGLU: gate at n, up at N + n)
      const int W = (EPI == GEMM_SWIGLU) ? 2 * N : N;
      float* prow = partial + ((size_t)ks * M + m) * W;
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) {
        int n, col;
        if (EPI == GEMM_SWIGLU) {
          n = nt * (BN / 2) + wn * (WN / 2) + 16 * (ni % (TN / 2)) + cq;
          col = ni < TN / 2 ? n : N + n;
        } else {
          n = nt * BN + wn * WN + 16 * ni + cq;
          col = n;
        }
        if (n >= N) continue;
        const f32x4 c = acc[mi][ni];
        st16(prow + col, u32x4{__float_as_uint(c[0]), __float_as_uint(c[1]), __float_as_uint(c[2]), __float_as_uint(c[3])});
      }
      continue;
    }
    if (EPI == GEMM_QKV_ROPE) {
      // the planner sends tiles that cannot rotate in-tile (rope_in_tile)
      // through a K split, so their rows are not built
      if constexpr (rope_in_tile(TM, TN, NW, 128)) {
        if (a.hd == 128) qkv_rope_row<TN, 4>(a, acc[mi], m, nt * BN + wn * WN, cq);
        else qkv_rope_row<TN, 2>(a, acc[mi], m, nt * BN + wn * WN, cq);
      } else if constexpr (rope_in_tile(TM, TN, NW, 64)) {
        if (a.hd == 64) qkv_rope_row<TN, 2>(a, acc[mi], m, nt * BN + wn * WN, cq);
      }
      continue;
    }
    if (EPI == GEMM_SWIGLU) {
#pragma unroll
      for (int ni = 0; ni < TN / 2; ++ni) {
        const int n = nt * (BN / 2) + wn * (WN / 2) + 16 * ni + cq;
        if (n >= N) continue;
        const f32x4 gt = acc[mi][ni], up = acc[mi][ni + TN / 2];
        u32x2 o;
        o[0] = pack_bf16x2(silu_f(gt[0]) * up[0], silu_f(gt[1]) * up[1]);
        o[1] = pack_bf16x2(silu_f(gt[2]) * up[2], silu_f(gt[3]) * up[3]);
        st8(reinterpret_cast<uint16_t*>(a.C) + (size_t)m * a.ldc + n, o);
      }
    } else if (EPI == GEMM_RESIDUAL) {
      // one straight-line row per residual / output kind (the kinds are
      // uniform over the launch)
      const int nb = nt * BN + wn * WN + cq;
      if (!a.R) {
        if (a.c_f32) residual_row<TN, 0, true>(a, acc[mi], m, nb);
        else residual_row<TN, 0, false>(a, acc[mi], m, nb);
      } else if (a.r_f32) {
        if (a.c_f32) residual_row<TN, 2, true>(a, acc[mi], m, nb);
        else residual_row<TN, 2, false>(a, acc[mi], m, nb);
      } else {
        if (a.c_f32) residual_row<TN, 1, true>(a, acc[mi], m, nb);
        else residual_row<TN, 1, false>(a, acc[mi], m, nb);
      }
    } else {
      residual_row<TN, 0, false>(a, acc[mi], m, nt * BN + wn * WN + cq);
    }
  }
}

// Sum of the split-K partials in split order, then the GEMM's epilogue: for
// the QKV GEMM the RoPE rotation of q and k and the pool scatter of k and v
// (a work item is 4 columns of a row and their rotation partners), for
// gate/up the SwiGLU product, else the residual add and the store.
// Largest K split the planner chooses; the reduce kernels are instantiated
// per split count so that all of a work item's partial loads are in flight
// together.
constexpr int kMaxKSplit = 8;

// Four consecutive fp32 partials summed over the KS splits, in split order.
template <int KS>
__device__ __forceinline__ f32x4 sum_splits(const float* p, size_t stride) {
  u32x4 v[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) v[s] = ld16(p + s * stride);
  f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < KS; ++s)
#pragma unroll
    for (int j = 0; j < 4; ++j) c[j] += __uint_as_float(v[s][j]);
  return c;
}

template <int EPI, int KS>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs a, const float* __restrict__ partial) {
  const int W = (EPI == GEMM_SWIGLU) ? 2 * a.N : a.N;
  const size_t split_stride = (size_t)a.M * W;
  auto sum4 = [&](int m, int n) { return sum_splits<KS>(partial + (size_t)m * W + n, split_stride); };
  const int64_t step = (int64_t)gridDim.x * 256;
  if (EPI == GEMM_QKV_ROPE) {
    // Workgroups [0, M * qk_wgs): one row each, a thread one (q or k head,
    // 4 columns and their rotation partners). The rest: V, one wave item of
    // (kv head, 32 dimensions, 8 consecutive rows) per wave, lane = (row
    // lane % 8, 4 dimensions lane / 8), so the 8 lanes of a dimension write
    // the 8 slots of one 16-byte V group together: a chunk's V lines are
    // written whole by one wave instead of 2 bytes at a time.
    const int hd = a.hd, half = hd / 2, qk_heads = a.nq + a.nkv;
    const int qs = half / 4;  // work items per q/k head (a power of two)
    const int qs_log = __builtin_ctz(qs);
    const int qk_units = qk_heads * qs, qk_wgs = (qk_units + 255) / 256;
    const int b = blockIdx.x;
    if (b < a.M * qk_wgs) {
      const int m = b / qk_wgs, r = (b - m * qk_wgs) * 256 + threadIdx.x;
      if (r >= qk_units) return;
      const int h = r >> qs_log, j = (r & (qs - 1)) * 4;
      const float* csr = a.rope_cs + (size_t)m * hd;
      const f32x4 lo = sum4(m, h * hd + j), hi = sum4(m, h * hd + half + j);
      const u32x4 c4 = ld16(csr + j), s4 = ld16(csr + half + j);
      float rl[4], rh[4];
      for (int e = 0; e < 4; ++e) {
        const float c = __uint_as_float(c4[e]), sn = __uint_as_float(s4[e]);
        rl[e] = lo[e] * c - hi[e] * sn;
        rh[e] = hi[e] * c + lo[e] * sn;
      }
      const u32x2 wl = {pack_bf16x2(rl[0], rl[1]), pack_bf16x2(rl[2], rl[3])};
      const u32x2 wh = {pack_bf16x2(rh[0], rh[1]), pack_bf16x2(rh[2], rh[3])};
      if (h < a.nq) {
        uint16_t* dst = reinterpret_cast<uint16_t*>(a.C) + (size_t)m * a.ldc + h * hd;
        st8(dst + j, wl);
        st8(dst + half + j, wh);
      } else {
        const int slotm = a.tok_slot[m], slot = slotm & 15;
        uint16_t* kb = a.k_pool + ((size_t)(slotm >> 4) * a.nkv + (h - a.nq)) * 16 * hd;
        st8(kb + k_block_offset(slot, j, hd), wl);
        st8(kb + k_block_offset(slot, half + j, hd), wh);
      }
      return;
    }
    const int dblocks = hd / 32;
    const int item = (b - a.M * qk_wgs) * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int rb = item / (a.nkv * dblocks), rem = item - rb * (a.nkv * dblocks);
    const int g = rem / dblocks, d = 32 * (rem - g * dblocks) + 4 * (lane >> 3);
    const int m = 8 * rb + (lane & 7);
    if (m >= a.M) return;
    const f32x4 c = sum4(m, (qk_heads + g) * hd + d);
    const int slotm = a.tok_slot[m], slot = slotm & 15;
    uint16_t* vp = a.v_pool + ((size_t)(slotm >> 4) * a.nkv + g) * 16 * hd + ((slot >> 3) * hd + d) * 8 + (slot & 7);
    for (int e = 0; e < 4; ++e) vp[8 * e] = (uint16_t)f32_to_bf16(c[e]);
    return;
  }
  const int64_t nvec = (int64_t)a.M * a.N / 4;
  for (int64_t v = blockIdx.x * 256ll + threadIdx.x; v < nvec; v += step) {
    const int64_t e = v * 4;
    const int m = (int)(e / a.N), n = (int)(e - (int64_t)m * a.N);
    f32x4 c = sum4(m, n);
    if (EPI == GEMM_SWIGLU) {
      const f32x4 up = sum4(m, a.N + n);
      const u32x2 o = {pack_bf16x2(silu_f(c[0]) * up[0], silu_f(c[1]) * up[1]),
                       pack_bf16x2(silu_f(c[2]) * up[2], silu_f(c[3]) * up[3])};
      st8(reinterpret_cast<uint16_t*>(a.C) + (size_t)m * a.ldc + n, o);
      continue;
    }
    if (EPI == GEMM_RESIDUAL && a.R) {
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

// Split-K reduce of the fp32 residual GEMM fused with the RMSNorm that
// follows it: one workgroup per row sums the partials in split order, adds the
// residual, stores the row (fp32) and normalises it into norm_out (bf16), with
// the same element-to-thread mapping and reduction order as the RMSNorm kernel.
template <int MAXV, int KS>
__global__ __launch_bounds__(256) void splitk_reduce_rmsnorm_kernel(GemmArgs a, const float* __restrict__ partial) {
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x, N = a.N;
  const int nvec = N >> 3;
  const size_t split_stride = (size_t)a.M * N;
  float v[MAXV][8];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int vi = tid + 256 * i;
    if (vi < nvec) {
      const float* p = partial + (size_t)row * N + 8 * vi;
      const f32x4 c0 = sum_splits<KS>(p, split_stride), c1 = sum_splits<KS>(p + 4, split_stride);
      float c[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
      if (!a.R) {
      } else if (a.r_f32) {
        const float* rr = reinterpret_cast<const float*>(a.R) + (size_t)row * a.ldr + 8 * vi;
        const u32x4 r0 = ld16(rr), r1 = ld16(rr + 4);
        for (int j = 0; j < 4; ++j) { c[j] += __uint_as_float(r0[j]); c[4 + j] += __uint_as_float(r1[j]); }
      } else {
        const u32x4 rr = ld16(reinterpret_cast<const uint16_t*>(a.R) + (size_t)row * a.ldr + 8 * vi);
        for (int j = 0; j < 4; ++j) { c[2 * j] += bf16_lo(rr[j]); c[2 * j + 1] += bf16_hi(rr[j]); }
      }
      float* cr = reinterpret_cast<float*>(a.C) + (size_t)row * a.ldc + 8 * vi;
      st16(cr, u32x4{__float_as_uint(c[0]), __float_as_uint(c[1]), __float_as_uint(c[2]), __float_as_uint(c[3])});
      st16(cr + 4, u32x4{__float_as_uint(c[4]), __float_as_uint(c[5]), __float_as_uint(c[6]), __float_as_uint(c[7])});
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        v[i][j] = c[j];
        ss += c[j] * c[j];
      }
    }
  }
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float r = 1.0f / sqrtf(tot / (float)N + a.norm_eps);
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int vi = tid + 256 * i;
    if (vi < nvec) {
      u32x4 gw = ld16(a.norm_g + 8 * vi), o;
      for (int j = 0; j < 4; ++j)
        o[j] = pack_bf16x2(v[i][2 * j] * r * bf16_lo(gw[j]), v[i][2 * j + 1] * r * bf16_hi(gw[j]));
      st16(a.norm_out + (size_t)row * N + 8 * vi, o);
    }
  }
}

}  // namespace gemm_detail

namespace {
using namespace gemm_detail;

struct TileCfg {
  int tm, tn, wr, wc, stages;  // per-wave MFMA blocks, wave grid, LDS stages
  // measured cost (us) of one 64-wide K stage: in a launch's first round with
  // one workgroup per CU, in a first round with two per CU (4-wave tiles with
  // small LDS rings only), in each later round (the weights then come from
  // the caches, not HBM); and a fixed cost per round
  float first_alone_us, first_pair_us, next_us, fixed_us;
};
// Accumulators and both fragment sets stay within the 256 VGPRs of a wave.
// 8-wave workgroups put two waves on each SIMD; 4-wave ones with LDS rings
// of at most 80 KB run two workgroups per CU. The costs were fitted to
// MI355X timings of the layer's four GEMMs at M = 384, 576, 1056, 2048 and
// 2374 (the first 14 shapes x splits 1, 2, 3, 4, 6, 8); the last shape's are
// the 192 x 384 tile's scaled by their measured time ratio (0.945).
constexpr TileCfg kTiles[] = {
    {8, 4, 2, 2, 3, 0.978f, 0.978f, 0.920f, 0.00f},  {4, 8, 2, 2, 3, 1.046f, 1.046f, 0.850f, 4.61f},
    {4, 4, 2, 2, 2, 0.849f, 1.040f, 0.798f, 9.68f},  {6, 4, 2, 2, 2, 1.012f, 1.458f, 1.260f, 1.14f},
    {3, 8, 2, 2, 3, 0.961f, 0.961f, 0.779f, 0.00f},  {9, 4, 2, 2, 3, 1.073f, 1.073f, 1.039f, 0.00f},
    {2, 8, 2, 2, 3, 0.911f, 0.911f, 0.690f, 0.00f},  {8, 4, 2, 4, 2, 1.525f, 1.525f, 1.353f, 8.74f},
    {6, 4, 2, 4, 2, 1.411f, 1.411f, 1.188f, 7.69f},  {4, 4, 2, 4, 3, 0.999f, 0.999f, 0.863f, 2.13f},
    {4, 8, 4, 2, 2, 1.512f, 1.512f, 1.305f, 10.75f}, {3, 8, 4, 2, 2, 1.427f, 1.427f, 1.235f, 5.37f},
    {2, 8, 4, 2, 3, 1.000f, 1.000f, 0.857f, 4.33f},  {6, 6, 2, 4, 2, 1.636f, 1.636f, 1.499f, 12.96f},
    {9, 4, 2, 4, 2, 1.546f, 1.546f, 1.417f, 12.96f},
};
constexpr int kNumTiles = (int)(sizeof(kTiles) / sizeof(kTiles[0]));

template <int TM, int TN, int WR, int WC, int ST, int EPI>
void launch_tile(hipStream_t s, const GemmArgs& a, int tiles_m, int tiles_n, int ksplit, int kchunk, float* partial) {
  constexpr int lds = ST * 16 * (TM * WR + TN * WC) * 128;
  static_assert(lds <= 160 * 1024, "LDS");
  static std::atomic<uint64_t> lds_raised{0};
  raise_dynamic_lds(reinterpret_cast<const void*>(&gemm_pipe_kernel<TM, TN, WR, WC, ST, EPI>), lds, lds_raised);
  gemm_pipe_kernel<TM, TN, WR, WC, ST, EPI>
      <<<tiles_m * tiles_n * ksplit, 64 * WR * WC, lds, s>>>(a, tiles_m, tiles_n, ksplit, kchunk, partial);
}

template <int EPI>
void launch_cfg(int idx, hipStream_t s, const GemmArgs& a, int tm, int tn, int ks, int kchunk, float* part) {
  switch (idx) {
    case 0: launch_tile<8, 4, 2, 2, 3, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 1: launch_tile<4, 8, 2, 2, 3, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 2: launch_tile<4, 4, 2, 2, 2, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 3: launch_tile<6, 4, 2, 2, 2, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 4: launch_tile<3, 8, 2, 2, 3, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 5: launch_tile<9, 4, 2, 2, 3, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 6: launch_tile<2, 8, 2, 2, 3, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 7: launch_tile<8, 4, 2, 4, 2, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 8: launch_tile<6, 4, 2, 4, 2, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 9: launch_tile<4, 4, 2, 4, 3, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 10: launch_tile<4, 8, 4, 2, 2, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 11: launch_tile<3, 8, 4, 2, 2, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 12: launch_tile<2, 8, 4, 2, 3, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    case 13: launch_tile<6, 6, 2, 4, 2, EPI>(s, a, tm, tn, ks, kchunk, part); break;
    default: launch_tile<9, 4, 2, 4, 2, EPI>(s, a, tm, tn, ks, kchunk, part); break;
  }
}

// The reduce grids fit one wave of workgroups over the chip (about four per
// CU), each thread looping over an equal share of the work items: short
// workgroups in a second, mostly empty round cost more than the loop.
constexpr int kReduceWgs = 1024;

template <int EPI, int KS>
void launch_reduce_ks(hipStream_t s, const GemmArgs& a, const float* partial) {
  if (EPI == GEMM_QKV_ROPE) {
    // q/k rows, then V wave items (kv head, 32 dimensions, 8 rows), 4 per workgroup
    const int qk_units = (a.nq + a.nkv) * (a.hd / 8);
    const int v_items = a.nkv * (a.hd / 32) * ((a.M + 7) / 8);
    splitk_reduce_kernel<EPI, KS><<<a.M * ((qk_units + 255) / 256) + (v_items + 3) / 4, 256, 0, s>>>(a, partial);
  } else {
    const int64_t wgs = ((int64_t)a.M * a.N / 4 + 255) / 256;
    const int64_t per = (wgs + kReduceWgs - 1) / kReduceWgs;
    splitk_reduce_kernel<EPI, KS><<<(int)((wgs + per - 1) / per), 256, 0, s>>>(a, partial);
  }
}

template <int EPI>
void launch_reduce(hipStream_t s, const GemmArgs& a, int ks, const float* partial) {
  static_assert(kMaxKSplit == 8, "one case per split count");
  switch (ks) {
    case 2: launch_reduce_ks<EPI, 2>(s, a, partial); break;
    case 3: launch_reduce_ks<EPI, 3>(s, a, partial); break;
    case 4: launch_reduce_ks<EPI, 4>(s, a, partial); break;
    case 5: launch_reduce_ks<EPI, 5>(s, a, partial); break;
    case 6: launch_reduce_ks<EPI, 6>(s, a, partial); break;
    case 7: launch_reduce_ks<EPI, 7>(s, a, partial); break;
    default: launch_reduce_ks<EPI, 8>(s, a, partial); break;
  }
}

template <int MAXV>
void launch_reduce_rmsnorm(hipStream_t s, const GemmArgs& a, int ks, const float* partial) {
  switch (ks) {
    case 2: splitk_reduce_rmsnorm_kernel<MAXV, 2><<<a.M, 256, 0, s>>>(a, partial); break;
    case 3: splitk_reduce_rmsnorm_kernel<MAXV, 3><<<a.M, 256, 0, s>>>(a, partial); break;
    case 4: splitk_reduce_rmsnorm_kernel<MAXV, 4><<<a.M, 256, 0, s>>>(a, partial); break;
    case 5: splitk_reduce_rmsnorm_kernel<MAXV, 5><<<a.M, 256, 0, s>>>(a, partial); break;
    case 6: splitk_reduce_rmsnorm_kernel<MAXV, 6><<<a.M, 256, 0, s>>>(a, partial); break;
    case 7: splitk_reduce_rmsnorm_kernel<MAXV, 7><<<a.M, 256, 0, s>>>(a, partial); break;
    default: splitk_reduce_rmsnorm_kernel<MAXV, 8><<<a.M, 256, 0, s>>>(a, partial); break;
  }
}
}  // namespace

int gemm_tile_count() { return kNumTiles; }

int partial_width(const GemmArgs& a) { return a.epi == GEMM_SWIGLU ? 2 * a.N : a.N; }

// Cost model (microseconds): workgroups run in rounds of one (two, for small
// LDS rings) per CU; the first round costs its K stages at the tile's
// first-round rate (for one or two workgroups per CU), every later round at
// the later-round rate, plus a fixed cost per round; a K split adds the fp32
// partials' round trip (fitted at 5.1 TB/s) and the reduce launch.
static int tiles_per_cu(const TileCfg& c) {
  const int lds = c.stages * 16 * (c.tm * c.wr + c.tn * c.wc) * 128;
  return (c.wr * c.wc == 4 && 2 * lds <= 160 * 1024) ? 2 : 1;
}

static GemmPlan search_plan(const GemmArgs& a, int cu_count, int force_cfg, int force_ksplit) {
  GemmPlan best{-1, 0, 0, 1, 0};
  double best_cost = 1e300;
  const int ksteps = a.K / 64;
  // tiles that cannot rotate in their epilogue take QKV with a K split, whose
  // reduce kernel rotates
  auto fits = [&](const TileCfg& c, int ks) {
    return a.epi != GEMM_QKV_ROPE || ks > 1 || rope_in_tile(c.tm, c.tn, c.wr * c.wc, a.hd);
  };
  const int W = partial_width(a);
  for (int i = 0; i < kNumTiles; ++i) {
    if (force_cfg >= 0 && i != force_cfg) continue;
    const TileCfg& c = kTiles[i];
    const int bm = 16 * c.tm * c.wr, bn = 16 * c.tn * c.wc;
    const int ncols = (a.epi == GEMM_SWIGLU) ? bn / 2 : bn;
    const int tm = (a.M + bm - 1) / bm, tn = (a.N + ncols - 1) / ncols;
    const int slots = std::max(1, cu_count) * tiles_per_cu(c);
    for (int ks = 1; ks <= kMaxKSplit; ++ks) {
      if (ks > 1 && ksteps < 4 * ks) break;
      if (force_ksplit > 0 && ks != force_ksplit) continue;
      if (!fits(c, ks)) continue;
      const int kst = (ksteps + ks - 1) / ks;
      if ((ks - 1) * kst >= ksteps) continue;  // every split gets at least one stage
      const int nwg = tm * tn * ks;
      const int cus = std::max(1, cu_count);
      const int rounds = (nwg + slots - 1) / slots;
      const float first = (slots > cus && nwg > cus) ? c.first_pair_us : c.first_alone_us;
      double cost = kst * (first + (rounds - 1) * c.next_us) + rounds * c.fixed_us;
      if (ks > 1) cost += (double)a.M * W * 4.0 * (2 * ks + 1) / 5.12e6 + 1.6;
      if (cost < best_cost * 0.999) {
        best_cost = cost;
        best = GemmPlan{i, tm, tn, ks, kst * 64};
      }
    }
  }
  return best;
}

GemmPlan plan_gemm(const GemmArgs& a, int cu_count, int force_cfg, int force_ksplit) {
  if (a.K % 64 != 0 || a.N % 8 != 0) return GemmPlan{-1, 0, 0, 1, 0};
  if (force_cfg >= kNumTiles) force_cfg = -1;
  // a forced shape or split that cannot run this GEMM is relaxed: first the
  // split, then the shape
  GemmPlan p = search_plan(a, cu_count, force_cfg, force_ksplit);
  if (p.cfg < 0) p = search_plan(a, cu_count, force_cfg, 0);
  if (p.cfg < 0) p = search_plan(a, cu_count, -1, 0);
  return p;
}

bool launch_gemm(hipStream_t s, const GemmArgs& a, const GemmPlan& p, float* partial) {
  if (a.M <= 0 || a.N <= 0) return false;
  if (p.cfg < 0) {
    launch_gemm_regstaged(s, a);
    return false;
  }
  switch (a.epi) {
    case GEMM_STORE_BF16: launch_cfg<GEMM_STORE_BF16>(p.cfg, s, a, p.tiles_m, p.tiles_n, p.ksplit, p.kchunk, partial); break;
    case GEMM_QKV_ROPE: launch_cfg<GEMM_QKV_ROPE>(p.cfg, s, a, p.tiles_m, p.tiles_n, p.ksplit, p.kchunk, partial); break;
    case GEMM_RESIDUAL: launch_cfg<GEMM_RESIDUAL>(p.cfg, s, a, p.tiles_m, p.tiles_n, p.ksplit, p.kchunk, partial); break;
    default: launch_cfg<GEMM_SWIGLU>(p.cfg, s, a, p.tiles_m, p.tiles_n, p.ksplit, p.kchunk, partial); break;
  }
  if (p.ksplit > 1 && a.epi == GEMM_RESIDUAL && a.c_f32 && a.norm_out && a.N % 8 == 0 && a.ldc == a.N &&
      a.N <= 8 * 256 * 8) {
    const int nvec = a.N / 8;
    if (nvec <= 256) launch_reduce_rmsnorm<1>(s, a, p.ksplit, partial);
    else if (nvec <= 1024) launch_reduce_rmsnorm<4>(s, a, p.ksplit, partial);
    else launch_reduce_rmsnorm<8>(s, a, p.ksplit, partial);
    return true;
  }
  if (p.ksplit > 1) {
    switch (a.epi) {
      case GEMM_QKV_ROPE: launch_reduce<GEMM_QKV_ROPE>(s, a, p.ksplit, partial); break;
      case GEMM_SWIGLU: launch_reduce<GEMM_SWIGLU>(s, a, p.ksplit, partial); break;
      case GEMM_RESIDUAL: launch_reduce<GEMM_RESIDUAL>(s, a, p.ksplit, partial); break;
      default: launch_reduce<GEMM_STORE_BF16>(s, a, p.ksplit, partial); break;
    }
  }
  return false;
}

}  // namespace hb
