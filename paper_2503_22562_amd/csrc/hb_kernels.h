// Host-side launch entry points of the gfx950 kernels (one per kernel family).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include <atomic>

#include "hb_plan.h"

namespace hb {

// A launch with more than 64 KB of dynamic LDS needs the kernel's limit
// raised first; HIP keeps that attribute per device, so it is raised once on
// each device the kernel runs on (done: one bit per device ordinal).
inline void raise_dynamic_lds(const void* kernel, int bytes, std::atomic<uint64_t>& done) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return;
  if (dev >= 64) {  // beyond the bit set: raise it on every call
    (void)hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    return;
  }
  const uint64_t bit = 1ull << dev;
  if (done.load(std::memory_order_acquire) & bit) return;
  if (hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes) == hipSuccess)
    done.fetch_or(bit, std::memory_order_release);
}

// Per-token RoPE inputs for the QKV epilogue, written by the first RMSNorm:
// cs[t][0..hd/2) = cos, cs[t][hd/2..hd) = sin of the angles pos(t) * inv_freq
// (formed and reduced mod 2 pi in fp64, evaluated in fp32), and slot[t] =
// 16 * pool block + slot of the token's new K/V.
struct RopePrep {
  const int32_t* tok_pos;
  const int32_t* tok_req;
  const int32_t* req_bt;
  const int32_t* bt;
  const double* inv_freq;
  int hd;
  float* cs;
  int32_t* slot;
};

// out[t][:] = bf16( x[t][:] / sqrt(mean(x[t]^2) + eps) * g ), x bf16 or fp32;
// with rope, also the RoPE inputs of every token.
void launch_rmsnorm(hipStream_t s, const void* x, bool x_f32, const uint16_t* g, uint16_t* out, int T, int H,
                    float eps, const RopePrep* rope = nullptr);

enum GemmEpilogue { GEMM_STORE_BF16 = 0, GEMM_RESIDUAL = 1, GEMM_SWIGLU = 2, GEMM_QKV_ROPE = 3 };

// Rows past M that a GEMM's A operand must keep readable (kGemmPadRows, in
// hb_plan.h): the LDS-pipelined kernels load whole row tiles (at most 288
// rows) and never store the rows past M. Their B operands need N % 8 == 0
// (8-row load groups). Every operand must fit kOperandWindow bytes.

// C[M][N] = A[M][K] * B[N][K]^T with an epilogue:
//   GEMM_STORE_BF16: C bf16
//   GEMM_RESIDUAL:   C = R + A B^T, R bf16 or fp32, C fp32 or bf16
//   GEMM_SWIGLU:     B has 2N rows [gate | up]; C bf16 = silu(A Bg^T) * (A Bu^T)
//   GEMM_QKV_ROPE:   the columns are [q heads | k heads | v heads] of head_dim
//                    each; q and k are rotated (rotate-half RoPE with the
//                    per-row cos/sin of rope_cs), q goes to C [M][nq*hd], k
//                    and v to the paged pool slot tok_slot[m]
// With a K split, the reduce kernel applies the epilogue. GEMM_RESIDUAL with
// fp32 C and norm_out set: the reduce also writes the RMSNorm of each C row
// (gain norm_g, epsilon norm_eps) to norm_out bf16 [M][N], one workgroup per
// row (launch_gemm then returns true; without a split it returns false and
// the caller normalises).
struct GemmArgs {
  const uint16_t* A; int lda;
  const uint16_t* B; int ldb;
  int M, N, K;
  void* C; int ldc; int c_f32;
  const void* R; int ldr; int r_f32;  // GEMM_RESIDUAL: residual added to the product (NULL: none)
  int epi;
  // GEMM_QKV_ROPE only
  const float* rope_cs; const int32_t* tok_slot;
  uint16_t* k_pool; uint16_t* v_pool;
  int nq, nkv, hd;
  // GEMM_RESIDUAL with a K split only: fused RMSNorm of the output rows
  const uint16_t* norm_g; uint16_t* norm_out; float norm_eps;
};
// Tile shape, grid and K split chosen for one GEMM (cfg < 0: the
// register-staged kernel, used when K is not a multiple of 64).
struct GemmPlan {
  int cfg, tiles_m, tiles_n, ksplit, kchunk;
};
// force_cfg >= 0 / force_ksplit > 0 restrict the choice to one tile shape /
// one K split where that split applies (testing).
GemmPlan plan_gemm(const GemmArgs& a, int cu_count, int force_cfg = -1, int force_ksplit = 0);
// Number of LDS-pipelined tile shapes (valid force_cfg values are 0..count-1).
int gemm_tile_count();
// Columns of one row of split-K partial sums (gate/up: 2 N, gate then up).
int partial_width(const GemmArgs& a);
// `partial` holds ksplit * M * partial_width(a) fp32 when plan.ksplit > 1.
// Returns true when the RMSNorm of the output rows was fused (see GemmArgs).
bool launch_gemm(hipStream_t s, const GemmArgs& a, const GemmPlan& plan, float* partial);

// Copy k, v [n][nkv][hd] into the pool slots of positions ctx..ctx+n-1.
void launch_append_kv(hipStream_t s, const uint16_t* k, const uint16_t* v, int n_tokens, int ctx,
                      const int32_t* bt, int nkv, int hd, uint16_t* k_pool, uint16_t* v_pool);

struct AttnArgs {
  const uint16_t* q;   // [T][nq*hd], rotated
  uint16_t* o;         // [T][nq*hd]
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* tiles;   // workgroup tiles (AttnItem)
  int n_tiles;
  const int32_t* items;   // wave items (AttnItem)
  int n_items;
  const int32_t* units;   // per workgroup: tile index, or -1 - (group of 4 items)
  int n_units;
  const int32_t* groups;
  int n_groups;
  const int32_t* merge_units;  // per merge workgroup: group * 16 + 16-column block
  int n_merge_units;
  const int32_t* req_bt;
  const int32_t* bt;
  float* part_o;   // [slots][hd]
  float* part_ml;  // [slots][2]
  int nq, nkv, hd;
  float scale_log2;  // log2(e) / sqrt(hd)
};
void launch_attention(hipStream_t s, const AttnArgs& a);
void launch_attn_merge(hipStream_t s, const AttnArgs& a);

// Seeded pseudo-random bf16 fill (profiling inputs).
void launch_fill_random_bf16(hipStream_t s, uint16_t* p, int64_t n, uint64_t seed, float scale);
// Fill whole pool blocks (K and V of every kv head) listed in blocks[n].
void launch_fill_blocks(hipStream_t s, const int32_t* blocks, int n, int nkv, int hd, uint16_t* k_pool,
                        uint16_t* v_pool, uint64_t seed);
// Overwrite a buffer (evicts earlier data from the Infinity Cache).
// Cold-cache preparation over buf[0, bytes): the first half is overwritten
// with `value`, then the second half is read, so that the caches hold no data
// of the caller's and none of the written lines are left dirty (their
// write-back would otherwise fall into whatever runs next).
void launch_flush(hipStream_t s, void* buf, int64_t bytes, uint32_t value);

// Sustained-rate probes (k_probe.hip): waves reading random 4-KB chunks of
// buf[0, 4096 n_chunks), a grid-stride read of buf[0, bytes), and a loop of
// bf16 MFMAs (blocks x 4 waves x iters x 16 of them). sink: a device word the
// kernels write only in a case that does not occur in practice.
void launch_probe_random_read(hipStream_t s, const void* buf, uint32_t n_chunks, int blocks, int iters,
                              uint32_t* sink);
void launch_probe_stream_read(hipStream_t s, const void* buf, int64_t bytes, int blocks, uint32_t* sink);
void launch_probe_mfma(hipStream_t s, int blocks, int iters, uint32_t* sink);
// out[r][:] = src[clamp(rows[r], 0, n_src - 1)][:] (bf16 rows of H, H % 8 == 0).
void launch_gather_rows(hipStream_t s, const uint16_t* src, int64_t n_src, const int32_t* rows, int n_rows, int H,
                        uint16_t* out);
// out[r] = index of the largest of x[r][0..V) (lowest index on ties).
void launch_argmax(hipStream_t s, const float* x, int n_rows, int V, int32_t* out);

}  // namespace hb
