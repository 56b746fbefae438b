// Host-side launch entry points of the gfx950 kernels (one per kernel family).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace hb {

// out[t][:] = bf16( x[t][:] / sqrt(mean(x[t]^2) + eps) * g ), x bf16 or fp32.
void launch_rmsnorm(hipStream_t s, const void* x, bool x_f32, const uint16_t* g, uint16_t* out, int T, int H,
                    float eps);

enum GemmEpilogue { GEMM_STORE_BF16 = 0, GEMM_RESIDUAL = 1, GEMM_SWIGLU = 2 };

// C[M][N] = A[M][K] * B[N][K]^T with an epilogue:
//   GEMM_STORE_BF16: C bf16
//   GEMM_RESIDUAL:   C = R + A B^T, R bf16 or fp32, C fp32 or bf16
//   GEMM_SWIGLU:     B has 2N rows [gate | up]; C bf16 = silu(A Bg^T) * (A Bu^T)
struct GemmArgs {
  const uint16_t* A; int lda;
  const uint16_t* B; int ldb;
  int M, N, K;
  void* C; int ldc; int c_f32;
  const void* R; int ldr; int r_f32;
  int epi;
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
// `partial` holds ksplit * M * N fp32 when plan.ksplit > 1.
void launch_gemm(hipStream_t s, const GemmArgs& a, const GemmPlan& plan, float* partial);

// Rotate q and k of every batch token at its position and store k and v in the
// paged pool; q goes to q_out [T][nq*hd].
struct RopeKvArgs {
  const uint16_t* qkv;  // [T][(nq + 2 nkv) hd]
  int T, nq, nkv, hd;
  const int32_t* tok_pos;
  const int32_t* tok_req;
  const int32_t* req_bt;
  const int32_t* bt;
  const double* inv_freq;  // [hd/2] theta^(-2j/hd)
  uint16_t* q_out;
  uint16_t* k_pool;
  uint16_t* v_pool;
};
void launch_rope_kv(hipStream_t s, const RopeKvArgs& a);

// Copy k, v [n][nkv][hd] into the pool slots of positions ctx..ctx+n-1.
void launch_append_kv(hipStream_t s, const uint16_t* k, const uint16_t* v, int n_tokens, int ctx,
                      const int32_t* bt, int nkv, int hd, uint16_t* k_pool, uint16_t* v_pool);

struct AttnArgs {
  const uint16_t* q;   // [T][nq*hd], rotated
  uint16_t* o;         // [T][nq*hd]
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* tiles;   // workgroup tiles (AttnItem)
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
void launch_flush(hipStream_t s, void* buf, int64_t bytes, uint32_t value);

}  // namespace hb
