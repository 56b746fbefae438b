// Varlen paged attention for a hybrid batch: causal chunk rows over their
// request's cached context and single-token decode rows, in one launch.
//
// Scores are formed transposed, S^T = K Q^T (16 keys x 16 query columns per
// 16x16x32 MFMA), so a lane owns one query column and keys 4*(lane/16)..+3 of
// each 16-key block: the online-softmax rescale is lane-local and only the
// running maximum needs two cross-lane exchanges per step. The PV product is
// also transposed, O^T += V^T P^T: the probabilities are reused from the score
// registers (the MFMA k order only has to agree between its two operands) and
// the pool's V blocks, grouped by eight keys and dimension-major inside a
// group, supply V^T fragments as 16-byte reads. A query column is one
// (position, q head) pair; the G = n_q / n_kv heads of a kv head sit in
// adjacent columns so each K/V byte serves all of them.
//
// Two kinds of work share the launch, one per 256-thread workgroup (4 waves;
// two workgroups per CU, so a compute-bound tile and a bandwidth-bound item
// group can run side by side on one CU; one per CU when the launch holds no
// tiles):
//  * chunk tiles: 128 columns (4 waves x 32) of one request and kv head over a
//    key range; 32-key K/V steps (two pool blocks) are copied as stored into
//    a 4-stage LDS ring by global-to-LDS loads and every wave reads them from
//    there (the pool's K layout puts a fragment read's 8 keys of one
//    dimension chunk in one 128-byte line; the second block sits 128 bytes
//    off, so reads do not collide in banks). Compute-bound: 32 MFMAs per wave
//    per step.
//  * wave items: 16 columns (decodes, short chunks) per wave, four per
//    workgroup; each wave streams its K/V straight into registers, the next
//    32-key step loading while the current one is multiplied. HBM-bound.
//    A long item range is cut into four consecutive sub-ranges, one per wave
//    of a workgroup, which combines them in LDS at the end.
// The planner interleaves the two kinds so compute- and bandwidth-bound
// workgroups run side by side. Key ranges longer than one work unit takes
// are divided over several units; a merge kernel combines their partial
// results with the log-sum-exp rule.
#include <algorithm>

#include "hb_device.h"
#include "hb_kernels.h"
#include "hb_plan.h"

namespace hb {
namespace attn_detail {

constexpr float NEG_BIG = -1.0e30f;
constexpr int WSTEP = 32;   // keys per wave-item step = 2 pool blocks
constexpr int WAVES = 4;    // waves per workgroup (one per SIMD; two workgroups per CU)
static_assert(WAVES == kItemsPerUnit && 32 * WAVES == kTileCols, "planner geometry");

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Online softmax of one column over the N raw scores (q.k) a lane holds for
// a key step, in log2 units (sc = log2(e)/sqrt(hd)). The running maximum m
// only moves when the weights 2^(s*sc - m) of some lane add up to more than
// 2^RESCALE_SLACK (so whenever a score exceeds m by more than the slack);
// below that the weights, at most 2^RESCALE_SLACK, are carried without loss
// by fp32 accumulation and bf16 weights. The result is exact either way (O,
// l and m change together), and the O rescale -- a read-modify-write of
// every accumulator -- is mostly skipped.
constexpr float RESCALE_SLACK = 8.0f;
constexpr float kRescaleSum = 256.0f;  // 2^RESCALE_SLACK

// Common case: the weights against the current running maximum and their
// sum. No step maximum is formed: the weights are non-negative, so a lane's
// sum bounds each of its weights, and the step is accepted (wave-uniform)
// when every lane's sum is at most 2^RESCALE_SLACK. Otherwise (some weight
// may exceed the slack; rarely, several large ones only add up past it) the
// caller runs softmax_rescale, which recomputes them exactly.
template <int N>
__device__ __forceinline__ bool softmax_fast(const float (&sv)[N], float sc, float m, float& ps, float (&p)[N]) {
  ps = 0.f;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    p[i] = __builtin_amdgcn_exp2f(fmaf(sv[i], sc, -m));  // 0 for masked keys; no denormal results needed
    ps += p[i];
  }
  return __any(!(ps <= kRescaleSum));
}

// Rare case: the column's exact step maximum (across the four lanes that
// hold its keys) moves the running maximum; l is scaled by alpha (the caller
// scales O) and the weights are recomputed.
template <int N>
__device__ __forceinline__ void softmax_rescale(const float (&sv)[N], float sc, float& m, float& l, float& alpha,
                                                float& ps, float (&p)[N]) {
  float mx = sv[0];
#pragma unroll
  for (int i = 1; i < N; ++i) mx = fmaxf(mx, sv[i]);
  const float ms = rows_max(mx) * sc;  // -inf when every key of the step is masked
  const float mn = fmaxf(m, ms);
  alpha = __builtin_amdgcn_exp2f(m - mn);  // 0 from the initial -1e30
  l *= alpha;
  m = mn;
  ps = 0.f;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    p[i] = __builtin_amdgcn_exp2f(fmaf(sv[i], sc, -m));
    ps += p[i];
  }
}

// P^T operand of keys 32kk..32kk+31: slots 0..3 from block 2kk, 4..7 from 2kk+1.
template <int N>
__device__ __forceinline__ bf16x8 p_operand(const float (&p)[N], int kk) {
  const int a = 8 * kk;
  u32x4 w = {pack_bf16x2(p[a], p[a + 1]), pack_bf16x2(p[a + 2], p[a + 3]), pack_bf16x2(p[a + 4], p[a + 5]),
             pack_bf16x2(p[a + 6], p[a + 7])};
  return as_bf16x8(w);
}

// Write the result of one column: normalised bf16 output, or fp32 partials.
template <int HD>
__device__ __forceinline__ void store_column(const AttnArgs& a, const AttnItem& it, int c, const f32x4 (&o)[HD / 16],
                                             float m, float l, int grp) {
  const int G = a.nq / a.nkv;
  const int pi = c / G;
  if (pi >= it.npos) return;  // column past the item's last position
  if (it.part < 0) {
    const int h = it.kv_head * G + (c - pi * G);
    const float inv = 1.0f / l;
    uint16_t* orow = a.o + (size_t)(it.tok0 + pi) * a.nq * HD + h * HD + 4 * grp;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      u32x2 w = {pack_bf16x2(o[dt][0] * inv, o[dt][1] * inv), pack_bf16x2(o[dt][2] * inv, o[dt][3] * inv)};
      st8(orow + 16 * dt, w);
    }
  } else {
    const size_t slot = (size_t)it.part + c;
    float* po = a.part_o + slot * HD + 4 * grp;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      u32x4 w = {__float_as_uint(o[dt][0]), __float_as_uint(o[dt][1]), __float_as_uint(o[dt][2]),
                 __float_as_uint(o[dt][3])};
      st16(po + 16 * dt, w);
    }
    if (grp == 0) {
      a.part_ml[slot * 2 + 0] = m;
      a.part_ml[slot * 2 + 1] = l;
    }
  }
}

// ---------------------------------------------------------------------------
// wave item: 16 columns, K/V streamed into registers, one step ahead
//
// Key order of a 32-key step (both pool blocks): score MFMA b takes, in its
// row r, key 8 (r / 4) + 4 b + r % 4, so the lanes of row group g end up with
// the scores of keys 8 g .. 8 g + 7 -- the eight keys one lane feeds to the
// PV MFMA, stored together (16 bytes) in the V pool.
// ---------------------------------------------------------------------------
template <int HD>
struct WaveStep {
  u32x4 k[2][HD / 32];  // per score MFMA: the lane's key row, 8 dims of each 32-dim chunk
  u32x4 v[HD / 16];     // per 16-dim tile: keys 8 grp..+7 of one dim
};

template <int HD>
__device__ __forceinline__ void wave_load(WaveStep<HD>& st, const AttnArgs& a, int id0, int id1, int g, int col,
                                          int grp) {
  const size_t blk_stride = (size_t)a.nkv * 16 * HD;
  const size_t head_off = (size_t)g * 16 * HD;
  // K: this lane's key (8 (col / 4) + 4 b + col % 4 of the step) is slot
  // col % 8 of slot group b in block col / 8, and its dimensions 32 kc +
  // 8 grp .. + 7 are chunk 4 kc + grp: a load's lanes cover whole lines
  const uint16_t* K = a.k_pool + (size_t)((col >> 3) ? id1 : id0) * blk_stride + head_off + (8 * grp + (col & 7)) * 8;
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int kc = 0; kc < HD / 32; ++kc) st.k[b][kc] = ld16_stream(K + (b * (HD / 8) + 4 * kc) * 64);
  // V: keys 8 grp..+7 are half grp % 2 of block grp / 2
  const uint16_t* V = a.v_pool + (size_t)((grp >> 1) ? id1 : id0) * blk_stride + head_off +
                      ((grp & 1) * HD + col) * 8;
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) st.v[dt] = ld16_stream(V + 16 * dt * 8);
}

// Lane mask of the eight keys j0 + 8 grp .. +7 of a V^T operand: keys at or
// past kv_end may be unwritten slots holding non-finite bits (0 * NaN would
// poison the sum), so their bf16 lanes are cleared.
__device__ __forceinline__ u32x4 v_key_mask(int j0, int kv_end, int grp) {
  u32x4 vm;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const int k = j0 + 8 * grp + 2 * w;
    vm[w] = (k < kv_end ? 0xFFFFu : 0u) | (k + 1 < kv_end ? 0xFFFF0000u : 0u);
  }
  return vm;
}

template <int HD>
__device__ __forceinline__ void wave_compute(const WaveStep<HD>& st, int j0, const AttnItem& it, int pos, int grp,
                                             float sc, const bf16x8 (&qf)[HD / 32], f32x4 (&o)[HD / 16], float& m,
                                             float& l) {
  f32x4 s[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    s[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < HD / 32; ++kc) s[b] = mfma16x16x32(as_bf16x8(st.k[b][kc]), qf[kc], s[b]);
  }
  float sv[8], p[8];
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) sv[4 * b + i] = s[b][i];
  if (j0 + WSTEP > it.kv_end || j0 + WSTEP > it.pos0) {  // causal / tail masking (wave-uniform)
    const int lim = min(pos, it.kv_end - 1);
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (j0 + 8 * grp + 4 * b + i > lim) sv[4 * b + i] = -INFINITY;
  }
  float ps;
  bf16x8 pf;
  if (softmax_fast<8>(sv, sc, m, ps, p)) {
    float alpha;
    softmax_rescale<8>(sv, sc, m, l, alpha, ps, p);
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) o[dt] *= alpha;
  }
  l += ps;
  pf = p_operand(p, 0);
  if (j0 + WSTEP > it.kv_end) {  // tail step (wave-uniform)
    const u32x4 vm = v_key_mask(j0, it.kv_end, grp);
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) o[dt] = mfma16x16x32(as_bf16x8(st.v[dt] & vm), pf, o[dt]);
  } else {
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) o[dt] = mfma16x16x32(as_bf16x8(st.v[dt]), pf, o[dt]);
  }
}

// One wave item's 16 columns over its key range: the unnormalised O^T, the
// running maximum m and the weight sum l of the lane's column (l summed over
// the column's four lanes; m is the same on all four).
template <int HD>
__device__ __forceinline__ void wave_run(const AttnArgs& a, const AttnItem& it, int lane, f32x4 (&o)[HD / 16],
                                         float& m, float& l) {
  const int G = a.nq / a.nkv;
  const int col = lane & 15, grp = lane >> 4;
  const int pi = col / G;
  const bool valid = pi < it.npos;
  const int pos = it.pos0 + pi;
  const int g = it.kv_head, h = g * G + (col - pi * G);
  bf16x8 qf[HD / 32];
#pragma unroll
  for (int kc = 0; kc < HD / 32; ++kc) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (valid) v = ld16(a.q + (size_t)(it.tok0 + pi) * a.nq * HD + h * HD + 32 * kc + 8 * grp);
    qf[kc] = as_bf16x8(v);
  }
  const int32_t* btab = a.bt + const_load(a.req_bt + it.req);
  const int kb_last = (it.kv_end - 1) >> 4;
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  m = NEG_BIG;
  l = 0.f;
  const int nsteps = (it.kv_end - it.kv_begin + WSTEP - 1) / WSTEP;
  // the table is padded with copies of its last id (kBtPad), so the two ids
  // of a step are one 8-byte read; steps past the end re-read the last block
  typedef int32_t i32x2 __attribute__((ext_vector_type(2)));
  auto ids_of = [&](int s) {
    return const_load(reinterpret_cast<const i32x2*>(btab + min((it.kv_begin >> 4) + 2 * s, kb_last)));
  };
  // Block ids are fetched one step before the loads that use them. Loads in
  // the steady-state loop are unconditional so the compiler can wait for one
  // step's registers while the next step's loads stay in flight; the last
  // one or two steps are peeled off.
  WaveStep<HD> A, B;
  i32x2 ids = ids_of(0);
  wave_load(A, a, ids[0], ids[1], g, col, grp);
  ids = ids_of(1);
  int s = 0;
  for (; s + 2 < nsteps; s += 2) {
    wave_load(B, a, ids[0], ids[1], g, col, grp);
    ids = ids_of(s + 2);
    __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of the compute
    wave_compute(A, it.kv_begin + WSTEP * s, it, pos, grp, a.scale_log2, qf, o, m, l);
    __builtin_amdgcn_sched_barrier(0);
    wave_load(A, a, ids[0], ids[1], g, col, grp);
    ids = ids_of(s + 3);
    __builtin_amdgcn_sched_barrier(0);
    wave_compute(B, it.kv_begin + WSTEP * (s + 1), it, pos, grp, a.scale_log2, qf, o, m, l);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (s + 1 < nsteps) {
    wave_load(B, a, ids[0], ids[1], g, col, grp);
    wave_compute(A, it.kv_begin + WSTEP * s, it, pos, grp, a.scale_log2, qf, o, m, l);
    wave_compute(B, it.kv_begin + WSTEP * (s + 1), it, pos, grp, a.scale_log2, qf, o, m, l);
  } else {
    wave_compute(A, it.kv_begin + WSTEP * s, it, pos, grp, a.scale_log2, qf, o, m, l);
  }
  l = rows_sum(l);
}

template <int HD>
__device__ __forceinline__ void wave_item(const AttnArgs& a, const AttnItem& it, int lane) {
  f32x4 o[HD / 16];
  float m, l;
  wave_run<HD>(a, it, lane, o, m, l);
  store_column<HD>(a, it, lane & 15, o, m, l, lane >> 4);
}

// A merged unit: its four items are consecutive key ranges of one (request,
// kv head, positions), one per wave (an empty range contributes nothing).
// The waves' results are combined in LDS with the log-sum-exp rule: with
// M = max_w m_w, O = sum_w O_w 2^(m_w - M) and l = sum_w l_w 2^(m_w - M).
// Wave w then finishes dimension tiles w DT/4 .. (w + 1) DT/4 - 1 of every
// column and writes them, normalised, or as a partial result (O, M, l).
template <int HD>
__device__ __forceinline__ void merged_unit(const AttnArgs& a, int v, uint8_t* smem) {
  constexpr int DT = HD / 16, PER = DT / WAVES;
  static_assert(PER * WAVES == DT, "dimension tiles per wave");
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int col = lane & 15, grp = lane >> 4;
  const AttnItem it = const_load(reinterpret_cast<const AttnItem*>(a.items) + WAVES * v + wave);
  f32x4 o[DT];
  float m = NEG_BIG, l = 0.f;
  if (it.kv_begin < it.kv_end) {
    wave_run<HD>(a, it, lane, o, m, l);
  } else {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  float* ml = reinterpret_cast<float*>(smem);                       // [wave][column] (m, l)
  f32x4* os = reinterpret_cast<f32x4*>(smem + WAVES * 16 * 2 * 4);  // [wave][dt][lane]
  if (grp == 0) {
    ml[(wave * 16 + col) * 2 + 0] = m;
    ml[(wave * 16 + col) * 2 + 1] = l;
  }
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) os[(wave * DT + dt) * 64 + lane] = o[dt];
  __syncthreads();
  float mw[WAVES], M = NEG_BIG;
#pragma unroll
  for (int w = 0; w < WAVES; ++w) {
    mw[w] = ml[(w * 16 + col) * 2];
    M = fmaxf(M, mw[w]);
  }
  float L = 0.f;
#pragma unroll
  for (int w = 0; w < WAVES; ++w) {
    mw[w] = exp2f(mw[w] - M);  // 0 for ranges with no key of this column
    L += ml[(w * 16 + col) * 2 + 1] * mw[w];
  }
  f32x4 r[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    r[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < WAVES; ++w) r[i] += os[(w * DT + wave * PER + i) * 64 + lane] * mw[w];
  }
  const int G = a.nq / a.nkv;
  const int pi = col / G;
  if (pi >= it.npos) return;  // column past the unit's last position
  if (it.part < 0) {
    const int h = it.kv_head * G + (col - pi * G);
    const float inv = 1.0f / L;
    uint16_t* orow = a.o + (size_t)(it.tok0 + pi) * a.nq * HD + h * HD + 4 * grp;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int dt = wave * PER + i;
      u32x2 w = {pack_bf16x2(r[i][0] * inv, r[i][1] * inv), pack_bf16x2(r[i][2] * inv, r[i][3] * inv)};
      st8(orow + 16 * dt, w);
    }
  } else {
    const size_t slot = (size_t)it.part + col;
    float* po = a.part_o + slot * HD + 4 * grp;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int dt = wave * PER + i;
      u32x4 w = {__float_as_uint(r[i][0]), __float_as_uint(r[i][1]), __float_as_uint(r[i][2]),
                 __float_as_uint(r[i][3])};
      st16(po + 16 * dt, w);
    }
    if (grp == 0 && wave == 0) {
      a.part_ml[slot * 2 + 0] = M;
      a.part_ml[slot * 2 + 1] = L;
    }
  }
}

// ---------------------------------------------------------------------------
// chunk tile: 256 columns, K/V staged in an LDS ring by the DMA path
// ---------------------------------------------------------------------------
constexpr int TSTEP = 32;    // keys per tile step = 2 pool blocks
constexpr int TSTAGES = 4;   // LDS ring depth of the tile path

template <int HD>
struct TileGeom {
  static constexpr int BLK = 16 * HD * 2;        // bytes of one K (or V) block of one head
  static constexpr int LOADS = BLK / 1024;       // 1-KB loads per block
  // Blocks are copied as stored: K [group][chunk][8 keys][8 dims], V
  // [half][dim][8 keys]. The second K block sits 128 bytes further on, so
  // the two blocks' halves of a fragment read fall in different banks.
  static constexpr int KPAD = 128;
  static constexpr int STAGE = 4 * BLK + KPAD;  // K of 2 blocks, then V of 2 blocks
  static constexpr __host__ __device__ int off(int b) { return b * BLK + (b > 0 ? KPAD : 0); }
};

// One step is four blocks in the stage: K of the two pool blocks, then their
// V. Wave b copies stage block b: the K (b = 0, 1) or V (b = 2, 3) of pool
// block b & 1.
template <int HD>
__device__ __forceinline__ void tile_issue(uint8_t* stage, const AttnArgs& a, int id, int g, int wave, int lane) {
  using TG = TileGeom<HD>;
  typedef __attribute__((address_space(3))) void* lds_ptr;
  const int b = wave;
  // a buffer resource over this wave's block (K or V of pool block b & 1):
  // the loads then carry only a lane offset and a scalar offset
  const uint16_t* blk = (b < 2 ? a.k_pool : a.v_pool) + ((size_t)id * a.nkv + g) * 16 * HD;
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(blk), (short)0, TG::BLK, 0x00020000);
  uint8_t* dst = stage + TG::off(b);
#pragma unroll
  for (int i = 0; i < TG::LOADS; ++i) {
    uint8_t* d = dst + i * 1024;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr)d, 16, (uint32_t)(lane * 16), (uint32_t)(i * 1024), 0, 0);
  }
}

// Fragments of one step from a stage. K: for score MFMA b, the lane's key
// (slot col % 8 of slot group b in block col / 8) and dimension chunk
// 4 kc + grp: k_lane = block offset + (8 grp + col % 8) * 16, plus
// (b hd/8 + 4 kc) * 128. V: keys 8 grp..+7 of dims 16 dt + col
// (v_lane = grp * HD * 16 + col * 16).
template <int HD>
__device__ __forceinline__ void tile_read_k(bf16x8 (&kf)[2][HD / 32], const uint8_t* st, int k_lane) {
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int kc = 0; kc < HD / 32; ++kc)
      kf[b][kc] = as_bf16x8(*reinterpret_cast<const u32x4*>(st + k_lane + (b * (HD / 8) + 4 * kc) * 128));
}

template <int HD>
__device__ __forceinline__ void tile_read_v(u32x4 (&vf)[HD / 16], const uint8_t* st, int v_lane) {
  using TG = TileGeom<HD>;
  const uint8_t* vs = st + TG::off(2) + v_lane;
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) vf[dt] = *reinterpret_cast<const u32x4*>(vs + dt * 256);
}

// MASKED: the V lanes of keys past kv_end are cleared.
template <int HD, bool MASKED>
__device__ __forceinline__ void tile_mask_v(u32x4 (&vf)[HD / 16], int j0, int kv_end, int grp) {
  if (!MASKED) return;
  const u32x4 vm = v_key_mask(j0, kv_end, grp);
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) vf[dt] &= vm;
}

template <int HD, int CT>
__device__ __forceinline__ void tile_scores(f32x4 (&sc)[CT][2], const bf16x8 (&kf)[2][HD / 32],
                                            const bf16x8 (&qf)[CT][HD / 32]) {
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      sc[ct][b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < HD / 32; ++kc) sc[ct][b] = mfma16x16x32(kf[b][kc], qf[ct][kc], sc[ct][b]);
    }
}

// Online softmax of one step for the wave's CT column tiles: the common
// case (branch-free, so the score MFMAs can be scheduled across it) gives
// the weights pf and their sums ps against the running maxima; it returns
// whether tile_rescale must run. MASKED: keys past a column's position or
// past kv_end get no weight.
template <int HD, int CT, bool MASKED>
__device__ __forceinline__ bool tile_softmax(const f32x4 (&sc)[CT][2], float (&sv)[CT][8], float (&p)[CT][8],
                                             float (&ps)[CT], const float (&m)[CT], const int (&pos)[CT], int j0,
                                             int kv_end, int grp, float scale) {
  bool rescale = false;
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) sv[ct][4 * b + i] = sc[ct][b][i];
    if (MASKED) {
      const int lim = min(pos[ct], kv_end - 1);
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (j0 + 8 * grp + 4 * b + i > lim) sv[ct][4 * b + i] = -INFINITY;
    }
    rescale |= softmax_fast<8>(sv[ct], scale, m[ct], ps[ct], p[ct]);
  }
  return rescale;
}

template <int HD, int CT>
__device__ __forceinline__ void tile_pv(f32x4 (&o)[CT][HD / 16], const u32x4 (&vf)[HD / 16], const bf16x8 (&pf)[CT]) {
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) o[ct][dt] = mfma16x16x32(as_bf16x8(vf[dt]), pf[ct], o[ct][dt]);
}

// One key step of a tile. The scores of this step (sc_cur) were formed one
// step earlier; while their softmax runs on the vector ALUs, the next step's
// scores go to the matrix cores (sc_next), so the two overlap within the wave.
template <int HD, int CT, bool MASKED, bool LAST>
__device__ __forceinline__ void tile_step(const AttnArgs& a, const AttnItem& it, uint8_t* smem, int kt, int nsteps,
                                          const int32_t* btab, int kb0, int kb_last, int& next_id, int wave,
                                          int lane, int k_lane, int v_lane, const bf16x8 (&qf)[CT][HD / 32],
                                          const int (&pos)[CT], f32x4 (&o)[CT][HD / 16], float (&m)[CT],
                                          float (&l)[CT], f32x4 (&sc_cur)[CT][2], f32x4 (&sc_next)[CT][2]) {
  using TG = TileGeom<HD>;
  const int grp = lane >> 4, col = lane & 15;
  // V fragments of this step (their LDS latency hides under the score MFMAs)
  const int j0 = it.kv_begin + TSTEP * kt;
  u32x4 vf[HD / 16];
  tile_read_v<HD>(vf, smem + (kt % TSTAGES) * TG::STAGE, v_lane);
  if (!LAST) {
    // step kt + 1 complete (the one issued after it may stay in flight); the
    // ring slot of step kt - 1 is free for step kt + TSTAGES - 1
    if (kt + 2 < nsteps) wait_vmcnt<TG::LOADS>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    if (kt + TSTAGES - 1 < nsteps) {
      tile_issue<HD>(smem + ((kt + TSTAGES - 1) % TSTAGES) * TG::STAGE, a, next_id, it.kv_head, wave, lane);
      if (kt + TSTAGES < nsteps) next_id = const_load(btab + min(kb0 + 2 * (kt + TSTAGES) + (wave & 1), kb_last));
    }
    bf16x8 kf[2][HD / 32];
    tile_read_k<HD>(kf, smem + ((kt + 1) % TSTAGES) * TG::STAGE, k_lane);
    tile_scores<HD, CT>(sc_next, kf, qf);
  }
  float sv[CT][8], p[CT][8], ps[CT];
  const bool rescale = tile_softmax<HD, CT, MASKED>(sc_cur, sv, p, ps, m, pos, j0, it.kv_end, grp, a.scale_log2);
  bf16x8 pf[CT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) pf[ct] = p_operand(p[ct], 0);
  // keep the weights' computation here, under the score MFMAs, rather than
  // letting it sink past the rescale branch into the PV block
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) {
    u32x4 w = __builtin_bit_cast(u32x4, pf[ct]);
    asm volatile("" : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3]));
    pf[ct] = __builtin_bit_cast(bf16x8, w);
  }
  __builtin_amdgcn_sched_barrier(0);
  if (rescale) {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      float alpha;
      softmax_rescale<8>(sv[ct], a.scale_log2, m[ct], l[ct], alpha, ps[ct], p[ct]);
      pf[ct] = p_operand(p[ct], 0);
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) o[ct][dt] *= alpha;
    }
  }
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) l[ct] += ps[ct];
  tile_mask_v<HD, MASKED>(vf, j0, it.kv_end, grp);
  tile_pv<HD, CT>(o, vf, pf);
}

template <int HD>
__device__ __forceinline__ void tile_unit(const AttnArgs& a, const AttnItem& it, uint8_t* smem) {
  using TG = TileGeom<HD>;
  constexpr int KC = HD / 32, DT = HD / 16;
  constexpr int CT = 2;  // 16-column tiles per wave (4 waves x 32 columns)
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int G = a.nq / a.nkv;
  const int col = lane & 15, grp = lane >> 4;
  const int g = it.kv_head;
  bf16x8 qf[CT][KC];
  int pos[CT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) {
    const int c = 32 * wave + 16 * ct + col;
    const int pi = c / G;
    const bool valid = pi < it.npos;
    pos[ct] = it.pos0 + pi;
    const int h = g * G + (c - pi * G);
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (valid) v = ld16(a.q + (size_t)(it.tok0 + pi) * a.nq * HD + h * HD + 32 * kc + 8 * grp);
      qf[ct][kc] = as_bf16x8(v);
    }
  }
  const int32_t* btab = a.bt + const_load(a.req_bt + it.req);
  const int kb_last = (it.kv_end - 1) >> 4;
  const int kb0 = it.kv_begin >> 4;
  const int nsteps = (it.kv_end - it.kv_begin + TSTEP - 1) / TSTEP;
  // steps whose keys all lie below the tile's first position and kv_end need no mask
  const int full = min(nsteps, max(0, (min(it.kv_end, it.pos0) - it.kv_begin) / TSTEP));

  f32x4 o[CT][DT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[ct][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m[CT], l[CT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) { m[ct] = NEG_BIG; l[ct] = 0.f; }

  const int k_lane = TG::off(col >> 3) + (8 * grp + (col & 7)) * 16;
  const int v_lane = grp * HD * 16 + col * 16;
  // prologue: steps 0..TSTAGES-2 in flight, scores of step 0
  int next_id = const_load(btab + min(kb0 + (wave & 1), kb_last));
#pragma unroll
  for (int s0 = 0; s0 < TSTAGES - 1; ++s0) {
    if (s0 < nsteps) tile_issue<HD>(smem + s0 * TG::STAGE, a, next_id, g, wave, lane);
    if (s0 + 1 < nsteps) next_id = const_load(btab + min(kb0 + 2 * (s0 + 1) + (wave & 1), kb_last));
  }
  if (nsteps >= 3) wait_vmcnt<2 * TG::LOADS>();
  else if (nsteps == 2) wait_vmcnt<TG::LOADS>();
  else wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  f32x4 sa[CT][2], sb[CT][2];
  {
    bf16x8 kf[2][KC];
    tile_read_k<HD>(kf, smem, k_lane);
    tile_scores<HD, CT>(sa, kf, qf);
  }
  // steps alternate the two score buffers; the last step is peeled
  int kt = 0;
  for (; kt + 2 <= full && kt + 2 < nsteps; kt += 2) {
    tile_step<HD, CT, false, false>(a, it, smem, kt, nsteps, btab, kb0, kb_last, next_id, wave, lane, k_lane, v_lane,
                                    qf, pos, o, m, l, sa, sb);
    tile_step<HD, CT, false, false>(a, it, smem, kt + 1, nsteps, btab, kb0, kb_last, next_id, wave, lane, k_lane,
                                    v_lane, qf, pos, o, m, l, sb, sa);
  }
  for (; kt + 2 < nsteps; kt += 2) {
    tile_step<HD, CT, true, false>(a, it, smem, kt, nsteps, btab, kb0, kb_last, next_id, wave, lane, k_lane, v_lane,
                                   qf, pos, o, m, l, sa, sb);
    tile_step<HD, CT, true, false>(a, it, smem, kt + 1, nsteps, btab, kb0, kb_last, next_id, wave, lane, k_lane,
                                   v_lane, qf, pos, o, m, l, sb, sa);
  }
  if (kt + 1 < nsteps) {
    tile_step<HD, CT, true, false>(a, it, smem, kt, nsteps, btab, kb0, kb_last, next_id, wave, lane, k_lane, v_lane,
                                   qf, pos, o, m, l, sa, sb);
    tile_step<HD, CT, true, true>(a, it, smem, kt + 1, nsteps, btab, kb0, kb_last, next_id, wave, lane, k_lane, v_lane,
                                  qf, pos, o, m, l, sb, sa);
  } else {
    tile_step<HD, CT, true, true>(a, it, smem, kt, nsteps, btab, kb0, kb_last, next_id, wave, lane, k_lane, v_lane,
                                  qf, pos, o, m, l, sa, sb);
  }
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) store_column<HD>(a, it, 32 * wave + 16 * ct + col, o[ct], m[ct], rows_sum(l[ct]), grp);
}

template <int HD>
__global__ __launch_bounds__(64 * WAVES, 2) void attn_kernel(AttnArgs a) {
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  const int unit = const_load(a.units + blockIdx.x);
  if (unit >= 0) {
    tile_unit<HD>(a, const_load(reinterpret_cast<const AttnItem*>(a.tiles) + unit), smem);
  } else if ((-unit - 1) & kUnitMerged) {
    merged_unit<HD>(a, (-unit - 1) & ~kUnitMerged, smem);
  } else {
    const int idx = (-unit - 1) * WAVES + wave_id();
    if (idx < a.n_items) {
      const AttnItem it = const_load(reinterpret_cast<const AttnItem*>(a.items) + idx);
      if (it.kv_begin < it.kv_end) wave_item<HD>(a, it, threadIdx.x & 63);
    }
  }
}

// Merge of split work: one workgroup per (merge group, 16 columns), one
// thread per (column, 8 dims), folding the parts in order with the online
// rule: M' = max(M, m_s), acc' = acc 2^(M-M') + O_s 2^(m_s-M'), likewise L
// (several parts per fold, all of their loads issued together).
template <int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  const int mu = const_load(a.merge_units + blockIdx.x);
  const MergeGroup gr = const_load(reinterpret_cast<const MergeGroup*>(a.groups) + (mu >> 4));
  const int G = a.nq / a.nkv;
  constexpr int TPC = HD / 8;  // threads per column
  const int c = (mu & 15) * 16 + threadIdx.x / TPC;
  if (threadIdx.x >= 16 * TPC || c >= gr.npos * G) return;
  const int d = (threadIdx.x % TPC) * 8;
  float M = NEG_BIG, L = 0.f, acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  // parts are folded four at a time so their loads are in flight together
  constexpr int B = 4;
  for (int s0 = 0; s0 < gr.nparts; s0 += B) {
    float ms[B], ls[B];
    u32x4 o0[B], o1[B];
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const int s = min(s0 + j, gr.nparts - 1);
      const size_t slot = (size_t)gr.part0 + (size_t)s * gr.stride + c;
      const u32x2 ml = ld8(a.part_ml + slot * 2);
      ms[j] = (s0 + j < gr.nparts) ? __uint_as_float(ml[0]) : NEG_BIG;
      ls[j] = __uint_as_float(ml[1]);
      o0[j] = ld16(a.part_o + slot * HD + d);
      o1[j] = ld16(a.part_o + slot * HD + d + 4);
    }
    float Mn = M;
#pragma unroll
    for (int j = 0; j < B; ++j) Mn = fmaxf(Mn, ms[j]);
    const float wa = exp2f(M - Mn);
    L *= wa;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] *= wa;
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const float wb = (s0 + j < gr.nparts) ? exp2f(ms[j] - Mn) : 0.f;
      L += ls[j] * wb;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[e] += __uint_as_float(o0[j][e]) * wb;
        acc[4 + e] += __uint_as_float(o1[j][e]) * wb;
      }
    }
    M = Mn;
  }
  const float inv = 1.0f / L;
  const int pi = c / G, h = gr.kv_head * G + (c - pi * G);
  u32x4 w = {pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
             pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv)};
  st16(a.o + (size_t)(gr.tok0 + pi) * a.nq * HD + h * HD + d, w);
}

// A launch without chunk tiles only streams K/V through wave items, and one
// workgroup per CU does that faster than two (64 decodes of 512-4096 keys:
// 109 -> 103 us; larger decode batches 0-1 % faster, none slower): such a
// launch asks for more LDS than half a CU holds, so one workgroup fits per CU.
// With tiles, two workgroups per CU (a tile beside a tile or an item group)
// stay far faster.
constexpr int kItemOnlyLds = 96 * 1024;

template <int HD>
void launch(hipStream_t s, const AttnArgs& a) {
  constexpr int lds = TSTAGES * TileGeom<HD>::STAGE;
  static_assert(2 * lds <= 160 * 1024 && 2 * kItemOnlyLds > 160 * 1024 && kItemOnlyLds <= 160 * 1024, "occupancy");
  static std::atomic<uint64_t> lds_raised{0};
  raise_dynamic_lds(reinterpret_cast<const void*>(&attn_kernel<HD>), kItemOnlyLds, lds_raised);
  attn_kernel<HD><<<a.n_units, 64 * WAVES, a.n_tiles > 0 ? lds : kItemOnlyLds, s>>>(a);
}

}  // namespace attn_detail

void launch_attention(hipStream_t s, const AttnArgs& a) {
  if (a.n_units <= 0) return;
  if (a.hd == 128) attn_detail::launch<128>(s, a);
  else attn_detail::launch<64>(s, a);
}

void launch_attn_merge(hipStream_t s, const AttnArgs& a) {
  if (a.n_merge_units <= 0) return;
  if (a.hd == 128) attn_detail::attn_merge_kernel<128><<<a.n_merge_units, 256, 0, s>>>(a);
  else attn_detail::attn_merge_kernel<64><<<a.n_merge_units, 256, 0, s>>>(a);
}

}  // namespace hb
