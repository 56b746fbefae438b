// Varlen paged attention for a hybrid batch: causal chunk rows over their
// request's cached context and single-token decode rows, in one launch.
//
// Work unit = one wavefront = 16 query columns (P = 16/G positions x the G
// q heads that share one kv head) of one request over a key range. Scores are
// formed transposed, S^T = K Q^T (16 keys x 16 columns per MFMA), so each lane
// owns one column and the keys 4*(lane/16)..+3 of a 16-key block: the online
// softmax rescale is lane-local and only the running maximum needs two
// cross-lane exchanges per 32 keys. The PV product is also formed transposed,
// O^T += V^T P^T, with the pool's dim-major V blocks supplying V^T fragments
// directly and the probabilities reused from the score registers (the MFMA
// k order only has to agree between its two operands). Long key ranges are
// split over several waves; a merge kernel combines their partial results
// with the log-sum-exp rule.
#include "hb_device.h"
#include "hb_kernels.h"
#include "hb_plan.h"

namespace hb {

namespace {
constexpr float NEG_BIG = -1.0e30f;

template <int HD>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  const int lane = threadIdx.x & 63;
  const int item_id = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item_id >= a.n_items) return;
  const AttnItem it = reinterpret_cast<const AttnItem*>(a.items)[item_id];
  const int G = a.nq / a.nkv;
  const int col = lane & 15, grp = lane >> 4;
  const int pi = col / G, hi = col - pi * G;
  const bool valid = pi < it.npos;
  const int tok = it.tok0 + pi, pos = it.pos0 + pi;
  const int g = it.kv_head, h = g * G + hi;
  const int qstride = a.nq * HD;

  bf16x8 qf[HD / 32];
#pragma unroll
  for (int kc = 0; kc < HD / 32; ++kc) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (valid) v = ld16(a.q + (size_t)tok * qstride + h * HD + 32 * kc + 8 * grp);
    qf[kc] = as_bf16x8(v);
  }
  const int32_t* btab = a.bt + a.req_bt[it.req];
  f32x4 o[HD / 16];
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = NEG_BIG, l = 0.f;
  const float sc = a.scale_log2;
  const size_t blk_stride = (size_t)a.nkv * 16 * HD;  // elements per pool block
  const size_t head_off = (size_t)g * 16 * HD;

  for (int j0 = it.kv_begin; j0 < it.kv_end; j0 += 32) {
    const int b0 = btab[j0 >> 4];
    const bool has1 = j0 + 16 < it.kv_end;
    const int b1 = has1 ? btab[(j0 >> 4) + 1] : b0;
    const uint16_t* K0 = a.k_pool + (size_t)b0 * blk_stride + head_off;
    const uint16_t* K1 = a.k_pool + (size_t)b1 * blk_stride + head_off;
    const uint16_t* V0 = a.v_pool + (size_t)b0 * blk_stride + head_off;
    const uint16_t* V1 = a.v_pool + (size_t)b1 * blk_stride + head_off;

    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < HD / 32; ++kc) {
      const bf16x8 ka = as_bf16x8(ld16(K0 + col * HD + 32 * kc + 8 * grp));
      const bf16x8 kb = as_bf16x8(ld16(K1 + col * HD + 32 * kc + 8 * grp));
      s0 = mfma16x16x32(ka, qf[kc], s0);
      s1 = mfma16x16x32(kb, qf[kc], s1);
    }
    // s0[i]: key j0 + 4 grp + i, s1[i]: key j0 + 16 + 4 grp + i, for column `col`
    float sv[8];
    const int kbase = j0 + 4 * grp;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k0i = kbase + i, k1i = kbase + 16 + i;
      sv[i] = (k0i <= pos && k0i < it.kv_end) ? s0[i] * sc : -INFINITY;
      sv[4 + i] = (k1i <= pos && k1i < it.kv_end) ? s1[i] * sc : -INFINITY;
    }
    float mx = sv[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mx = fmaxf(mx, sv[i]);
    mx = wave_max_xor(mx, 16);
    mx = wave_max_xor(mx, 32);
    const float mn = fmaxf(m, mx);
    const float alpha = exp2f(m - mn);
    float pv[8], ps = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      pv[i] = exp2f(sv[i] - mn);
      ps += pv[i];
    }
    l = l * alpha + ps;
    m = mn;
    u32x4 pw = {pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]), pack_bf16x2(pv[4], pv[5]),
                pack_bf16x2(pv[6], pv[7])};
    const bf16x8 pf = as_bf16x8(pw);
    // keys at or past kv_end may be unwritten slots: their V must not reach the MFMA
    const bool tail = j0 + 32 > it.kv_end;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      const int d = 16 * dt + col;
      u32x2 va = ld8(V0 + d * 16 + 4 * grp);
      u32x2 vb = ld8(V1 + d * 16 + 4 * grp);
      if (tail) {
#pragma unroll
        for (int i = 0; i < 4; i += 2) {
          const int k0i = kbase + i, k1i = kbase + 16 + i;
          uint32_t ma = (k0i < it.kv_end ? 0xFFFFu : 0u) | (k0i + 1 < it.kv_end ? 0xFFFF0000u : 0u);
          uint32_t mb = (k1i < it.kv_end ? 0xFFFFu : 0u) | (k1i + 1 < it.kv_end ? 0xFFFF0000u : 0u);
          va[i >> 1] &= ma;
          vb[i >> 1] &= mb;
        }
      }
      u32x4 vw = {va[0], va[1], vb[0], vb[1]};
      o[dt] *= alpha;
      o[dt] = mfma16x16x32(as_bf16x8(vw), pf, o[dt]);
    }
  }
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (it.part < 0) {
    if (!valid) return;
    const float inv = 1.0f / l;
    uint16_t* orow = a.o + (size_t)tok * qstride + h * HD + 4 * grp;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      u32x2 w = {pack_bf16x2(o[dt][0] * inv, o[dt][1] * inv), pack_bf16x2(o[dt][2] * inv, o[dt][3] * inv)};
      st8(orow + 16 * dt, w);
    }
  } else {
    float* po = a.part_o + ((size_t)it.part * 16 + col) * HD + 4 * grp;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      u32x4 w = {__float_as_uint(o[dt][0]), __float_as_uint(o[dt][1]), __float_as_uint(o[dt][2]),
                 __float_as_uint(o[dt][3])};
      st16(po + 16 * dt, w);
    }
    if (grp == 0) {
      a.part_ml[((size_t)it.part * 16 + col) * 2 + 0] = m;
      a.part_ml[((size_t)it.part * 16 + col) * 2 + 1] = l;
    }
  }
}

// One workgroup per split tile: o = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s.
template <int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  const MergeGroup gr = reinterpret_cast<const MergeGroup*>(a.groups)[blockIdx.x];
  const int G = a.nq / a.nkv;
  const int ncol = gr.npos * G;
  const int qstride = a.nq * HD;
  for (int idx = threadIdx.x; idx < ncol * (HD / 4); idx += 256) {
    const int c = idx / (HD / 4), d = (idx - c * (HD / 4)) * 4;
    float M = NEG_BIG;
    for (int s = 0; s < gr.nparts; ++s) M = fmaxf(M, a.part_ml[((size_t)(gr.part0 + s) * 16 + c) * 2]);
    float L = 0.f, acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < gr.nparts; ++s) {
      const size_t pc = (size_t)(gr.part0 + s) * 16 + c;
      const float w = exp2f(a.part_ml[pc * 2] - M);
      L += w * a.part_ml[pc * 2 + 1];
      const u32x4 v = ld16(a.part_o + pc * HD + d);
      for (int j = 0; j < 4; ++j) acc[j] += w * __uint_as_float(v[j]);
    }
    const float inv = 1.0f / L;
    const int pi = c / G, h = gr.kv_head * G + (c - pi * G);
    u32x2 w = {pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv)};
    st8(a.o + (size_t)(gr.tok0 + pi) * qstride + h * HD + d, w);
  }
}
}  // namespace

void launch_attention(hipStream_t s, const AttnArgs& a) {
  if (a.n_items <= 0) return;
  const int grid = (a.n_items + 3) / 4;
  if (a.hd == 128) attn_kernel<128><<<grid, 256, 0, s>>>(a);
  else attn_kernel<64><<<grid, 256, 0, s>>>(a);
}

void launch_attn_merge(hipStream_t s, const AttnArgs& a) {
  if (a.n_groups <= 0) return;
  if (a.hd == 128) attn_merge_kernel<128><<<a.n_groups, 256, 0, s>>>(a);
  else attn_merge_kernel<64><<<a.n_groups, 256, 0, s>>>(a);
}

}  // namespace hb
