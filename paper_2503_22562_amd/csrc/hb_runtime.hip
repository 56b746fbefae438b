// Host runtime behind the C ABI: layer object, workspace, metadata staging,
// the launch sequence of one iteration, per-kernel timing and the latency
// profiler.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include <hip/hip_runtime.h>

#include "hb.h"
#include "hb_kernels.h"
#include "hb_plan.h"
#include "hb_runtime.h"

using namespace hb;

#define HB_HIP(call)                                                                        \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess) return fail(HB_ERR_HIP, "%s failed: %s", #call, hipGetErrorString(e_)); \
  } while (0)

// Scratch of the allocation-free entry point (hb_run_iteration_noalloc):
// metadata, split-K partials and attention split partials of one iteration.
// Every GPU the library runs on holds its own copy for the life of the
// process. In host code `scratch` names a host-side stand-in, never the
// device memory: its device address comes from hipGetSymbolAddress, once per
// device (scratch_address below), and only that address is passed on.
constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {
constexpr int kStages = 4;
// Pinned host staging of the allocation-free entry point's metadata (int32).
constexpr size_t kNoAllocMetaInts = (size_t)1 << 18;
constexpr int kMaxDevices = 64;
constexpr double kPeakHbm = 8.0e12;      // MI355X HBM3E, bytes/s
constexpr double kPeakBf16 = 2.5e15;     // MI355X dense bf16 MFMA, flop/s

// One slot of the metadata ring: pinned host staging and its device copy.
// The upload runs on the layer's copy stream, so it overlaps the previous
// iteration's kernels; the layer's stream waits for it (copied), and the
// next upload into the slot waits for the kernels that read it (consumed).
struct Stage {
  int32_t* host = nullptr;  // pinned
  size_t cap = 0;           // int32 elements
  int32_t* dev = nullptr;
  size_t dev_cap = 0;
  hipEvent_t copied = nullptr, consumed = nullptr;
  bool pending = false;     // copied / consumed recorded, not yet waited on by the host
};

struct TimedLaunch {
  hipEvent_t start, stop;
  int kernel;
};
}  // namespace

struct hb_layer {
  Dims d;
  hb_layer_weights w{};
  hb_kv_pool pool{};
  hipStream_t stream = nullptr;
  int device = 0, cu_count = 0;
  int gemm_tile = -1;   // HB_GEMM_TILE at creation: force one GEMM tile shape (testing)
  int gemm_ksplit = 0;  // HB_GEMM_KSPLIT at creation: force one K split (testing)
  PlanOptions plan_opt;  // HB_ATTN_SPLIT_TILE / HB_ATTN_SPLIT_ITEM at creation (tuning, testing)
  // workspace
  uint16_t *xn = nullptr, *q_rot = nullptr, *attn = nullptr, *mlp = nullptr;
  float* rope_cs = nullptr;    // [max_T][hd]: per-token cos | sin (RoPE)
  int32_t* tok_slot = nullptr; // [max_T]: pool block * 16 + slot of each new token
  float* h2 = nullptr;
  double* inv_freq = nullptr;
  float *part_o = nullptr, *part_ml = nullptr;
  int part_cap = 0;
  hipStream_t copy_stream = nullptr;  // metadata uploads
  float* splitk = nullptr;  // split-K partial sums
  size_t splitk_cap = 0;    // floats
  Stage stage[kStages];
  int stage_next = 0;
  SlotMarks marks;
  Plan plan;
  int last_T = 0;
  GemmPlan last_plans[HB_GEMM_COUNT] = {};  // of the most recent iteration
  // allocation-free entry point: the device's scratch, pinned metadata
  // staging and the event guarding its reuse
  uint8_t* scratch = nullptr;
  int32_t* na_host = nullptr;
  // device bytes the layer holds, and the most it may hold (HB_DEVICE_ALLOC_LIMIT
  // at creation, testing: makes the out-of-memory paths reachable on demand)
  size_t dev_bytes = 0, dev_limit = SIZE_MAX;
  hipEvent_t na_copied = nullptr;
  bool na_pending = false;
  // timing
  uint32_t timing_mask = 0;  // bit k: bracket kernel k with events
  std::vector<hipEvent_t> ev_free;
  std::vector<TimedLaunch> timed;
  double tot_ms[HB_K_COUNT] = {};
  int64_t launches[HB_K_COUNT] = {};
};

namespace {

// Device address of `scratch` on device `dev`, which must be current: looked
// up once per device and kept.
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

hb_status scratch_address(int dev, uint8_t** out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(HB_ERR_UNSUPPORTED, "device %d beyond %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return fail(HB_ERR_HIP, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(e));
    g_scratch_dev[dev] = p;
  }
  *out = static_cast<uint8_t*>(g_scratch_dev[dev]);
  return HB_OK;
}

// hipMalloc for the layer's own buffers, within its device-memory limit.
bool dev_alloc(hb_layer* L, void** p, size_t bytes) {
  *p = nullptr;
  if (bytes > L->dev_limit - std::min(L->dev_limit, L->dev_bytes)) return false;
  if (hipMalloc(p, bytes) != hipSuccess) {
    *p = nullptr;
    return false;
  }
  L->dev_bytes += bytes;
  return true;
}

void dev_free(hb_layer* L, void* p, size_t bytes) {
  if (!p) return;
  (void)hipFree(p);
  L->dev_bytes -= std::min(L->dev_bytes, bytes);
}

hb_status ensure_splitk(hb_layer* L, size_t floats) {
  if (floats <= L->splitk_cap) return HB_OK;
  HB_HIP(hipStreamSynchronize(L->stream));
  dev_free(L, L->splitk, L->splitk_cap * sizeof(float));
  L->splitk = nullptr;
  L->splitk_cap = 0;
  if (!dev_alloc(L, (void**)&L->splitk, floats * sizeof(float)))
    return fail(HB_ERR_OOM, "split-K workspace of %zu B", floats * 4);
  L->splitk_cap = floats;
  return HB_OK;
}

// Partial-result column slots of split attention work.
hb_status ensure_parts(hb_layer* L, int n) {
  if (n <= L->part_cap) return HB_OK;
  int cap = std::max(n, L->part_cap * 2);
  HB_HIP(hipStreamSynchronize(L->stream));
  dev_free(L, L->part_o, (size_t)L->part_cap * L->d.hd * sizeof(float));
  dev_free(L, L->part_ml, (size_t)L->part_cap * 2 * sizeof(float));
  L->part_o = L->part_ml = nullptr;
  L->part_cap = 0;
  if (!dev_alloc(L, (void**)&L->part_o, (size_t)cap * L->d.hd * sizeof(float)) ||
      !dev_alloc(L, (void**)&L->part_ml, (size_t)cap * 2 * sizeof(float)))
    return fail(HB_ERR_OOM, "attention split buffers for %d column slots", cap);
  L->part_cap = cap;
  return HB_OK;
}

// Upload `n` int32 through the next slot of the staging ring; *dev receives
// the slot's device copy, valid for the work enqueued on the layer's stream
// until stage_consumed(L, slot) is called after that work.
hb_status stage_upload(hb_layer* L, const int32_t* src, size_t n, const int32_t** dev, int* slot) {
  const int k = L->stage_next;
  Stage& s = L->stage[k];
  L->stage_next = (L->stage_next + 1) % kStages;
  if (s.pending) {
    HB_HIP(hipEventSynchronize(s.copied));  // the host buffer is free again
    s.pending = false;
  }
  if (n > s.cap) {
    if (s.host) HB_HIP(hipHostFree(s.host));
    s.host = nullptr;
    s.cap = 0;
    size_t cap = std::max<size_t>(n, 1 << 16);
    if (hipHostMalloc((void**)&s.host, cap * sizeof(int32_t), hipHostMallocDefault) != hipSuccess)
      return fail(HB_ERR_OOM, "pinned staging of %zu B", cap * 4);
    s.cap = cap;
  }
  if (n > s.dev_cap) {
    HB_HIP(hipEventSynchronize(s.consumed));  // no kernel reads the old copy any more
    dev_free(L, s.dev, s.dev_cap * sizeof(int32_t));
    s.dev = nullptr;
    s.dev_cap = 0;
    size_t cap = std::max<size_t>(n, 1 << 16);
    if (!dev_alloc(L, (void**)&s.dev, cap * sizeof(int32_t)))
      return fail(HB_ERR_OOM, "metadata buffer of %zu B", cap * 4);
    s.dev_cap = cap;
  }
  std::memcpy(s.host, src, n * sizeof(int32_t));
  HB_HIP(hipStreamWaitEvent(L->copy_stream, s.consumed, 0));
  HB_HIP(hipMemcpyAsync(s.dev, s.host, n * sizeof(int32_t), hipMemcpyHostToDevice, L->copy_stream));
  HB_HIP(hipEventRecord(s.copied, L->copy_stream));
  HB_HIP(hipStreamWaitEvent(L->stream, s.copied, 0));
  s.pending = true;
  *dev = s.dev;
  *slot = k;
  return HB_OK;
}

hb_status stage_consumed(hb_layer* L, int slot) {
  HB_HIP(hipEventRecord(L->stage[slot].consumed, L->stream));
  return HB_OK;
}

hb_status collect_timing(hb_layer* L) {
  if (L->timed.empty()) return HB_OK;
  HB_HIP(hipStreamSynchronize(L->stream));
  for (const TimedLaunch& t : L->timed) {
    float ms = 0.f;
    HB_HIP(hipEventElapsedTime(&ms, t.start, t.stop));
    L->tot_ms[t.kernel] += ms;
    L->launches[t.kernel] += 1;
    L->ev_free.push_back(t.start);
    L->ev_free.push_back(t.stop);
  }
  L->timed.clear();
  return HB_OK;
}

hb_status get_event(hb_layer* L, hipEvent_t* e) {
  if (L->ev_free.empty()) {
    HB_HIP(hipEventCreate(e));
    return HB_OK;
  }
  *e = L->ev_free.back();
  L->ev_free.pop_back();
  return HB_OK;
}

// Launch wrapper: brackets the launch with events when bit `kernel` of mask is set.
template <typename F>
hb_status timed(hb_layer* L, uint32_t mask, int kernel, F&& launch) {
  if (!((mask >> kernel) & 1u)) {
    launch();
    return HB_OK;
  }
  if (L->timed.size() >= 4096) {
    hb_status st = collect_timing(L);
    if (st != HB_OK) return st;
  }
  TimedLaunch t;
  t.kernel = kernel;
  hb_status st = get_event(L, &t.start);
  if (st == HB_OK) st = get_event(L, &t.stop);
  if (st != HB_OK) return st;
  HB_HIP(hipEventRecord(t.start, L->stream));
  launch();
  HB_HIP(hipEventRecord(t.stop, L->stream));
  L->timed.push_back(t);
  return HB_OK;
}

void free_layer(hb_layer* L) {
  if (!L) return;
  (void)hipStreamSynchronize(L->stream);
  for (void* p : {(void*)L->xn, (void*)L->rope_cs, (void*)L->tok_slot, (void*)L->q_rot, (void*)L->attn, (void*)L->mlp, (void*)L->h2,
                  (void*)L->inv_freq, (void*)L->part_o, (void*)L->part_ml, (void*)L->splitk})
    if (p) (void)hipFree(p);
  if (L->copy_stream) (void)hipStreamSynchronize(L->copy_stream);
  for (Stage& s : L->stage) {
    if (s.host) (void)hipHostFree(s.host);
    if (s.dev) (void)hipFree(s.dev);
    if (s.copied) (void)hipEventDestroy(s.copied);
    if (s.consumed) (void)hipEventDestroy(s.consumed);
  }
  if (L->copy_stream) (void)hipStreamDestroy(L->copy_stream);
  if (L->na_host) (void)hipHostFree(L->na_host);
  if (L->na_copied) (void)hipEventDestroy(L->na_copied);
  for (const TimedLaunch& t : L->timed) {
    (void)hipEventDestroy(t.start);
    (void)hipEventDestroy(t.stop);
  }
  for (hipEvent_t e : L->ev_free) (void)hipEventDestroy(e);
  delete L;
}

hb_status check_hip(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(HB_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return HB_OK;
}

// A planned batch made ready to launch: GEMM shapes and plans, workspaces
// sized, metadata uploaded (the layer's stream waits for the copy).
struct Prepared {
  const Plan* plan = nullptr;  // the batch's plan (metadata offsets, T)
  GemmArgs gq, go, gu, gd;
  GemmPlan pq, po, pu, pd;
  const int32_t* meta = nullptr;
  int slot = -1;             // metadata ring slot (-1: the metadata is not in the ring)
  float* splitk = nullptr;   // split-K partials
  float *part_o = nullptr, *part_ml = nullptr;  // attention split partials
  uint32_t timing_mask = 0;  // kernels bracketed by events
};

// The four GEMMs of an iteration over T tokens: shapes, epilogues and (when
// the layer is given) the buffers they read and write.
void layer_gemms(const Dims& d, int T, const hb_layer* L, const hb_batch_desc* desc, GemmArgs* g) {
  GemmArgs &gq = g[HB_GEMM_QKV], &go = g[HB_GEMM_O], &gu = g[HB_GEMM_GATE_UP], &gd = g[HB_GEMM_DOWN];
  gq = go = gu = gd = GemmArgs{};
  gq.lda = d.H; gq.ldb = d.H;
  gq.M = T; gq.N = d.qkv_n; gq.K = d.H;
  gq.ldc = d.nq * d.hd; gq.epi = GEMM_QKV_ROPE;
  gq.nq = d.nq; gq.nkv = d.nkv; gq.hd = d.hd;

  go.lda = d.nq * d.hd; go.ldb = d.nq * d.hd;
  go.M = T; go.N = d.H; go.K = d.nq * d.hd;
  go.ldc = d.H; go.c_f32 = 1;
  go.ldr = d.H; go.r_f32 = 0; go.epi = GEMM_RESIDUAL;
  go.norm_eps = d.eps;

  gu.lda = d.H; gu.ldb = d.H;
  gu.M = T; gu.N = d.F; gu.K = d.H;
  gu.ldc = d.F; gu.epi = GEMM_SWIGLU;

  gd.lda = d.F; gd.ldb = d.F;
  gd.M = T; gd.N = d.H; gd.K = d.F;
  gd.ldc = d.H; gd.c_f32 = 1;
  gd.ldr = d.H; gd.r_f32 = 1; gd.epi = GEMM_RESIDUAL;
  if (!L) return;

  gq.A = L->xn; gq.B = static_cast<const uint16_t*>(L->w.w_qkv); gq.C = L->q_rot;
  gq.rope_cs = L->rope_cs; gq.tok_slot = L->tok_slot;
  gq.k_pool = static_cast<uint16_t*>(L->pool.k_pool); gq.v_pool = static_cast<uint16_t*>(L->pool.v_pool);

  go.A = L->attn; go.B = static_cast<const uint16_t*>(L->w.w_o); go.C = L->h2;
  go.R = desc->x_in;
  // with a K split, the reduce also applies the pre-FFN RMSNorm
  go.norm_g = static_cast<const uint16_t*>(L->w.g_ffn); go.norm_out = L->xn;

  gu.A = L->xn; gu.B = static_cast<const uint16_t*>(L->w.w_gate_up); gu.C = L->mlp;

  gd.A = L->mlp; gd.B = static_cast<const uint16_t*>(L->w.w_down); gd.C = desc->x_out;
  gd.c_f32 = desc->out_dtype == HB_OUT_F32;
  gd.R = L->h2;
}

// An iteration's GEMM shapes and plans and the layer's buffers sized, for
// the batch planned in p (the metadata upload is left to the caller).
hb_status prepare_gemms(hb_layer* L, const hb_batch_desc* desc, const Plan& p, Prepared* pp) {
  const Dims& d = L->d;
  const int T = p.T;
  GemmArgs g[HB_GEMM_COUNT];
  layer_gemms(d, T, L, desc, g);
  const GemmArgs &gq = g[HB_GEMM_QKV], &go = g[HB_GEMM_O], &gu = g[HB_GEMM_GATE_UP], &gd = g[HB_GEMM_DOWN];

  const GemmPlan pq = plan_gemm(gq, L->cu_count, L->gemm_tile, L->gemm_ksplit),
                 po = plan_gemm(go, L->cu_count, L->gemm_tile, L->gemm_ksplit);
  const GemmPlan pu = plan_gemm(gu, L->cu_count, L->gemm_tile, L->gemm_ksplit),
                 pd = plan_gemm(gd, L->cu_count, L->gemm_tile, L->gemm_ksplit);
  size_t sk = 0;
  for (const auto& [pl, ga] : {std::make_pair(pq, gq), std::make_pair(po, go), std::make_pair(pu, gu),
                                std::make_pair(pd, gd)})
    if (pl.ksplit > 1) sk = std::max(sk, (size_t)pl.ksplit * ga.M * partial_width(ga));

  hb_status st = ensure_parts(L, p.n_slots);
  if (st == HB_OK) st = ensure_splitk(L, sk);
  if (st != HB_OK) return st;
  pp->gq = gq; pp->go = go; pp->gu = gu; pp->gd = gd;
  pp->pq = pq; pp->po = po; pp->pu = pu; pp->pd = pd;
  pp->splitk = L->splitk;
  pp->part_o = L->part_o;
  pp->part_ml = L->part_ml;
  pp->timing_mask = L->timing_mask;
  L->last_plans[HB_GEMM_QKV] = pq; L->last_plans[HB_GEMM_O] = po;
  L->last_plans[HB_GEMM_GATE_UP] = pu; L->last_plans[HB_GEMM_DOWN] = pd;
  pp->plan = &p;
  return HB_OK;
}

// Everything of an iteration up to its launches, for the batch in L->plan.
hb_status prepare_layer(hb_layer* L, const hb_batch_desc* desc, Prepared* pp) {
  const hb_status st = prepare_gemms(L, desc, L->plan, pp);
  if (st != HB_OK) return st;
  return stage_upload(L, L->plan.meta.data(), L->plan.meta.size(), &pp->meta, &pp->slot);
}

// The launches of a prepared iteration.
hb_status launch_layer(hb_layer* L, const hb_batch_desc* desc, const Prepared& pp) {
  // the metadata slot may be refilled once everything enqueued below has run
  struct Consumed {
    hb_layer* L;
    int slot;
    ~Consumed() {
      if (slot >= 0) (void)stage_consumed(L, slot);
    }
  } consumed{L, pp.slot};
  const uint32_t tm = pp.timing_mask;
  const Dims& d = L->d;
  const Plan& p = *pp.plan;
  const int T = p.T;
  hipStream_t s = L->stream;
  const uint16_t* x_in = static_cast<const uint16_t*>(desc->x_in);
  const GemmArgs &gq = pp.gq, &go = pp.go, &gu = pp.gu, &gd = pp.gd;
  const GemmPlan &pq = pp.pq, &po = pp.po, &pu = pp.pu, &pd = pp.pd;
  const int32_t* meta = pp.meta;
  hb_status st = HB_OK;

  RopePrep rp{};
  rp.tok_pos = meta + p.off_tok_pos; rp.tok_req = meta + p.off_tok_req;
  rp.req_bt = meta + p.off_req_bt; rp.bt = meta + p.off_bt;
  rp.inv_freq = L->inv_freq; rp.hd = d.hd; rp.cs = L->rope_cs; rp.slot = L->tok_slot;
  st = timed(L, tm, HB_K_RMSNORM_ATTN, [&] {
    launch_rmsnorm(s, x_in, false, static_cast<const uint16_t*>(L->w.g_attn), L->xn, T, d.H, d.eps, &rp);
  });
  if (st != HB_OK) return st;
  // q, k rotated and k, v scattered into the pool by the epilogue
  st = timed(L, tm, HB_K_GEMM_QKV, [&] { launch_gemm(s, gq, pq, pp.splitk); });
  if (st != HB_OK) return st;

  AttnArgs at{};
  at.q = L->q_rot; at.o = L->attn;
  at.k_pool = gq.k_pool; at.v_pool = gq.v_pool;
  at.tiles = meta + p.off_tiles; at.n_tiles = p.n_tiles;
  at.items = meta + p.off_items; at.n_items = p.n_items;
  at.units = meta + p.off_units; at.n_units = p.n_units;
  at.groups = meta + p.off_groups; at.n_groups = p.n_groups;
  at.merge_units = meta + p.off_merge; at.n_merge_units = p.n_merge_units;
  at.req_bt = rp.req_bt; at.bt = rp.bt;
  at.part_o = pp.part_o; at.part_ml = pp.part_ml;
  at.nq = d.nq; at.nkv = d.nkv; at.hd = d.hd;
  at.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)d.hd));
  st = timed(L, tm, HB_K_ATTENTION, [&] { launch_attention(s, at); });
  if (st != HB_OK) return st;
  if (p.n_groups > 0) {
    st = timed(L, tm, HB_K_ATTN_MERGE, [&] { launch_attn_merge(s, at); });
    if (st != HB_OK) return st;
  }
  bool ffn_norm_done = false;
  st = timed(L, tm, HB_K_GEMM_O, [&] { ffn_norm_done = launch_gemm(s, go, po, pp.splitk); });
  if (st != HB_OK) return st;
  if (!ffn_norm_done) {
    st = timed(L, tm, HB_K_RMSNORM_FFN, [&] {
      launch_rmsnorm(s, L->h2, true, static_cast<const uint16_t*>(L->w.g_ffn), L->xn, T, d.H, d.eps);
    });
    if (st != HB_OK) return st;
  }
  st = timed(L, tm, HB_K_GEMM_GATE_UP, [&] { launch_gemm(s, gu, pu, pp.splitk); });
  if (st != HB_OK) return st;
  st = timed(L, tm, HB_K_GEMM_DOWN, [&] { launch_gemm(s, gd, pd, pp.splitk); });
  if (st != HB_OK) return st;
  L->last_T = T;
  return check_hip("kernel launch");
}

// Enqueue the whole layer for the batch in L->plan.
hb_status enqueue_layer(hb_layer* L, const hb_batch_desc* desc) {
  Prepared pp;
  const hb_status st = prepare_layer(L, desc, &pp);
  if (st != HB_OK) return st;
  return launch_layer(L, desc, pp);
}

// Bring the device to its steady clocks before the first timed cell: after
// an idle period the GPU runs its first tens of milliseconds of work at lower
// clocks, which would inflate the first cells of a profile. Runs the batch
// untimed for at least kSettleMs of device time.
constexpr float kSettleMs = 100.f;

hb_status settle_device(hb_layer* L, const hb_batch_desc* desc, hipEvent_t e0, hipEvent_t e1) {
  hb_status st = hb_run_iteration(L, desc);  // plans, sizes the workspaces
  if (st != HB_OK) return st;
  HB_HIP(hipEventRecord(e0, L->stream));
  st = hb_run_iteration(L, desc);
  if (st != HB_OK) return st;
  HB_HIP(hipEventRecord(e1, L->stream));
  HB_HIP(hipEventSynchronize(e1));
  float ms = 0.f;
  HB_HIP(hipEventElapsedTime(&ms, e0, e1));
  const int n = std::min(2000, (int)std::ceil(kSettleMs / std::max(ms, 1e-3f)));
  for (int i = 0; i < n && st == HB_OK; ++i) st = hb_run_iteration(L, desc);
  return st;
}

// Time one batch as the profiler does: `warmup` untimed iterations, then
// `iters` iterations, each after a write of the first half of the
// `flush_bytes` buffer (no data left in the 256 MB Infinity Cache) and a
// read of its second half (which evicts the written lines, so that their
// write-back does not fall into the timed interval); the batch is planned
// and its metadata uploaded before the start event, so the interval holds
// the kernels alone. Fills the cell.
hb_status time_batch(hb_layer* L, const hb_batch_desc* desc, int warmup, int iters, void* flush,
                     int64_t flush_bytes, std::vector<hipEvent_t>& ev, std::vector<float>& lat, hb_profile_cell* cell) {
  hb_status st = check_batch(L->d, L->pool.num_blocks, desc, &L->marks);
  if (st != HB_OK) return st;
  for (int i = 0; i < warmup && st == HB_OK; ++i) st = hb_run_iteration(L, desc);
  if (st != HB_OK) return st;
  build_plan(L->d, desc, L->cu_count, &L->plan, L->plan_opt);
  for (int i = 0; i < iters && st == HB_OK; ++i) {
    launch_flush(L->stream, flush, flush_bytes, (uint32_t)i);
    Prepared pp;
    st = prepare_layer(L, desc, &pp);
    if (st != HB_OK) break;
    if (hipEventRecord(ev[2 * i], L->stream) != hipSuccess) st = fail(HB_ERR_HIP, "hipEventRecord failed");
    const hb_status sl = launch_layer(L, desc, pp);  // also releases the metadata slot
    if (st == HB_OK) st = sl;
    if (st == HB_OK && hipEventRecord(ev[2 * i + 1], L->stream) != hipSuccess)
      st = fail(HB_ERR_HIP, "hipEventRecord failed");
  }
  if (st != HB_OK) return st;
  if (hipStreamSynchronize(L->stream) != hipSuccess) return fail(HB_ERR_HIP, "profiler sync failed");
  for (int i = 0; i < iters; ++i)
    if (hipEventElapsedTime(&lat[i], ev[2 * i], ev[2 * i + 1]) != hipSuccess)
      return fail(HB_ERR_HIP, "hipEventElapsedTime failed");
  std::vector<float> sorted(lat.begin(), lat.begin() + iters);
  std::sort(sorted.begin(), sorted.end());
  auto pct = [&](double q) { return sorted[std::min<size_t>(sorted.size() - 1, (size_t)(q * (sorted.size() - 1) + 0.5))]; };
  cell->median_ms = pct(0.5);
  cell->p10_ms = pct(0.1);
  cell->p90_ms = pct(0.9);
  double flops, bytes;
  iteration_work(L->d, desc->requests, desc->n_requests, &flops, &bytes);
  int64_t T = 0;
  for (int r = 0; r < desc->n_requests; ++r) T += desc->requests[r].chunk_len;
  const double sec = cell->median_ms * 1e-3;
  cell->tokens_per_s = (float)(T / sec);
  cell->hbm_frac = (float)(bytes / sec / kPeakHbm);
  cell->mfma_frac = (float)(flops / sec / kPeakBf16);
  return HB_OK;
}

// splitmix64 stream for the profiler's host-side draws
struct SplitMix {
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
};

}  // namespace

namespace hb {

// Every layer is checked and its buffers sized before anything is enqueued,
// so a failure leaves every pool untouched. The metadata goes through the
// first layer's ring; its slot is released after the last layer's kernels.
hb_status run_layer_stack(hb_layer* const* layers, int n, const hb_batch_desc* desc, const void* const* x_in,
                          void* const* x_out) {
  if (n < 1 || !layers || !x_in || !x_out) return fail(HB_ERR_INVALID, "empty layer stack");
  for (int l = 0; l < n; ++l)
    if (!layers[l] || layers[l]->stream != layers[0]->stream)
      return fail(HB_ERR_INVALID, "layer %d is null or runs on another stream", l);
  hb_layer* L0 = layers[0];
  hb_status st = check_batch(L0->d, L0->pool.num_blocks, desc, &L0->marks);
  if (st != HB_OK) return st;
  if (desc->n_requests == 0) return HB_OK;
  build_plan(L0->d, desc, L0->cu_count, &L0->plan, L0->plan_opt);
  std::vector<hb_batch_desc> dl(n, *desc);
  std::vector<Prepared> pp(n);
  for (int l = 0; l < n; ++l) {
    dl[l].x_in = x_in[l];
    dl[l].x_out = x_out[l];
    st = prepare_gemms(layers[l], &dl[l], L0->plan, &pp[l]);
    if (st != HB_OK) return st;
  }
  const int32_t* meta = nullptr;
  int slot = -1;
  st = stage_upload(L0, L0->plan.meta.data(), L0->plan.meta.size(), &meta, &slot);
  if (st != HB_OK) return st;
  for (int l = 0; l < n && st == HB_OK; ++l) {
    pp[l].meta = meta;
    pp[l].slot = -1;
    st = launch_layer(layers[l], &dl[l], pp[l]);
  }
  const hb_status sc = stage_consumed(L0, slot);
  return st != HB_OK ? st : sc;
}

}  // namespace hb

extern "C" {

const char* hb_last_error(void) { return last_error(); }

hb_status hb_validate_batch(const hb_layer_config* cfg, int32_t num_blocks, const hb_batch_desc* desc) {
  Dims d;
  hb_status st = check_config(cfg, &d);
  if (st != HB_OK) return st;
  return check_batch(d, num_blocks, desc, nullptr);
}

hb_status hb_create_layer(const hb_layer_config* cfg, const hb_layer_weights* w, const hb_kv_pool* pool,
                          void* hip_stream, hb_layer** out) {
  if (!out) return fail(HB_ERR_INVALID, "null output handle");
  *out = nullptr;
  Dims d;
  hb_status st = check_config(cfg, &d);
  if (st != HB_OK) return st;
  if (d.H > 16384) return fail(HB_ERR_UNSUPPORTED, "hidden above 16384");
  if (!w || !w->w_qkv || !w->w_o || !w->w_gate_up || !w->w_down || !w->g_attn || !w->g_ffn)
    return fail(HB_ERR_INVALID, "null weight pointer");
  if (!pool || !pool->k_pool || !pool->v_pool || pool->num_blocks <= 0)
    return fail(HB_ERR_INVALID, "null or empty KV pool");
  hb_layer* L = new (std::nothrow) hb_layer();
  if (!L) return fail(HB_ERR_OOM, "host allocation of the layer");
  L->d = d;
  L->w = *w;
  L->pool = *pool;
  L->stream = static_cast<hipStream_t>(hip_stream);
  auto bail = [&](hb_status s) { free_layer(L); return s; };
  if (hipGetDevice(&L->device) != hipSuccess) return bail(fail(HB_ERR_HIP, "hipGetDevice failed"));
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, L->device) != hipSuccess) return bail(fail(HB_ERR_HIP, "hipGetDeviceProperties failed"));
  L->cu_count = prop.multiProcessorCount;
  if (const char* e = std::getenv("HB_GEMM_TILE")) L->gemm_tile = std::atoi(e);
  if (const char* e = std::getenv("HB_GEMM_KSPLIT")) L->gemm_ksplit = std::atoi(e);
  if (const char* e = std::getenv("HB_ATTN_SPLIT_TILE")) L->plan_opt.split_tile = std::atoi(e);
  if (const char* e = std::getenv("HB_ATTN_SPLIT_ITEM")) L->plan_opt.split_item = std::atoi(e);
  if (const char* e = std::getenv("HB_ATTN_UNIT_BLOCK")) L->plan_opt.unit_block = std::atoi(e);
  if (const char* e = std::getenv("HB_DEVICE_ALLOC_LIMIT")) L->dev_limit = std::strtoull(e, nullptr, 10);
  const size_t T = d.max_T;
  const size_t TA = T + kGemmPadRows;  // GEMM A operands: rows past M stay readable
  struct Alloc { void** p; size_t bytes; } allocs[] = {
      {(void**)&L->xn, TA * d.H * 2},        {(void**)&L->rope_cs, T * d.hd * 4},
      {(void**)&L->tok_slot, T * 4},
      {(void**)&L->q_rot, T * d.nq * d.hd * 2}, {(void**)&L->attn, TA * d.nq * d.hd * 2},
      {(void**)&L->mlp, TA * d.F * 2},       {(void**)&L->h2, T * d.H * 4},
      {(void**)&L->inv_freq, (size_t)d.hd / 2 * sizeof(double)},
  };
  for (auto& a : allocs)
    if (!dev_alloc(L, a.p, a.bytes)) return bail(fail(HB_ERR_OOM, "workspace allocation of %zu B", a.bytes));
  std::vector<double> inv(d.hd / 2);
  for (int j = 0; j < d.hd / 2; ++j) inv[j] = std::pow((double)d.theta, -2.0 * j / d.hd);
  if (hipMemcpy(L->inv_freq, inv.data(), inv.size() * sizeof(double), hipMemcpyHostToDevice) != hipSuccess)
    return bail(fail(HB_ERR_HIP, "upload of RoPE frequencies failed"));
  if (hipStreamCreateWithFlags(&L->copy_stream, hipStreamNonBlocking) != hipSuccess)
    return bail(fail(HB_ERR_HIP, "hipStreamCreate failed"));
  for (Stage& s : L->stage)
    if (hipEventCreateWithFlags(&s.copied, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&s.consumed, hipEventDisableTiming) != hipSuccess)
      return bail(fail(HB_ERR_HIP, "hipEventCreate failed"));
  st = ensure_parts(L, 1 << 16);
  if (st != HB_OK) return bail(st);
  st = scratch_address(L->device, &L->scratch);
  if (st != HB_OK) return bail(st);
  if (hipHostMalloc((void**)&L->na_host, kNoAllocMetaInts * sizeof(int32_t), hipHostMallocDefault) != hipSuccess)
    return bail(fail(HB_ERR_OOM, "pinned staging of %zu B", kNoAllocMetaInts * 4));
  if (hipEventCreateWithFlags(&L->na_copied, hipEventDisableTiming) != hipSuccess)
    return bail(fail(HB_ERR_HIP, "hipEventCreate failed"));
  *out = L;
  return HB_OK;
}

void hb_destroy_layer(hb_layer* layer) { free_layer(layer); }

hb_status hb_append_kv(hb_layer* L, const int32_t* block_table, int32_t n_blocks, int32_t context_len,
                       int32_t n_tokens, const void* k, const void* v) {
  if (!L) return fail(HB_ERR_INVALID, "null layer");
  if (n_tokens < 0 || context_len < 0) return fail(HB_ERR_INVALID, "negative n_tokens or context_len");
  if (n_tokens == 0) return HB_OK;
  if (!block_table || !k || !v) return fail(HB_ERR_INVALID, "null block_table, k or v");
  const int64_t kv = (int64_t)context_len + n_tokens;
  if (kv > ((int64_t)1 << 30)) return fail(HB_ERR_INVALID, "context too long");
  const int64_t nb = (kv + 15) / 16;
  if (n_blocks < nb) return fail(HB_ERR_INVALID, "block table has %d blocks, needs %lld", n_blocks, (long long)nb);
  for (int64_t i = context_len / 16; i < nb; ++i)
    if (block_table[i] < 0 || block_table[i] >= L->pool.num_blocks)
      return fail(HB_ERR_RANGE, "block_table[%lld] = %d outside [0, %d)", (long long)i, block_table[i],
                  L->pool.num_blocks);
  const int32_t* bt = nullptr;
  int slot = 0;
  hb_status st = stage_upload(L, block_table, (size_t)nb, &bt, &slot);
  if (st != HB_OK) return st;
  launch_append_kv(L->stream, static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), n_tokens,
                   context_len, bt, L->d.nkv, L->d.hd, static_cast<uint16_t*>(L->pool.k_pool),
                   static_cast<uint16_t*>(L->pool.v_pool));
  st = stage_consumed(L, slot);
  if (st != HB_OK) return st;
  return check_hip("append_kv launch");
}

hb_status hb_run_iteration(hb_layer* L, const hb_batch_desc* desc) {
  if (!L) return fail(HB_ERR_INVALID, "null layer");
  hb_status st = check_batch(L->d, L->pool.num_blocks, desc, &L->marks);
  if (st != HB_OK) return st;
  if (desc->n_requests == 0) return HB_OK;
  build_plan(L->d, desc, L->cu_count, &L->plan, L->plan_opt);
  return enqueue_layer(L, desc);
}

hb_status hb_run_iteration_noalloc(hb_layer* L, const hb_batch_desc* desc) {
  if (!L) return fail(HB_ERR_INVALID, "null layer");
  hb_status st = check_batch(L->d, L->pool.num_blocks, desc, &L->marks);
  if (st != HB_OK) return st;
  if (desc->n_requests == 0) return HB_OK;
  const Dims& d = L->d;
  build_plan(d, desc, L->cu_count, &L->plan, L->plan_opt);
  const Plan& p = L->plan;
  Prepared pp;
  GemmArgs g[HB_GEMM_COUNT];
  layer_gemms(d, p.T, L, desc, g);
  GemmPlan pl[HB_GEMM_COUNT];
  size_t splitk_floats = 0;
  for (int i = 0; i < HB_GEMM_COUNT; ++i) {
    pl[i] = plan_gemm(g[i], L->cu_count, L->gemm_tile, L->gemm_ksplit);
    if (pl[i].ksplit > 1) splitk_floats = std::max(splitk_floats, (size_t)pl[i].ksplit * g[i].M * partial_width(g[i]));
  }
  // scratch layout: metadata | split-K partials | attention partials (o, then m and l)
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t meta_bytes = p.meta.size() * sizeof(int32_t);
  const size_t off_splitk = up(meta_bytes);
  const size_t off_part_o = off_splitk + up(splitk_floats * sizeof(float));
  const size_t off_part_ml = off_part_o + up((size_t)p.n_slots * d.hd * sizeof(float));
  const size_t need = off_part_ml + up((size_t)p.n_slots * 2 * sizeof(float));
  if (need > kScratchBytes || p.meta.size() > kNoAllocMetaInts)
    return fail(HB_ERR_UNSUPPORTED,
                "batch needs %zu B of scratch (%zu B of metadata), the allocation-free entry point has %zu B "
                "(%zu B of metadata staging); use hb_run_iteration",
                need, meta_bytes, kScratchBytes, kNoAllocMetaInts * sizeof(int32_t));
  // the pinned staging is reused once the previous copy out of it is done
  if (L->na_pending) {
    HB_HIP(hipEventSynchronize(L->na_copied));
    L->na_pending = false;
  }
  std::memcpy(L->na_host, p.meta.data(), meta_bytes);
  HB_HIP(hipMemcpyAsync(L->scratch, L->na_host, meta_bytes, hipMemcpyHostToDevice, L->stream));
  HB_HIP(hipEventRecord(L->na_copied, L->stream));
  L->na_pending = true;
  pp.gq = g[HB_GEMM_QKV]; pp.go = g[HB_GEMM_O]; pp.gu = g[HB_GEMM_GATE_UP]; pp.gd = g[HB_GEMM_DOWN];
  pp.pq = pl[HB_GEMM_QKV]; pp.po = pl[HB_GEMM_O]; pp.pu = pl[HB_GEMM_GATE_UP]; pp.pd = pl[HB_GEMM_DOWN];
  pp.plan = &p;
  pp.meta = reinterpret_cast<const int32_t*>(L->scratch);
  pp.slot = -1;
  pp.splitk = reinterpret_cast<float*>(L->scratch + off_splitk);
  pp.part_o = reinterpret_cast<float*>(L->scratch + off_part_o);
  pp.part_ml = reinterpret_cast<float*>(L->scratch + off_part_ml);
  pp.timing_mask = 0;  // no events: creating them may allocate
  for (int i = 0; i < HB_GEMM_COUNT; ++i) L->last_plans[i] = pl[i];
  return launch_layer(L, desc, pp);
}

hb_status hb_set_kernel_timing(hb_layer* L, uint32_t mask) {
  if (!L) return fail(HB_ERR_INVALID, "null layer");
  if (mask >> HB_K_COUNT) return fail(HB_ERR_INVALID, "timing mask 0x%x has bits beyond the %d kernels", mask, HB_K_COUNT);
  L->timing_mask = mask;
  return HB_OK;
}

hb_status hb_kernel_times(hb_layer* L, double* total_ms, int64_t* launches, int32_t reset) {
  if (!L) return fail(HB_ERR_INVALID, "null layer");
  hb_status st = collect_timing(L);
  if (st != HB_OK) return st;
  for (int k = 0; k < HB_K_COUNT; ++k) {
    if (total_ms) total_ms[k] = L->tot_ms[k];
    if (launches) launches[k] = L->launches[k];
  }
  if (reset) {
    std::fill(L->tot_ms, L->tot_ms + HB_K_COUNT, 0.0);
    std::fill(L->launches, L->launches + HB_K_COUNT, (int64_t)0);
  }
  return HB_OK;
}

const char* hb_kernel_name(int32_t k) {
  static const char* names[HB_K_COUNT] = {"rmsnorm_attn", "gemm_qkv",  "attention", "attn_merge",
                                          "gemm_o",       "rmsnorm_ffn", "gemm_gate_up", "gemm_down"};
  return (k >= 0 && k < HB_K_COUNT) ? names[k] : "unknown";
}

int32_t hb_gemm_tile_count(void) { return gemm_tile_count(); }

hb_status hb_plan_gemms(const hb_layer_config* cfg, int32_t n_tokens, int32_t cu_count, int32_t force_tile,
                        int32_t force_ksplit, int32_t* tile, int32_t* ksplit) {
  if (!tile || !ksplit || n_tokens < 1 || cu_count < 1)
    return fail(HB_ERR_INVALID, "hb_plan_gemms: null pointer, n_tokens < 1 or cu_count < 1");
  Dims d;
  const hb_status st = check_config(cfg, &d);
  if (st != HB_OK) return st;
  GemmArgs g[HB_GEMM_COUNT];
  layer_gemms(d, n_tokens, nullptr, nullptr, g);
  for (int i = 0; i < HB_GEMM_COUNT; ++i) {
    const GemmPlan p = plan_gemm(g[i], cu_count, force_tile, force_ksplit);
    tile[i] = p.cfg;
    ksplit[i] = p.ksplit;
  }
  return HB_OK;
}

hb_status hb_layer_gemm_plans(hb_layer* L, int32_t* tile, int32_t* ksplit) {
  if (!L || !tile || !ksplit) return fail(HB_ERR_INVALID, "hb_layer_gemm_plans: null pointer");
  for (int i = 0; i < HB_GEMM_COUNT; ++i) {
    tile[i] = L->last_T > 0 ? L->last_plans[i].cfg : -1;
    ksplit[i] = L->last_T > 0 ? L->last_plans[i].ksplit : 0;
  }
  return HB_OK;
}

namespace {
// Two events, destroyed with the scope.
struct EventPair {
  hipEvent_t a = nullptr, b = nullptr;
  ~EventPair() {
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
  }
};
}  // namespace

hb_status hb_measure_device_rates(void* buf, int64_t bytes, void* stream, hb_device_rates* out) {
  if (!buf || !out || bytes < ((int64_t)1 << 30))
    return fail(HB_ERR_INVALID, "hb_measure_device_rates: null pointer or a buffer below 1 GiB (%lld bytes)",
                (long long)bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = 0, cus = 0;
  HB_HIP(hipGetDevice(&dev));
  HB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  cus = std::max(1, cus);
  const int64_t region = std::min<int64_t>(bytes, (int64_t)8 << 30) & ~(int64_t)4095;
  uint32_t* sink = static_cast<uint32_t*>(buf);
  EventPair ev;
  HB_HIP(hipEventCreate(&ev.a));
  HB_HIP(hipEventCreate(&ev.b));
  // best of three timed launches (ms)
  auto best_ms = [&](auto&& launch, float* ms) -> hipError_t {
    *ms = 0.f;
    for (int r = 0; r < 3; ++r) {
      hipError_t e = hipEventRecord(ev.a, s);
      if (e == hipSuccess) { launch(); e = hipGetLastError(); }
      if (e == hipSuccess) e = hipEventRecord(ev.b, s);
      if (e == hipSuccess) e = hipEventSynchronize(ev.b);
      float t = 0.f;
      if (e == hipSuccess) e = hipEventElapsedTime(&t, ev.a, ev.b);
      if (e != hipSuccess) return e;
      if (r == 0 || t < *ms) *ms = t;
    }
    return hipSuccess;
  };
  constexpr int kReadWgs = 2048, kChunksPerWave = 32, kMfmaIters = 4096;
  float ms_rand = 0.f, ms_stream = 0.f, ms_mfma = 0.f;
  HB_HIP(best_ms([&] { launch_probe_random_read(s, buf, (uint32_t)(region / 4096), kReadWgs, kChunksPerWave, sink); },
                 &ms_rand));
  HB_HIP(best_ms([&] { launch_probe_stream_read(s, buf, region, 8 * cus, sink); }, &ms_stream));
  HB_HIP(best_ms([&] { launch_probe_mfma(s, 2 * cus, kMfmaIters, sink); }, &ms_mfma));
  const double rand_bytes = (double)kReadWgs * 4 * kChunksPerWave * 4096;
  const double mfma_flops = (double)(2 * cus) * 4 * kMfmaIters * 16 * (2.0 * 16 * 16 * 32);
  out->random_4kb_read_bytes_per_s = ms_rand > 0.f ? rand_bytes / (ms_rand * 1e-3) : 0.0;
  out->stream_read_bytes_per_s = ms_stream > 0.f ? (double)region / (ms_stream * 1e-3) : 0.0;
  out->mfma_bf16_flop_per_s = ms_mfma > 0.f ? mfma_flops / (ms_mfma * 1e-3) : 0.0;
  return HB_OK;
}

hb_status hb_layer_stage(hb_layer* L, int32_t stage, void** dev_ptr, int64_t* row_stride) {
  if (!L || !dev_ptr || !row_stride) return fail(HB_ERR_INVALID, "null argument");
  switch (stage) {
    case HB_STAGE_Q: *dev_ptr = L->q_rot; *row_stride = (int64_t)L->d.nq * L->d.hd; break;
    case HB_STAGE_ATTN: *dev_ptr = L->attn; *row_stride = (int64_t)L->d.nq * L->d.hd; break;
    case HB_STAGE_H2: *dev_ptr = L->h2; *row_stride = L->d.H; break;
    case HB_STAGE_MLP: *dev_ptr = L->mlp; *row_stride = L->d.F; break;
    default: return fail(HB_ERR_INVALID, "unknown stage %d", stage);
  }
  return HB_OK;
}

hb_status hb_profile(hb_layer* L, const int32_t* chunk_sizes, int32_t n_chunk, const hb_decode_mix* mixes,
                     int32_t n_mix, int32_t warmup, int32_t iters, uint64_t seed, hb_profile_cell* out) {
  if (!L || !chunk_sizes || !mixes || !out) return fail(HB_ERR_INVALID, "null argument");
  if (n_chunk < 1 || n_mix < 1 || iters < 1 || warmup < 0) return fail(HB_ERR_INVALID, "empty grid or iters < 1");
  const Dims& d = L->d;
  const int NB = L->pool.num_blocks;
  // validate every cell before touching the device
  for (int mi = 0; mi < n_mix; ++mi) {
    const hb_decode_mix& mx = mixes[mi];
    if (mx.n_decode < 0 || (mx.n_decode > 0 && !mx.decode_contexts) || mx.chunk_context < 0)
      return fail(HB_ERR_INVALID, "mix %d malformed", mi);
    int64_t dec_blocks = 0;
    for (int i = 0; i < mx.n_decode; ++i) {
      if (mx.decode_contexts[i] < 0) return fail(HB_ERR_INVALID, "mix %d: negative decode context", mi);
      dec_blocks += (mx.decode_contexts[i] + 1 + 15) / 16;
    }
    for (int ci = 0; ci < n_chunk; ++ci) {
      const int c = chunk_sizes[ci];
      if (c < 1) return fail(HB_ERR_INVALID, "chunk size %d < 1", c);
      if ((int64_t)c + mx.n_decode > d.max_T || 1 + mx.n_decode > d.max_R)
        return fail(HB_ERR_INVALID, "cell (%d, mix %d) exceeds the layer's batch capacity", c, mi);
      if (dec_blocks + ((int64_t)mx.chunk_context + c + 15) / 16 > NB)
        return fail(HB_ERR_INVALID, "cell (%d, mix %d) needs more blocks than the pool holds", c, mi);
    }
  }
  int max_c = 0;
  for (int ci = 0; ci < n_chunk; ++ci) max_c = std::max(max_c, chunk_sizes[ci]);
  int max_dec = 0;
  for (int mi = 0; mi < n_mix; ++mi) max_dec = std::max(max_dec, mixes[mi].n_decode);
  const int64_t maxT = (int64_t)max_c + max_dec;
  const int64_t flush_bytes = (int64_t)1 << 30;  // 512 MiB written, 512 MiB read
  void *x_in = nullptr, *x_out = nullptr, *flush = nullptr;
  int32_t* blocks_dev = nullptr;
  std::vector<hipEvent_t> ev;
  hb_status st = HB_OK;
  auto cleanup = [&]() {
    (void)hipStreamSynchronize(L->stream);
    if (x_in) (void)hipFree(x_in);
    if (x_out) (void)hipFree(x_out);
    if (flush) (void)hipFree(flush);
    if (blocks_dev) (void)hipFree(blocks_dev);
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);
  };
  if (hipMalloc(&x_in, maxT * d.H * 2) != hipSuccess || hipMalloc(&x_out, maxT * d.H * 4) != hipSuccess ||
      hipMalloc(&flush, flush_bytes) != hipSuccess || hipMalloc(&blocks_dev, (size_t)NB * sizeof(int32_t)) != hipSuccess) {
    cleanup();
    return fail(HB_ERR_OOM, "profiler buffers");
  }
  ev.resize(2 * (size_t)iters);
  for (auto& e : ev)
    if (hipEventCreate(&e) != hipSuccess) { cleanup(); return fail(HB_ERR_HIP, "hipEventCreate failed"); }
  launch_fill_random_bf16(L->stream, static_cast<uint16_t*>(x_in), maxT * d.H, seed ^ 0xA5A5u, 1.7f);

  std::vector<int32_t> perm(NB);
  std::vector<hb_request> reqs;
  std::vector<float> lat(iters);
  for (int mi = 0; mi < n_mix && st == HB_OK; ++mi) {
    const hb_decode_mix& mx = mixes[mi];
    for (int ci = 0; ci < n_chunk && st == HB_OK; ++ci) {
      const int c = chunk_sizes[ci];
      // block ids: seeded Fisher-Yates permutation of the pool, consumed in request order
      SplitMix rng{seed * 1000003ull + (uint64_t)mi * 7919ull + (uint64_t)ci};
      for (int i = 0; i < NB; ++i) perm[i] = i;
      for (int i = NB - 1; i > 0; --i) std::swap(perm[i], perm[rng.next() % (uint64_t)(i + 1)]);
      reqs.clear();
      int used = 0;
      reqs.push_back({c, mx.chunk_context, perm.data() + used, (mx.chunk_context + c + 15) / 16});
      used += reqs.back().n_blocks;
      for (int i = 0; i < mx.n_decode; ++i) {
        reqs.push_back({1, mx.decode_contexts[i], perm.data() + used, (mx.decode_contexts[i] + 1 + 15) / 16});
        used += reqs.back().n_blocks;
      }
      if (hipMemcpyAsync(blocks_dev, perm.data(), (size_t)used * 4, hipMemcpyHostToDevice, L->stream) != hipSuccess ||
          hipStreamSynchronize(L->stream) != hipSuccess) {
        st = fail(HB_ERR_HIP, "profiler block upload failed");
        break;
      }
      launch_fill_blocks(L->stream, blocks_dev, used, d.nkv, d.hd, static_cast<uint16_t*>(L->pool.k_pool),
                         static_cast<uint16_t*>(L->pool.v_pool), seed + (uint64_t)used);
      hb_batch_desc desc{(int32_t)reqs.size(), reqs.data(), x_in, x_out, HB_OUT_F32};
      if (mi == 0 && ci == 0) st = settle_device(L, &desc, ev[0], ev[1]);
      if (st == HB_OK) st = time_batch(L, &desc, warmup, iters, flush, flush_bytes, ev, lat, &out[mi * n_chunk + ci]);
    }
  }
  cleanup();
  return st;
}

hb_status hb_profile_batches(hb_layer* L, const hb_batch_desc* batches, int32_t n_batches, int32_t warmup,
                             int32_t iters, hb_profile_cell* out) {
  if (!L || !out || n_batches < 0 || (n_batches > 0 && !batches)) return fail(HB_ERR_INVALID, "null argument");
  if (iters < 1 || warmup < 0) return fail(HB_ERR_INVALID, "iters < 1 or warmup < 0");
  for (int b = 0; b < n_batches; ++b) {
    const hb_status st = check_batch(L->d, L->pool.num_blocks, &batches[b], &L->marks);
    if (st != HB_OK) return st;
    if (batches[b].n_requests == 0) return fail(HB_ERR_INVALID, "batch %d is empty", b);
  }
  const int64_t flush_bytes = (int64_t)1 << 30;  // 512 MiB written, 512 MiB read
  void* flush = nullptr;
  std::vector<hipEvent_t> ev(2 * (size_t)iters, nullptr);
  std::vector<float> lat(iters);
  auto cleanup = [&]() {
    (void)hipStreamSynchronize(L->stream);
    if (flush) (void)hipFree(flush);
    for (hipEvent_t e : ev)
      if (e) (void)hipEventDestroy(e);
  };
  if (hipMalloc(&flush, flush_bytes) != hipSuccess) {
    cleanup();
    return fail(HB_ERR_OOM, "profiler flush buffer");
  }
  for (auto& e : ev)
    if (hipEventCreate(&e) != hipSuccess) { cleanup(); return fail(HB_ERR_HIP, "hipEventCreate failed"); }
  hb_status st = n_batches > 0 ? settle_device(L, &batches[0], ev[0], ev[1]) : HB_OK;
  for (int b = 0; b < n_batches && st == HB_OK; ++b)
    st = time_batch(L, &batches[b], warmup, iters, flush, flush_bytes, ev, lat, &out[b]);
  cleanup();
  return st;
}

}  // extern "C"
