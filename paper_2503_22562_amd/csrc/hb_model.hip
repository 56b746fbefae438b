// Whole-model iteration: token embedding, a stack of hybrid-batch decoder
// layers, final RMSNorm, LM head and greedy next-token choice. Every layer is
// an hb_layer; the stack runs through the layer runtime with the batch
// validated, planned and uploaded once per iteration. The model adds the
// embedding gather, the selection of each request's last row, the head GEMM
// (the layer GEMM with an fp32 store and no residual) and the argmax.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <vector>

#include "hb.h"
#include "hb_kernels.h"
#include "hb_plan.h"
#include "hb_runtime.h"

using namespace hb;

struct hb_model {
  hb_layer_config cfg{};
  std::vector<hb_layer*> layers;
  const uint16_t *embed = nullptr, *g_final = nullptr, *lm_head = nullptr;
  int vocab = 0, num_blocks = 0, cu_count = 0;
  hipStream_t stream = nullptr;
  uint16_t* x[2] = {nullptr, nullptr};  // bf16 [max_T][H]: hidden states between layers
  uint16_t* last = nullptr;             // bf16 [max_R][H]: each request's last row
  uint16_t* normed = nullptr;           // bf16 [max_R + kGemmPadRows][H]: head input
  float* logits = nullptr;              // fp32 [max_R][vocab] when the caller keeps none
  float* partial = nullptr;             // head GEMM split-K partials
  size_t partial_cap = 0;
  int32_t* rows_dev = nullptr;          // [max_R] last-row indices
  int32_t* rows_host = nullptr;         // pinned staging of rows_dev
  hipEvent_t rows_copied = nullptr;
  bool rows_pending = false;
};

namespace {

void free_model(hb_model* m) {
  if (!m) return;
  if (m->stream || !m->layers.empty()) (void)hipStreamSynchronize(m->stream);
  for (hb_layer* l : m->layers) hb_destroy_layer(l);
  for (void* p : {(void*)m->x[0], (void*)m->x[1], (void*)m->last, (void*)m->normed, (void*)m->logits,
                  (void*)m->partial, (void*)m->rows_dev})
    if (p) (void)hipFree(p);
  if (m->rows_host) (void)hipHostFree(m->rows_host);
  if (m->rows_copied) (void)hipEventDestroy(m->rows_copied);
  delete m;
}

}  // namespace

extern "C" {

hb_status hb_create_model(const hb_layer_config* cfg, const hb_model_desc* md, void* hip_stream, hb_model** out) {
  if (!out) return fail(HB_ERR_INVALID, "null output pointer");
  *out = nullptr;
  if (!cfg || !md || !md->layers || !md->pools || !md->embed || !md->g_final || !md->lm_head)
    return fail(HB_ERR_INVALID, "null model argument");
  Dims d;
  hb_status st = check_config(cfg, &d);
  if (st != HB_OK) return st;
  if (md->n_layers < 1) return fail(HB_ERR_INVALID, "n_layers %d < 1", md->n_layers);
  if (md->vocab < 8 || md->vocab % 8) return fail(HB_ERR_INVALID, "vocab %d: a positive multiple of 8", md->vocab);
  for (int l = 1; l < md->n_layers; ++l)
    if (md->pools[l].num_blocks != md->pools[0].num_blocks)
      return fail(HB_ERR_INVALID, "layer %d pool has %d blocks, layer 0 %d", l, md->pools[l].num_blocks,
                  md->pools[0].num_blocks);
  // the LM head is a B operand of the layer GEMM
  st = check_window("lm_head", md->vocab, d.H);
  if (st != HB_OK) return st;
  hb_model* m = new hb_model;
  m->cfg = *cfg;
  m->embed = static_cast<const uint16_t*>(md->embed);
  m->g_final = static_cast<const uint16_t*>(md->g_final);
  m->lm_head = static_cast<const uint16_t*>(md->lm_head);
  m->vocab = md->vocab;
  m->num_blocks = md->pools[0].num_blocks;
  m->stream = static_cast<hipStream_t>(hip_stream);
  auto bail = [&](hb_status s) { free_model(m); return s; };
  int dev = 0;
  hipDeviceProp_t prop;
  if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess)
    return bail(fail(HB_ERR_HIP, "device query failed"));
  m->cu_count = prop.multiProcessorCount;
  for (int l = 0; l < md->n_layers; ++l) {
    hb_layer* L = nullptr;
    st = hb_create_layer(cfg, &md->layers[l], &md->pools[l], hip_stream, &L);
    if (st != HB_OK) return bail(st);
    m->layers.push_back(L);
  }
  const size_t T = d.max_T, R = d.max_R, H = d.H;
  if (hipMalloc(&m->x[0], T * H * 2) != hipSuccess || hipMalloc(&m->x[1], T * H * 2) != hipSuccess ||
      hipMalloc(&m->last, R * H * 2) != hipSuccess ||
      hipMalloc(&m->normed, (R + kGemmPadRows) * H * 2) != hipSuccess ||
      hipMalloc(&m->logits, R * (size_t)m->vocab * 4) != hipSuccess ||
      hipMalloc(&m->rows_dev, R * 4) != hipSuccess ||
      hipHostMalloc((void**)&m->rows_host, R * 4, hipHostMallocDefault) != hipSuccess)
    return bail(fail(HB_ERR_OOM, "model workspace"));
  // the head reads whole row tiles: its padding rows stay finite
  if (hipMemsetAsync(m->normed, 0, (R + kGemmPadRows) * H * 2, m->stream) != hipSuccess ||
      hipEventCreateWithFlags(&m->rows_copied, hipEventDisableTiming) != hipSuccess)
    return bail(fail(HB_ERR_HIP, "model workspace setup"));
  *out = m;
  return HB_OK;
}

void hb_destroy_model(hb_model* m) { free_model(m); }

hb_layer* hb_model_layer(hb_model* m, int32_t index) {
  if (!m || index < 0 || index >= (int32_t)m->layers.size()) return nullptr;
  return m->layers[index];
}

hb_status hb_run_model(hb_model* m, const hb_model_batch* b) {
  if (!m || !b) return fail(HB_ERR_INVALID, "null model or batch");
  if (!b->token_ids || !b->next_tokens) return fail(HB_ERR_INVALID, "null token_ids or next_tokens");
  if (b->n_requests < 1) return fail(HB_ERR_INVALID, "empty batch");
  const hb_layer_config& c = m->cfg;
  const int H = c.hidden, R = b->n_requests;
  // validate through the first layer's check (all layers share shape and pool size)
  hb_batch_desc desc{b->n_requests, b->requests, m->x[0], m->x[1], HB_OUT_BF16};
  hb_status st = hb_validate_batch(&c, m->num_blocks, &desc);
  if (st != HB_OK) return st;
  int T = 0;
  for (int r = 0; r < R; ++r) T += b->requests[r].chunk_len;
  // last row of each request, staged through a pinned buffer
  if (m->rows_pending) {
    if (hipEventSynchronize(m->rows_copied) != hipSuccess) return fail(HB_ERR_HIP, "row staging wait failed");
    m->rows_pending = false;
  }
  for (int r = 0, t = 0; r < R; ++r) {
    t += b->requests[r].chunk_len;
    m->rows_host[r] = t - 1;
  }
  if (hipMemcpyAsync(m->rows_dev, m->rows_host, (size_t)R * 4, hipMemcpyHostToDevice, m->stream) != hipSuccess ||
      hipEventRecord(m->rows_copied, m->stream) != hipSuccess)
    return fail(HB_ERR_HIP, "row index upload failed");
  m->rows_pending = true;

  launch_gather_rows(m->stream, m->embed, m->vocab, b->token_ids, T, H, m->x[0]);
  // hidden states ping-pong between two buffers, or go to the caller's
  // per-layer slices
  // per-layer slices; every layer reads the one metadata upload
  uint16_t* hs = static_cast<uint16_t*>(b->hidden_states);
  const size_t nl = m->layers.size();
  std::vector<const void*> xin(nl);
  std::vector<void*> xout(nl);
  const uint16_t* cur = m->x[0];
  for (size_t l = 0; l < nl; ++l) {
    uint16_t* next = hs ? hs + l * (size_t)T * H : m->x[(cur == m->x[0]) ? 1 : 0];
    xin[l] = cur;
    xout[l] = next;
    cur = next;
  }
  st = run_layer_stack(m->layers.data(), (int)nl, &desc, xin.data(), xout.data());
  if (st != HB_OK) return st;
  launch_gather_rows(m->stream, cur, T, m->rows_dev, R, H, m->last);
  launch_rmsnorm(m->stream, m->last, false, m->g_final, m->normed, R, H, c.rms_eps);

  float* logits = b->logits ? b->logits : m->logits;
  GemmArgs g{};
  g.A = m->normed; g.lda = H;
  g.B = m->lm_head; g.ldb = H;
  g.M = R; g.N = m->vocab; g.K = H;
  g.C = logits; g.ldc = m->vocab; g.c_f32 = 1;
  g.R = nullptr; g.epi = GEMM_RESIDUAL;
  const GemmPlan p = plan_gemm(g, m->cu_count);
  if (p.ksplit > 1) {
    const size_t need = (size_t)p.ksplit * R * m->vocab;
    if (need > m->partial_cap) {
      if (hipStreamSynchronize(m->stream) != hipSuccess) return fail(HB_ERR_HIP, "model sync failed");
      if (m->partial) (void)hipFree(m->partial);
      m->partial = nullptr;
      m->partial_cap = 0;
      if (hipMalloc(&m->partial, need * 4) != hipSuccess) return fail(HB_ERR_OOM, "head split-K partials");
      m->partial_cap = need;
    }
  }
  launch_gemm(m->stream, g, p, m->partial);
  launch_argmax(m->stream, logits, R, m->vocab, b->next_tokens);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(HB_ERR_HIP, "model launch: %s", hipGetErrorString(e));
  return HB_OK;
}

}  // extern "C"
