/*
 * hb.h -- C ABI of the hybrid-batch decoder-layer library (libhb.so, gfx950).
 *
 * One call of hb_run_iteration executes one scheduler iteration of the kind
 * described in Section 3.1 (steps 5 and 6) and Section 3.3 of the Niyama
 * paper (arXiv 2503.22562): a single forward pass of one decoder layer over a
 * mixed batch that holds every decoding request (one new token each) and
 * prefill chunks whose length the dynamic-chunking policy chose. All linear
 * layers run once over the concatenated tokens (the fused prefill-decode MLP
 * of Section 3.3); attention reads each request's cached keys and values
 * through a paged KV cache (PagedAttention, Section 3.6). hb_profile measures
 * the latency of such iterations against chunk size and decode load, the
 * offline profile that the chunk-size predictor of Section 3.6 is trained on.
 *
 * The layer is the Llama-3 pre-norm decoder layer (the paper evaluates
 * Llama3-8B, evaluation setup): RMSNorm -> QKV projection -> rotate-half RoPE
 * -> causal GQA attention over the paged cache -> O projection + residual ->
 * RMSNorm -> SwiGLU FFN + residual. No biases.
 *
 * Conventions for every entry point:
 *  - Device pointers are HIP device memory on the device that was current
 *    when the layer was created; host pointers are ordinary host memory.
 *  - bf16 is IEEE bfloat16 (uint16 bit patterns), fp32 is IEEE binary32.
 *  - Every status other than HB_OK is returned before anything is enqueued,
 *    so nothing on the device is modified; hb_last_error() then describes it.
 *  - hb_run_iteration and hb_append_kv only enqueue work on the layer's
 *    stream and return; the caller synchronises that stream before reading
 *    results or reusing inputs. Host arrays passed to them (request tables,
 *    block tables) are copied during the call and may be freed on return.
 *  - A layer is used from one host thread at a time.
 */
#ifndef HB_H_
#define HB_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HB_OK = 0,
  HB_ERR_INVALID = 1,     /* malformed argument: null pointer, bad length, overlap */
  HB_ERR_RANGE = 2,       /* a block id outside [0, num_blocks) */
  HB_ERR_OOM = 3,         /* device or pinned host allocation failed */
  HB_ERR_HIP = 4,         /* a HIP runtime call failed; hb_last_error() names it */
  HB_ERR_UNSUPPORTED = 5  /* a shape the kernels do not implement */
} hb_status;

typedef struct hb_layer hb_layer; /* opaque, library-owned */

/* Layer shape and capacity.
 *   hidden        H, multiple of 64
 *   n_q_heads     query heads; n_q_heads % n_kv_heads == 0 and the group
 *                 size G = n_q_heads / n_kv_heads divides 16
 *   n_kv_heads    key/value heads (GQA: q head h reads kv head h / G)
 *   head_dim      64 or 128
 *   ffn_dim       F, multiple of 16
 *   kv_block_size must be 16 (tokens per paged block)
 *   rope_theta    RoPE base; angle of pair j at position p is p*theta^(-2j/head_dim)
 *   rms_eps       RMSNorm epsilon
 *   max_batch_tokens  largest T = sum of chunk_len accepted by hb_run_iteration
 *   max_requests      largest number of requests in one batch
 * Size limit: the GEMMs address each operand through a buffer window of
 * 2^31 - 16 bytes, so every weight matrix ((n_q + 2 n_kv) head_dim x H,
 * H x n_q head_dim, 2F x H, H x F) and every activation operand
 * ((max_batch_tokens + 512) rows of H, n_q head_dim or F bf16 values) must
 * fit in it; a configuration that does not is HB_ERR_UNSUPPORTED. */
typedef struct {
  int32_t hidden, n_q_heads, n_kv_heads, head_dim, ffn_dim, kv_block_size;
  float rope_theta, rms_eps;
  int32_t max_batch_tokens, max_requests;
} hb_layer_config;

/* Layer weights: device bf16, row-major [out][in], caller-owned, must outlive
 * the layer and stay unchanged while iterations run.
 *   w_qkv      [(n_q + 2 n_kv) head_dim][H]; rows = [q heads | k heads | v heads]
 *   w_o        [H][n_q head_dim]
 *   w_gate_up  [2F][H]; rows = [gate (F rows) | up (F rows)]
 *   w_down     [H][F]
 *   g_attn, g_ffn  [H] RMSNorm gains */
typedef struct {
  const void *w_qkv, *w_o, *w_gate_up, *w_down, *g_attn, *g_ffn;
} hb_layer_weights;

/* Paged KV cache of one layer: device bf16, caller-owned.
 *   k_pool  [num_blocks][n_kv_heads][2][head_dim/8][8][8]  K of slot s at
 *           [..][(s/4)%2][d/8][4(s/8) + s%4][d%8]
 *   v_pool  [num_blocks][n_kv_heads][2][head_dim][8]       V of slot s at [..][s/8][d][s%8]
 * Position p of a request lives in block block_table[p / 16], slot p % 16.
 * Keys are stored after RoPE. Both layouts keep a block of one kv head
 * (16 slots x head_dim) contiguous, 16 x head_dim x 2 bytes. K groups slots
 * 0-3, 8-11 and 4-7, 12-15 (the keys one score product takes), and stores
 * each group eight dimensions at a time, so a 16-byte read of eight
 * dimensions of eight keys is one 128-byte line. V is split into two halves
 * of eight slots, dimension-major inside a half: the eight keys of one
 * dimension are one 16-byte operand of the PV product. */
typedef struct {
  void *k_pool, *v_pool;
  int32_t num_blocks;
} hb_kv_pool;

/* Create a layer bound to weights, pool and a HIP stream (hipStream_t; NULL
 * selects the null stream). Allocates the library's workspace for
 * max_batch_tokens / max_requests on the current device.
 * Errors: HB_ERR_INVALID (null pointer, non-positive size),
 * HB_ERR_UNSUPPORTED (shape outside the limits above, including the 2 GiB
 * operand window), HB_ERR_OOM, HB_ERR_HIP. Configuration errors are found
 * before any HIP call. On error *out is set to NULL. */
hb_status hb_create_layer(const hb_layer_config* cfg, const hb_layer_weights* w,
                          const hb_kv_pool* pool, void* hip_stream, hb_layer** out);

/* Free the workspace (after synchronising the layer's stream). NULL is a no-op. */
void hb_destroy_layer(hb_layer* layer);

/* Write already-rotated keys and values of one request into the paged cache
 * (the cache of Section 3.6 that later iterations read).
 *   block_table  host int32 [n_blocks], physical block ids of the request
 *   context_len  position of the first token written
 *   n_tokens     tokens written: positions [context_len, context_len + n_tokens)
 *   k, v         device bf16 [n_tokens][n_kv_heads][head_dim]
 * Only those slots change; every other byte of the pool is left untouched.
 * Errors: HB_ERR_INVALID (null pointer, n_tokens < 0, context_len < 0,
 * n_blocks < ceil((context_len + n_tokens) / 16)), HB_ERR_RANGE (a used block
 * id outside [0, num_blocks)). n_tokens == 0 is a no-op. */
hb_status hb_append_kv(hb_layer* layer, const int32_t* block_table, int32_t n_blocks,
                       int32_t context_len, int32_t n_tokens, const void* k, const void* v);

/* One request of a hybrid batch (Section 3.1, step 5). A decode has
 * chunk_len == 1; a prefill chunk has chunk_len >= 1 new prompt tokens.
 *   context_len  tokens of this request already in the cache; the new tokens
 *                take positions [context_len, context_len + chunk_len) and
 *                each attends to every earlier position and to itself
 *   block_table  host int32 [n_blocks], n_blocks >= ceil((context_len + chunk_len) / 16) */
typedef struct {
  int32_t chunk_len, context_len;
  const int32_t* block_table;
  int32_t n_blocks;
} hb_request;

enum { HB_OUT_F32 = 0, HB_OUT_BF16 = 1 };

/* A hybrid batch: requests in any order; token rows of x_in / x_out are the
 * requests' new tokens concatenated in this order (chunk_len rows each).
 *   x_in   device bf16 [T][H] layer input (residual stream)
 *   x_out  device [T][H] layer output, fp32 (HB_OUT_F32) or bf16 (HB_OUT_BF16);
 *          must not overlap x_in */
typedef struct {
  int32_t n_requests;
  const hb_request* requests;
  const void* x_in;
  void* x_out;
  int32_t out_dtype;
} hb_batch_desc;

/* Run the decoder layer over the batch: write the new tokens' keys and values
 * into the cache, then compute x_out. Enqueues on the layer's stream.
 * Errors: as hb_validate_batch, plus HB_ERR_HIP / HB_ERR_OOM. n_requests == 0
 * is a no-op. Two requests may read the same block (shared prefix) but must
 * not write the same slot. */
hb_status hb_run_iteration(hb_layer* layer, const hb_batch_desc* desc);

/* hb_run_iteration for callers that cannot allocate device memory during the
 * call (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same kernels and launch plans, with the iteration's
 * scratch -- its metadata, split-K partial sums and attention split partials
 * -- in a fixed 64 MiB device array that the library holds on each GPU it
 * runs on for the life of the process (looked up when a layer is created),
 * and the metadata staged through pinned host memory the layer allocated at
 * creation (1 MiB). The call allocates no device or pinned memory and
 * records no timing events (hb_set_kernel_timing does not apply). Every call
 * on one GPU shares that GPU's array: calls whose iterations overlap on one
 * GPU (layers on different streams) race; calls on one stream are ordered.
 * Errors: those of hb_run_iteration, and HB_ERR_UNSUPPORTED for a batch whose
 * scratch exceeds 64 MiB or whose metadata exceeds 2^18 int32 (nothing is
 * enqueued then). */
hb_status hb_run_iteration_noalloc(hb_layer* layer, const hb_batch_desc* desc);

/* Check a batch against a layer configuration and pool size without touching
 * any device (no HIP call). Errors: HB_ERR_INVALID (null pointer,
 * chunk_len < 1, context_len < 0, short block table, T > max_batch_tokens,
 * n_requests > max_requests or < 0, bad out_dtype, overlapping x_in/x_out,
 * two requests writing one slot), HB_ERR_RANGE (a used block id outside
 * [0, num_blocks)), HB_ERR_UNSUPPORTED (config outside the limits). */
hb_status hb_validate_batch(const hb_layer_config* cfg, int32_t num_blocks, const hb_batch_desc* desc);

/* Decode load of one profile row: n_decode decodes with the given contexts
 * (host int32 [n_decode]) next to one prefill chunk starting at chunk_context. */
typedef struct {
  int32_t n_decode;
  const int32_t* decode_contexts;
  int32_t chunk_context;
} hb_decode_mix;

/* One profile cell: iteration latency (ms, median / 10th / 90th percentile),
 * new tokens per second at the median, and the algorithmic HBM bytes and MFMA
 * flops of the iteration divided by latency and by the MI355X peaks
 * (8 TB/s, 2.5 PFLOP/s bf16 dense). */
typedef struct {
  float median_ms, p10_ms, p90_ms, tokens_per_s, hbm_frac, mfma_frac;
} hb_profile_cell;

/* Latency profile for dynamic chunking (Section 3.3; the offline profiles of
 * Section 3.6): for every mix m and chunk size c, synthesise a batch of one
 * c-token chunk at mix.chunk_context plus the mix's decodes, with block tables
 * drawn from a seeded permutation of the whole pool, fill the blocks it uses
 * and its input with seeded pseudo-random bf16 (before the first cell, run
 * its batch untimed for 100 ms of device time, so that the GPU is at its
 * steady clocks), run `warmup` untimed
 * iterations, then `iters` iterations each preceded by a write of a 512 MiB
 * buffer (so no data stays in the 256 MB Infinity Cache) and a read of
 * another 512 MiB (so that no written line is left dirty: their write-back
 * would otherwise fall into the timed iteration), and timed with HIP
 * events; each timed iteration is planned and its metadata uploaded before
 * its start event, so the interval holds the layer's kernels alone.
 * out[m * n_chunk + c] receives the cell. Synchronous. Overwrites the
 * pool blocks it uses (an offline step). Errors: HB_ERR_INVALID (null
 * pointer, a batch that does not fit the pool or the layer's capacity,
 * iters < 1), HB_ERR_OOM, HB_ERR_HIP. */
hb_status hb_profile(hb_layer* layer, const int32_t* chunk_sizes, int32_t n_chunk,
                     const hb_decode_mix* mixes, int32_t n_mix, int32_t warmup, int32_t iters,
                     uint64_t seed, hb_profile_cell* out);

/* Latency of given batches, timed as hb_profile times its cells (the first
 * batch first run untimed for 100 ms of device time): for each
 * batch, `warmup` untimed iterations, then `iters` iterations each after a
 * write of a 512 MiB buffer and a read of another 512 MiB, each planned and its metadata uploaded before
 * the start event, so an interval holds the layer's kernels alone. The
 * caller supplies each batch's inputs, outputs and block tables (and the
 * pool contents); the iterations write the batch's new K/V as
 * hb_run_iteration does. out[b] receives batch b's cell. Synchronous.
 * Errors: those of hb_validate_batch for any batch (before anything runs),
 * HB_ERR_INVALID (null pointer, an empty batch, iters < 1, warmup < 0),
 * HB_ERR_OOM, HB_ERR_HIP. */
hb_status hb_profile_batches(hb_layer* layer, const hb_batch_desc* batches, int32_t n_batches, int32_t warmup,
                             int32_t iters, hb_profile_cell* out);

/* Iteration latency model: the lightweight predictor of Section 3.1 (step 4)
 * and Section 3.3, which the paper trains on offline profiles (Section 3.6),
 * here fitted to hb_profile cells. The predicted latency (ms) of a batch is
 * sum_i coef[i] * f_i over the features of the batch:
 *   f_0  1                                   (fixed per-iteration cost)
 *   f_1  T / 1000, T = sum of chunk_len       (the linear layers run over T tokens)
 *   f_2  KV bytes attention reads, GB: sum over requests of
 *        (context_len + chunk_len) * 2 n_kv_heads head_dim * 2 B
 *   f_3  attention flops against cached context, TFLOP:
 *        4 n_q_heads head_dim * sum over requests of chunk_len * context_len
 *   f_4  attention flops within the new tokens (the causal triangle), TFLOP:
 *        4 n_q_heads head_dim * sum over requests of chunk_len (chunk_len + 1) / 2
 * (long-context chunk rows run near the matrix-core rate, the triangle of a
 * fresh chunk much slower per flop, hence two terms).
 * A request with chunk_len 0 contributes nothing (it is not in the batch).
 * All coefficients are >= 0, so the prediction never falls as a chunk grows. */
#define HB_LAT_FEATURES 5
typedef struct {
  double coef[HB_LAT_FEATURES];
  double fit_rel_rms;   /* root mean square of (predicted - measured) / measured over the cells */
  double fit_max_under; /* largest measured / predicted - 1 over the cells (0 if none is under-predicted):
                           the margin hb_select_chunk needs for no fitted cell to exceed its slack */
  int32_t n_cells;
} hb_latency_model;

/* Features f_0..f_4 above of a batch (only chunk_len and context_len are read;
 * block tables may be NULL). Host only. Errors: HB_ERR_INVALID (null pointer,
 * n_requests < 0, chunk_len < 0 or context_len < 0 in a request). */
hb_status hb_latency_features(const hb_layer_config* cfg, const hb_request* requests, int32_t n_requests,
                              double* features);

/* Fit a model to the median latencies of an hb_profile run, given the same
 * chunk_sizes and mixes that produced cells[n_mix * n_chunk]: non-negative
 * least squares on relative error (each cell's row scaled by 1 / median), the
 * exact optimum over every subset of features. Host only. Errors:
 * HB_ERR_INVALID (null pointer, fewer cells than features, a median that is
 * not positive and finite). */
hb_status hb_fit_latency_model(const hb_layer_config* cfg, const int32_t* chunk_sizes, int32_t n_chunk,
                               const hb_decode_mix* mixes, int32_t n_mix, const hb_profile_cell* cells,
                               hb_latency_model* out);

/* Predicted latency (ms) of a batch. Host only. Errors as hb_latency_features. */
hb_status hb_predict_latency(const hb_latency_model* model, const hb_layer_config* cfg,
                             const hb_request* requests, int32_t n_requests, double* ms);

/* Dynamic chunking (Section 3.3): the slack of the decode queue is the least,
 * over its requests, of the deadline of the next token (the TBT deadline
 * equation of Section 3.2, decode_deadlines_ms[i], on the clock of now_ms)
 * minus now_ms; with no decodes it is unbounded. The chunk is the largest
 * c in {granularity, 2 granularity, ...} below max_chunk, or max_chunk itself
 * (the rest of the prompt), whose batch -- one c-token chunk at chunk_context
 * next to the decodes -- fits the slack with the caller's safety margin:
 * predicted latency * (1 + margin) <= slack (margin >= 0 covers the model's
 * error, e.g. model->fit_max_under, so that the chosen chunk violates no
 * deadline as Section 3.3 requires); 0 when none fits or max_chunk is 0.
 * *predicted_ms receives the predicted latency (without the margin) of the
 * chosen batch (decodes only when *chunk is 0). Host only. Errors:
 * HB_ERR_INVALID (null pointer, n_decode < 0, a negative context,
 * chunk_context < 0, max_chunk < 0, granularity < 1, margin < 0 or NaN, a NaN
 * deadline or now_ms). */
hb_status hb_select_chunk(const hb_latency_model* model, const hb_layer_config* cfg,
                          const int32_t* decode_contexts, const double* decode_deadlines_ms, int32_t n_decode,
                          double now_ms, int32_t chunk_context, int32_t max_chunk, int32_t granularity,
                          double margin, int32_t* chunk, double* predicted_ms);

/* Whole-model iteration: n_layers decoder layers (each an hb_layer with its
 * own weights and its own paged pool) between a token embedding and a final
 * RMSNorm + LM head, so the time between tokens of one scheduler iteration
 * (Section 3.1, steps 5-6) can be set against the TBT targets of the QoS
 * buckets (evaluation, QoS table: 50 ms for the strictest). Hidden states
 * pass between layers as bf16; greedy decoding takes the argmax.
 *   layers  [n_layers] weights as for hb_create_layer
 *   pools   [n_layers] paged pools, all with the same num_blocks: a request's
 *           block table names the same blocks in every layer's pool
 *   embed   device bf16 [vocab][H]; g_final device bf16 [H]; lm_head device
 *           bf16 [vocab][H]; vocab % 8 == 0, vocab * H * 2 bytes within the
 *           2 GiB operand window of the layer GEMMs
 * Caller-owned; everything must outlive the model. */
typedef struct hb_model hb_model; /* opaque, library-owned */
typedef struct {
  int32_t n_layers, vocab;
  const hb_layer_weights* layers;
  const hb_kv_pool* pools;
  const void *embed, *g_final, *lm_head;
} hb_model_desc;

/* Create a model on a HIP stream (all its layers use it). Errors as
 * hb_create_layer, HB_ERR_INVALID for n_layers < 1, vocab < 8 or not a
 * multiple of 8, pools of different sizes, null pointers, and
 * HB_ERR_UNSUPPORTED for an LM head beyond the 2 GiB operand window; all are
 * found before any HIP call. *out is NULL on error. */
hb_status hb_create_model(const hb_layer_config* cfg, const hb_model_desc* desc, void* hip_stream,
                          hb_model** out);
void hb_destroy_model(hb_model* model);

/* Layer `index` of a model (NULL for an index outside [0, n_layers)), owned
 * by the model: for hb_append_kv into that layer's pool, hb_layer_stage and
 * the per-kernel timing calls; not to be destroyed by the caller. */
hb_layer* hb_model_layer(hb_model* model, int32_t index);

/* One model iteration over a hybrid batch: requests as for hb_run_iteration
 * (their K/V are written into every layer's pool); token_ids device int32
 * [T] in descriptor order (ids outside [0, vocab) read the nearest embedding
 * row); for the last row of each request, logits (device fp32
 * [n_requests][vocab], or NULL to keep them internal) and next_tokens
 * (device int32 [n_requests]: the lowest index of the largest logit).
 * hidden_states: NULL, or device bf16 [n_layers][T][H] that receives every
 * layer's output (layer l reads its input from slice l - 1; for per-layer
 * checks); must not overlap the other buffers.
 * Enqueues on the model's stream and returns. Errors: those of
 * hb_run_iteration, HB_ERR_INVALID for null token_ids / next_tokens or an
 * empty batch. */
typedef struct {
  int32_t n_requests;
  const hb_request* requests;
  const int32_t* token_ids;
  float* logits;
  int32_t* next_tokens;
  void* hidden_states;
} hb_model_batch;
hb_status hb_run_model(hb_model* model, const hb_model_batch* batch);

/* Per-kernel timing of hb_run_iteration, for roofline accounting. Every
 * launch of kernel k with bit k of kernel_mask set is bracketed by HIP events
 * on the layer's stream (mask 0 turns timing off; timing one kernel keeps the
 * event overhead off the others). hb_kernel_times synchronises the stream and
 * adds the elapsed time (ms) and launch count of each kernel since the last
 * reset into total_ms[HB_K_COUNT] / launches[HB_K_COUNT]; reset != 0 starts a
 * new tally. Errors: HB_ERR_INVALID (null layer, mask bits beyond
 * HB_K_COUNT), HB_ERR_HIP. */
enum {
  HB_K_RMSNORM_ATTN = 0, HB_K_GEMM_QKV, HB_K_ATTENTION, HB_K_ATTN_MERGE,
  HB_K_GEMM_O, HB_K_RMSNORM_FFN, HB_K_GEMM_GATE_UP, HB_K_GEMM_DOWN, HB_K_COUNT
};
hb_status hb_set_kernel_timing(hb_layer* layer, uint32_t kernel_mask);
hb_status hb_kernel_times(hb_layer* layer, double* total_ms, int64_t* launches, int32_t reset);
const char* hb_kernel_name(int32_t kernel);

/* Intermediate results of the most recent iteration, for per-step checks.
 * Returns the library-owned device buffer of one step and its row stride in
 * elements; valid until the next hb_run_iteration or hb_destroy_layer.
 *   HB_STAGE_Q     bf16 [T][n_q head_dim]  queries after RoPE
 *   HB_STAGE_ATTN  bf16 [T][n_q head_dim]  attention output (before W_o)
 *   HB_STAGE_H2    fp32 [T][H]             x + attention @ W_o^T
 *   HB_STAGE_MLP   bf16 [T][F]             silu(gate) * up */
enum { HB_STAGE_Q = 0, HB_STAGE_ATTN = 1, HB_STAGE_H2 = 2, HB_STAGE_MLP = 3 };
hb_status hb_layer_stage(hb_layer* layer, int32_t stage, void** dev_ptr, int64_t* row_stride);

/* GEMM launch plans, for tests and tuning. The four GEMMs of the layer are
 * numbered HB_GEMM_QKV, HB_GEMM_O, HB_GEMM_GATE_UP, HB_GEMM_DOWN; a plan is a
 * tile-shape index in [0, hb_gemm_tile_count()) (-1: the register-staged
 * kernel used when K is not a multiple of 64) and a K split (1: none; > 1:
 * fp32 partials summed by a second kernel that applies the epilogue). */
enum { HB_GEMM_QKV = 0, HB_GEMM_O = 1, HB_GEMM_GATE_UP = 2, HB_GEMM_DOWN = 3, HB_GEMM_COUNT = 4 };
int32_t hb_gemm_tile_count(void);

/* The plans the library chooses for a batch of n_tokens tokens on a GPU with
 * cu_count compute units (host only). force_tile >= 0 / force_ksplit > 0
 * restrict the choice to one tile shape / K split as the HB_GEMM_TILE /
 * HB_GEMM_KSPLIT environment variables do when a layer is created (testing):
 * a forced choice that cannot run a GEMM is relaxed, the split first.
 * tile[HB_GEMM_COUNT], ksplit[HB_GEMM_COUNT] receive the plans. Errors:
 * HB_ERR_INVALID (null pointer, n_tokens < 1, cu_count < 1), configuration
 * errors as hb_create_layer. */
hb_status hb_plan_gemms(const hb_layer_config* cfg, int32_t n_tokens, int32_t cu_count, int32_t force_tile,
                        int32_t force_ksplit, int32_t* tile, int32_t* ksplit);

/* The plans of the layer's most recent iteration (0 tokens: all -1 / 0).
 * Errors: HB_ERR_INVALID (null pointer). */
hb_status hb_layer_gemm_plans(hb_layer* layer, int32_t* tile, int32_t* ksplit);

/* Sustained rates of the current device on three fixed access patterns,
 * measured for reading the kernels' roofline fractions against what the
 * device delivers (the published peaks remain the denominators of record):
 *   random_4kb_read_bytes_per_s  waves reading random 4-KB chunks of the first
 *                                min(bytes, 8 GiB) of buf (the pool-block pattern
 *                                of paged attention; the rate depends on the region
 *                                size), 2048 workgroups x 4 waves x 32 chunks;
 *   stream_read_bytes_per_s      a sequential grid-stride read of that region;
 *   mfma_bf16_flop_per_s         16x16x32 bf16 MFMAs on pseudo-random operands held
 *                                in registers, two 4-wave workgroups per CU (varied
 *                                data draws more power than constant operands).
 * Each is the best of three timed launches on `stream` (hipStream_t, 0 = the
 * null stream); the call waits for them. buf: device memory of `bytes` bytes,
 * at least 1 GiB so that the reads exceed the last-level cache, whose contents
 * are overwritten only in a case that does not occur in practice (treat it as
 * scratch). Errors: HB_ERR_INVALID (null pointer, bytes < 1 GiB), HB_ERR_HIP. */
typedef struct {
  double random_4kb_read_bytes_per_s;
  double stream_read_bytes_per_s;
  double mfma_bf16_flop_per_s;
} hb_device_rates;
hb_status hb_measure_device_rates(void* buf, int64_t bytes, void* stream, hb_device_rates* out);

/* Message for the last non-OK status returned on this host thread. */
const char* hb_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* HB_H_ */
