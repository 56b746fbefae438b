// Host-side validation and planning of a hybrid-batch iteration (no HIP).
#include "hb_plan.h"

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>

namespace hb {

static thread_local std::string g_err;

hb_status fail(hb_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

const char* last_error() { return g_err.c_str(); }

hb_status check_config(const hb_layer_config* c, Dims* d) {
  if (!c) return fail(HB_ERR_INVALID, "null layer config");
  if (c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
      c->ffn_dim <= 0 || c->max_batch_tokens <= 0 || c->max_requests <= 0)
    return fail(HB_ERR_INVALID, "layer config sizes must be positive");
  if (!(c->rope_theta > 1.f) || !(c->rms_eps >= 0.f))
    return fail(HB_ERR_INVALID, "rope_theta must exceed 1 and rms_eps be >= 0");
  if (c->kv_block_size != 16) return fail(HB_ERR_UNSUPPORTED, "kv_block_size must be 16 (got %d)", c->kv_block_size);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(HB_ERR_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", c->head_dim);
  if (c->n_q_heads % c->n_kv_heads)
    return fail(HB_ERR_UNSUPPORTED, "n_q_heads (%d) must be a multiple of n_kv_heads (%d)", c->n_q_heads, c->n_kv_heads);
  int G = c->n_q_heads / c->n_kv_heads;
  if (G > 16 || 16 % G)
    return fail(HB_ERR_UNSUPPORTED, "q heads per kv head (%d) must divide 16", G);
  if (c->hidden % 64) return fail(HB_ERR_UNSUPPORTED, "hidden must be a multiple of 64 (got %d)", c->hidden);
  if (c->ffn_dim % 16) return fail(HB_ERR_UNSUPPORTED, "ffn_dim must be a multiple of 16 (got %d)", c->ffn_dim);
  if (c->max_batch_tokens > (1 << 20) || c->max_requests > (1 << 20))
    return fail(HB_ERR_UNSUPPORTED, "max_batch_tokens / max_requests above 2^20");
  {
    // every GEMM operand within the buffer window: the four weight matrices
    // and the three activation operands (with their padding rows)
    const int64_t H = c->hidden, F = c->ffn_dim, qd = (int64_t)c->n_q_heads * c->head_dim;
    const int64_t qkv = (int64_t)(c->n_q_heads + 2 * c->n_kv_heads) * c->head_dim;
    const int64_t TA = (int64_t)c->max_batch_tokens + kGemmPadRows;
    hb_status st = check_window("w_qkv", qkv, H);
    if (st == HB_OK) st = check_window("w_o", H, qd);
    if (st == HB_OK) st = check_window("w_gate_up", 2 * F, H);
    if (st == HB_OK) st = check_window("w_down", H, F);
    if (st == HB_OK) st = check_window("normed activations (max_batch_tokens + 512 rows)", TA, H);
    if (st == HB_OK) st = check_window("attention output (max_batch_tokens + 512 rows)", TA, qd);
    if (st == HB_OK) st = check_window("SwiGLU activations (max_batch_tokens + 512 rows)", TA, F);
    if (st != HB_OK) return st;
  }
  d->H = c->hidden;
  d->nq = c->n_q_heads;
  d->nkv = c->n_kv_heads;
  d->hd = c->head_dim;
  d->F = c->ffn_dim;
  d->blk = 16;
  d->G = G;
  d->P = 16 / G;
  d->BQ = kTileCols / G;
  d->qkv_n = (d->nq + 2 * d->nkv) * d->hd;
  d->theta = c->rope_theta;
  d->eps = c->rms_eps;
  d->max_T = c->max_batch_tokens;
  d->max_R = c->max_requests;
  return HB_OK;
}

hb_status check_window(const char* what, int64_t rows, int64_t cols) {
  if (rows * cols * 2 > kOperandWindow)
    return fail(HB_ERR_UNSUPPORTED, "%s: %lld x %lld bf16 values exceed the %lld-byte GEMM operand window", what,
                (long long)rows, (long long)cols, (long long)kOperandWindow);
  return HB_OK;
}

static int64_t blocks_for(int64_t kv_len) { return (kv_len + 15) / 16; }

hb_status check_batch(const Dims& d, int num_blocks, const hb_batch_desc* desc, SlotMarks* marks) {
  if (!desc) return fail(HB_ERR_INVALID, "null batch descriptor");
  const int R = desc->n_requests;
  if (R < 0) return fail(HB_ERR_INVALID, "n_requests < 0");
  if (R == 0) return HB_OK;
  if (R > d.max_R) return fail(HB_ERR_INVALID, "n_requests %d exceeds max_requests %d", R, d.max_R);
  if (!desc->requests) return fail(HB_ERR_INVALID, "null request array");
  if (!desc->x_in || !desc->x_out) return fail(HB_ERR_INVALID, "null x_in or x_out");
  if (desc->out_dtype != HB_OUT_F32 && desc->out_dtype != HB_OUT_BF16)
    return fail(HB_ERR_INVALID, "out_dtype must be HB_OUT_F32 or HB_OUT_BF16");
  if (num_blocks <= 0) return fail(HB_ERR_INVALID, "pool has no blocks");
  int64_t T = 0;
  for (int r = 0; r < R; ++r) {
    const hb_request& q = desc->requests[r];
    if (q.chunk_len < 1) return fail(HB_ERR_INVALID, "request %d: chunk_len %d < 1", r, q.chunk_len);
    if (q.context_len < 0) return fail(HB_ERR_INVALID, "request %d: context_len %d < 0", r, q.context_len);
    int64_t kv = (int64_t)q.context_len + q.chunk_len;
    if (kv > (int64_t)1 << 30) return fail(HB_ERR_INVALID, "request %d: context too long", r);
    if (!q.block_table) return fail(HB_ERR_INVALID, "request %d: null block_table", r);
    if (q.n_blocks < blocks_for(kv))
      return fail(HB_ERR_INVALID, "request %d: block table has %d blocks, needs %lld", r, q.n_blocks,
                  (long long)blocks_for(kv));
    for (int64_t i = 0; i < blocks_for(kv); ++i) {
      int32_t b = q.block_table[i];
      if (b < 0 || b >= num_blocks)
        return fail(HB_ERR_RANGE, "request %d: block_table[%lld] = %d outside [0, %d)", r, (long long)i, b, num_blocks);
    }
    T += q.chunk_len;
  }
  if (T > d.max_T) return fail(HB_ERR_INVALID, "batch has %lld tokens, max_batch_tokens is %d", (long long)T, d.max_T);
  // x_in (bf16) and x_out must not overlap
  {
    uintptr_t a0 = (uintptr_t)desc->x_in, a1 = a0 + (uintptr_t)T * d.H * 2;
    uintptr_t b0 = (uintptr_t)desc->x_out, b1 = b0 + (uintptr_t)T * d.H * (desc->out_dtype == HB_OUT_F32 ? 4 : 2);
    if (a0 < b1 && b0 < a1) return fail(HB_ERR_INVALID, "x_out overlaps x_in");
  }
  // no two new tokens may be written to the same physical slot
  SlotMarks local;
  SlotMarks* m = marks ? marks : &local;
  if ((int)m->mask.size() < num_blocks) m->mask.assign(num_blocks, 0);
  m->touched.clear();
  hb_status st = HB_OK;
  for (int r = 0; r < R && st == HB_OK; ++r) {
    const hb_request& q = desc->requests[r];
    for (int64_t p = q.context_len; p < (int64_t)q.context_len + q.chunk_len; ++p) {
      int32_t b = q.block_table[p / 16];
      uint16_t bit = (uint16_t)(1u << (p % 16));
      if (m->mask[b] == 0) m->touched.push_back(b);
      if (m->mask[b] & bit) {
        st = fail(HB_ERR_INVALID, "request %d writes slot %lld of block %d, already written by this batch", r,
                  (long long)(p % 16), b);
        break;
      }
      m->mask[b] |= bit;
    }
  }
  for (int32_t b : m->touched) m->mask[b] = 0;
  m->touched.clear();
  return st;
}

static int align16(int x) { return (x + 15) & ~15; }

void iteration_work(const Dims& d, const hb_request* reqs, int n, double* flops, double* bytes) {
  double T = 0, pairs = 0, kv_tokens = 0;
  for (int r = 0; r < n; ++r) {
    double c = reqs[r].chunk_len, x = reqs[r].context_len;
    T += c;
    pairs += c * x + c * (c + 1) / 2;
    kv_tokens += x + c;
  }
  double p_lin = (double)d.H * d.qkv_n + (double)d.nq * d.hd * d.H + 3.0 * d.H * d.F;
  *flops = 2.0 * T * p_lin + 4.0 * d.nq * d.hd * pairs;
  double kv_tok_bytes = 2.0 * d.nkv * d.hd * 2.0;  // K and V, bf16
  *bytes = 2.0 * p_lin + 2.0 * 2.0 * d.H         // weights and gains, bf16, once
           + kv_tokens * kv_tok_bytes            // cached + new K/V read once per (request, kv head)
           + T * kv_tok_bytes                    // new K/V written
           + T * d.H * 2.0 + T * d.H * 4.0;      // x_in bf16, y fp32
}

static int round_up(int64_t x, int m) { return (int)((x + m - 1) / m * m); }

void build_plan(const Dims& d, const hb_batch_desc* desc, int cu_count, Plan* p, const PlanOptions& opt) {
  const int R = desc->n_requests;
  const hb_request* rq = desc->requests;
  int T = 0, nbt = 0;
  std::vector<int> tok_start(R + 1, 0);
  for (int r = 0; r < R; ++r) {
    tok_start[r] = T;
    T += rq[r].chunk_len;
    nbt += (int)blocks_for((int64_t)rq[r].context_len + rq[r].chunk_len) + kBtPad;
  }
  tok_start[R] = T;
  p->T = T;
  p->R = R;

  // A chunk that fills at least half a workgroup tile goes to the workgroup
  // path; decodes and short chunks become 16-column wave items.
  auto is_tile = [&](int r) { return (int64_t)rq[r].chunk_len * d.G >= kTileCols / 2; };
  double tile_keys = 0, item_keys = 0;
  for (int r = 0; r < R; ++r) {
    const int c = rq[r].chunk_len, x = rq[r].context_len, w = is_tile(r) ? d.BQ : d.P;
    for (int i0 = 0; i0 < c; i0 += w) (is_tile(r) ? tile_keys : item_keys) += (double)d.nkv * (x + std::min(c, i0 + w));
  }
  // split lengths (multiples of 64 keys): about one round of tile workgroups
  // (each split also writes kTileCols columns of fp32 partials), and for
  // items about two wave slots' worth of keys per wave (4 per compute unit),
  // at least 1024 keys, so a merged unit spans up to 4 S_i keys and most
  // decodes need no merge kernel. When both kinds are present, tiles run
  // beside the bandwidth-bound items, and a tile is split only as far as it
  // would otherwise outlast the launch: the launch takes about the longer of
  // the items' K/V bytes at the HBM rate and the tile steps spread over the
  // workgroup slots (two per compute unit), and a tile step of 32 keys
  // (beside an item workgroup) takes about kMixedStepUs. Measured on MI355X
  // over chunk/decode mixes of the 8B and 70B layers and of their
  // tensor-parallel shards (item split 256 .. 4096, tile split 1024 .. 16384).
  constexpr double kMixedStepUs = 0.6, kItemBytesPerUs = 6.0e6;
  const int cus = std::max(1, cu_count);
  const bool mixed = tile_keys > 0 && item_keys > 0;
  double s_t = tile_keys / (1.0 * cus);
  if (mixed) {
    const double launch_us = std::max(item_keys * 4.0 * d.hd / kItemBytesPerUs,
                                      tile_keys / 32.0 * kMixedStepUs / (2.0 * cus));
    s_t = launch_us / kMixedStepUs * 32.0;
  }
  const int S_t_auto = std::max(1024, round_up((int64_t)std::min(s_t, 1.0e9) + 1, 64));
  const int S_t = opt.split_tile > 0 ? round_up(opt.split_tile, 64) : S_t_auto;
  const int S_i = opt.split_item > 0 ? round_up(opt.split_item, 64)
                                     : std::max(1024, round_up((int64_t)(item_keys / (16.0 * cus)) + 1, 64));
  p->split_tile = S_t;
  p->split_item = S_i;

  // Tiles: one work unit per (request, kv head, position block, key split).
  // Items: a (request, kv head, position group) whose keys fit one split
  // length is one wave item, packed four to a unit with items of similar
  // length. A longer range is cut over k = ceil(n / 4) workgroups of four
  // waves (n = its split count); each workgroup's four waves take
  // consecutive sub-ranges and combine them in LDS, so only ranges that need
  // more than one workgroup leave partial results for the merge kernel.
  std::vector<AttnItem> tiles, singles;
  struct Unit {
    int64_t len;     // keys of the unit's longest wave
    int first;       // first item (merged) or first single
    bool merged;
  };
  std::vector<AttnItem> merged_items;
  std::vector<Unit> merged_units;
  struct SplitTile {
    int first, n, kv_len;  // its pieces are tiles[first .. first + n)
  };
  std::vector<SplitTile> split_tiles;
  std::vector<MergeGroup> groups;
  int slots = 0;
  for (int r = 0; r < R; ++r) {
    const int c = rq[r].chunk_len, x = rq[r].context_len;
    const bool tile = is_tile(r);
    const int w = tile ? d.BQ : d.P, S = tile ? S_t : S_i;
    for (int g = 0; g < d.nkv; ++g) {
      for (int i0 = 0; i0 < c; i0 += w) {
        const int npos = std::min(w, c - i0);
        const int kv_len = x + i0 + npos;
        const int nspl = (kv_len + S - 1) / S;
        if (tile) {
          int part0 = -1;
          if (nspl > 1) {
            part0 = slots;
            groups.push_back({slots, nspl, kTileCols, tok_start[r] + i0, npos, g, 0, 0});
            slots += nspl * kTileCols;
          }
          if (nspl > 1) split_tiles.push_back({(int)tiles.size(), nspl, kv_len});
          for (int s = 0; s < nspl; ++s)
            tiles.push_back({r, g, tok_start[r] + i0, x + i0, npos, s * S, std::min(kv_len, (s + 1) * S),
                             nspl > 1 ? part0 + s * kTileCols : -1});
          continue;
        }
        if (nspl == 1) {
          singles.push_back({r, g, tok_start[r] + i0, x + i0, npos, 0, kv_len, -1});
          continue;
        }
        const int k = (nspl + kItemsPerUnit - 1) / kItemsPerUnit;
        const int wlen = round_up((kv_len + k - 1) / k, 64);
        int part0 = -1;
        if (k > 1) {
          part0 = slots;
          groups.push_back({slots, k, 16, tok_start[r] + i0, npos, g, 0, 0});
          slots += 16 * k;
        }
        for (int j = 0; j < k; ++j) {
          const int b = j * wlen, e = std::min(kv_len, b + wlen);
          const int plen = round_up((e - b + kItemsPerUnit - 1) / kItemsPerUnit, 64);
          merged_units.push_back({plen, (int)merged_items.size(), true});
          for (int q = 0; q < kItemsPerUnit; ++q) {
            const int pb = std::min(e, b + q * plen), pe = std::min(e, pb + plen);
            merged_items.push_back({r, g, tok_start[r] + i0, x + i0, npos, pb, pe, k > 1 ? part0 + 16 * j : -1});
          }
        }
      }
    }
  }
  // A split tile is cut at multiples of S_t (full pieces and a shorter
  // last one). When every work unit gets a workgroup slot of its own (two
  // per compute unit), nothing queues behind a piece and the launch lasts as
  // long as the longest one, so the pieces are evened out instead (64-key
  // multiples, at most S_t; the piece count is unchanged). With more units
  // than slots, even pieces would add long units to the queue; the short
  // last pieces fill gaps there.
  const int64_t item_unit_count = (int64_t)merged_units.size() + ((int64_t)singles.size() + kItemsPerUnit - 1) / kItemsPerUnit;
  if ((int64_t)tiles.size() + item_unit_count <= 2 * (int64_t)std::max(1, cu_count)) {
    for (const SplitTile& st : split_tiles) {
      const int piece = round_up((st.kv_len + st.n - 1) / st.n, 64);
      for (int s = 0; s < st.n; ++s) {
        tiles[st.first + s].kv_begin = s * piece;
        tiles[st.first + s].kv_end = std::min(st.kv_len, (s + 1) * piece);
      }
    }
  }
  // longest first (greedy list scheduling over the compute units), and items
  // of similar length share a workgroup, which lasts as long as its longest
  auto longer = [](const AttnItem& x, const AttnItem& y) {
    return (x.kv_end - x.kv_begin) * (int64_t)x.npos > (y.kv_end - y.kv_begin) * (int64_t)y.npos;
  };
  std::stable_sort(tiles.begin(), tiles.end(), longer);
  std::stable_sort(singles.begin(), singles.end(), [](const AttnItem& x, const AttnItem& y) {
    return (x.kv_end - x.kv_begin) > (y.kv_end - y.kv_begin);
  });
  std::vector<Unit> item_units = merged_units;
  for (int i = 0; i < (int)singles.size(); i += kItemsPerUnit)
    item_units.push_back({singles[i].kv_end - singles[i].kv_begin, i, false});
  std::stable_sort(item_units.begin(), item_units.end(), [](const Unit& x, const Unit& y) { return x.len > y.len; });
  // items in unit order: unit v's items are 4 v .. 4 v + 3 (the last unit of
  // singles is padded with empty items)
  std::vector<AttnItem> items;
  std::vector<int32_t> item_unit_codes;
  items.reserve(merged_items.size() + singles.size() + kItemsPerUnit);
  for (const Unit& u : item_units) {
    const int v = (int)(items.size() / kItemsPerUnit);
    item_unit_codes.push_back(-1 - (u.merged ? (v | kUnitMerged) : v));
    const std::vector<AttnItem>& src = u.merged ? merged_items : singles;
    const int n = std::min<int>(kItemsPerUnit, (int)src.size() - u.first);
    for (int q = 0; q < n; ++q) items.push_back(src[u.first + q]);
    for (int q = n; q < kItemsPerUnit; ++q) {
      AttnItem e = src[u.first];
      e.kv_begin = e.kv_end;  // empty: the wave does nothing
      items.push_back(e);
    }
  }
  // work units: one per tile, one per item unit, in alternating runs of one
  // unit per CU: workgroups are handed out round-robin over the CUs, two per
  // CU, so a CU's first two workgroups are a compute-bound tile and a
  // bandwidth-bound item unit, which overlap well
  const int nt = (int)tiles.size(), ni_units = (int)item_unit_codes.size();
  std::vector<int32_t> units;
  units.reserve(nt + ni_units);
  const int run = opt.unit_block != 0 ? opt.unit_block : cus;
  if (run > 0) {
    for (int a = 0, b = 0; a < nt || b < ni_units;) {
      for (int k = 0; k < run && a < nt; ++k) units.push_back(a++);
      for (int k = 0; k < run && b < ni_units; ++k) units.push_back(item_unit_codes[b++]);
    }
  } else {
    for (int a = 0, b = 0; a < nt || b < ni_units;) {
      if (b >= ni_units || (a < nt && (int64_t)a * ni_units <= (int64_t)b * nt)) units.push_back(a++);
      else units.push_back(item_unit_codes[b++]);
    }
  }
  p->n_tiles = nt;
  p->n_items = (int)items.size();
  p->n_units = (int)units.size();
  p->n_groups = (int)groups.size();
  p->n_slots = slots;
  std::vector<int32_t> merge;
  for (int gi = 0; gi < p->n_groups; ++gi)
    for (int cb = 0; cb * 16 < groups[gi].npos * d.G; ++cb) merge.push_back(gi * 16 + cb);
  p->n_merge_units = (int)merge.size();

  int off = 0;
  p->off_tok_pos = off;  off += align16(T);
  p->off_tok_req = off;  off += align16(T);
  p->off_req_bt = off;   off += align16(R);
  p->off_bt = off;       off += align16(nbt);
  p->off_tiles = off;    off += align16(8 * nt);
  p->off_items = off;    off += align16(8 * p->n_items);
  p->off_units = off;    off += align16(p->n_units);
  p->off_groups = off;   off += align16(8 * p->n_groups);
  p->off_merge = off;    off += align16(p->n_merge_units);
  p->meta.assign(off, 0);
  int32_t* m = p->meta.data();
  int bt_off = 0;
  for (int r = 0; r < R; ++r) {
    for (int i = 0; i < rq[r].chunk_len; ++i) {
      m[p->off_tok_pos + tok_start[r] + i] = rq[r].context_len + i;
      m[p->off_tok_req + tok_start[r] + i] = r;
    }
    m[p->off_req_bt + r] = bt_off;
    const int nb = (int)blocks_for((int64_t)rq[r].context_len + rq[r].chunk_len);
    std::memcpy(m + p->off_bt + bt_off, rq[r].block_table, sizeof(int32_t) * nb);
    for (int i = 0; i < kBtPad; ++i) m[p->off_bt + bt_off + nb + i] = rq[r].block_table[nb - 1];
    bt_off += nb + kBtPad;
  }
  if (nt) std::memcpy(m + p->off_tiles, tiles.data(), sizeof(AttnItem) * nt);
  if (!items.empty()) std::memcpy(m + p->off_items, items.data(), sizeof(AttnItem) * items.size());
  if (!units.empty()) std::memcpy(m + p->off_units, units.data(), sizeof(int32_t) * units.size());
  if (!groups.empty()) std::memcpy(m + p->off_groups, groups.data(), sizeof(MergeGroup) * groups.size());
  if (!merge.empty()) std::memcpy(m + p->off_merge, merge.data(), sizeof(int32_t) * merge.size());
  iteration_work(d, rq, R, &p->flops, &p->bytes);
}

}  // namespace hb
