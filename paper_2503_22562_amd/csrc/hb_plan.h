// Host-side planning of one hybrid-batch iteration (no HIP calls).
//
// Turns a batch descriptor into the int32 metadata the kernels read: per-token
// position and request, per-request block-table offset, the block ids, the
// attention work list and the split-merge groups. Everything is packed into
// one array so one host-to-device copy moves it.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "hb.h"

namespace hb {

// Set the thread-local message returned by hb_last_error(); returns `st`.
hb_status fail(hb_status st, const char* fmt, ...);
const char* last_error();

struct Dims {
  int H = 0, nq = 0, nkv = 0, hd = 0, F = 0, blk = 16;
  int G = 0;      // q heads per kv head
  int P = 0;      // query positions of a 16-column wave item = 16 / G
  int BQ = 0;     // query positions of a workgroup tile = kTileCols / G
  int qkv_n = 0;  // (nq + 2 nkv) * hd
  float theta = 0.f, eps = 0.f;
  int max_T = 0, max_R = 0;
};

// Bytes of an operand the GEMMs can address: each operand is read through a
// raw buffer resource of this many records (and 32-bit byte offsets), so
// nothing past it may be needed. Rows past M that the GEMMs read from their
// activation operands (whole row tiles): kGemmPadRows.
constexpr int64_t kOperandWindow = 0x7FFFFFF0;
constexpr int kGemmPadRows = 512;

hb_status check_config(const hb_layer_config* cfg, Dims* d);

// HB_ERR_UNSUPPORTED unless rows x cols bf16 values fit the operand window.
hb_status check_window(const char* what, int64_t rows, int64_t cols);

// Attention work over the key positions [kv_begin, kv_end) of one request
// and kv head: a wave item covers 16 query columns (P positions x G heads), a
// workgroup tile kTileCols columns (BQ positions x G heads). part < 0: the unit
// writes the normalised output; otherwise its columns' partial results go to
// column slots part + c.
struct AttnItem {
  int32_t req, kv_head, tok0, pos0, npos, kv_begin, kv_end, part;
};
// Columns whose key range was split: part s of column c sits in slot
// part0 + s * stride + c.
struct MergeGroup {
  int32_t part0, nparts, stride, tok0, npos, kv_head, pad0, pad1;
};
static_assert(sizeof(AttnItem) == 32 && sizeof(MergeGroup) == 32, "packed as 8 int32");

// Each request's block ids are followed by kBtPad copies of its last id, so
// the four ids of a 64-key step can be read as one vector even at the end.
constexpr int kBtPad = 3;
// Query columns of a workgroup tile (32 per wave), and wave items grouped to
// a workgroup (one per wave): the attention workgroup has 4 waves.
constexpr int kTileCols = 128;
constexpr int kItemsPerUnit = 4;
// Work unit encoding: u >= 0 is tile u; -1 - v runs items 4 w .. 4 w + 3 with
// w = v & ~kUnitMerged, one per wave. Without kUnitMerged the four items are
// independent. With it they are consecutive key ranges of one (request, kv
// head, query positions), possibly empty (kv_begin == kv_end): the workgroup
// combines them in LDS and writes one result, to the output when item 4 w's
// part is < 0, else to that part's column slots.
constexpr int32_t kUnitMerged = 1 << 29;

struct Plan {
  int T = 0, R = 0;
  int n_tiles = 0, n_items = 0, n_units = 0, n_groups = 0, n_merge_units = 0;
  int n_slots = 0;  // partial-result column slots
  int split_tile = 0, split_item = 0;
  // offsets (int32 units) of each section inside meta
  int off_tok_pos = 0, off_tok_req = 0, off_req_bt = 0, off_bt = 0;
  int off_tiles = 0, off_items = 0, off_units = 0, off_groups = 0, off_merge = 0;
  std::vector<int32_t> meta;
  // algorithmic work of the iteration (for roofline accounting)
  double flops = 0, bytes = 0;
};

// Scratch reused across calls for the duplicate-slot check.
struct SlotMarks {
  std::vector<uint16_t> mask;    // per block: bit o set when slot o is written
  std::vector<int32_t> touched;  // blocks to clear afterwards
};

// Validate `desc` against the layer shape and a pool of num_blocks blocks.
hb_status check_batch(const Dims& d, int num_blocks, const hb_batch_desc* desc, SlotMarks* marks);

// Fixed split lengths (keys, multiples of 64; 0 = chosen from the batch),
// for tuning and tests.
struct PlanOptions {
  int split_tile = 0, split_item = 0;
  int unit_block = 0;  // runs of tiles / item groups in the unit order (0: one per CU; < 0: fine interleave)
};

// Build the plan of a validated batch for a GPU with cu_count compute units.
void build_plan(const Dims& d, const hb_batch_desc* desc, int cu_count, Plan* p,
                const PlanOptions& opt = PlanOptions());

// Algorithmic flops and HBM bytes of one iteration (what the method must
// compute and move, not what an implementation happens to do).
void iteration_work(const Dims& d, const hb_request* reqs, int n, double* flops, double* bytes);

}  // namespace hb
