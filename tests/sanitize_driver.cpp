// Host-code driver for the sanitizer test: exercises the batch validation,
// the planner, the work accounting, the latency model and the chunk selector
// (hb_plan.cpp, hb_predict.cpp; no HIP) on seeded random batches, valid and
// malformed. Built with AddressSanitizer and UndefinedBehaviorSanitizer; any
// report aborts the process with a non-zero status.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "hb.h"
#include "hb_plan.h"

namespace {

struct Batch {
  std::vector<hb_request> reqs;
  std::vector<std::vector<int32_t>> tables;
};

// Requests of random chunk / context lengths with block ids from a shuffled
// pool; `malform` corrupts one field of one request.
Batch random_batch(std::mt19937_64& rng, int num_blocks, int max_req, int max_ctx, int malform) {
  Batch b;
  const int R = 1 + (int)(rng() % max_req);
  std::vector<int32_t> perm(num_blocks);
  for (int i = 0; i < num_blocks; ++i) perm[i] = i;
  std::shuffle(perm.begin(), perm.end(), rng);
  int used = 0;
  for (int r = 0; r < R; ++r) {
    const int chunk = (rng() % 4 == 0) ? 1 + (int)(rng() % 700) : 1;
    const int ctx = (int)(rng() % (max_ctx + 1));
    const int nb = (ctx + chunk + 15) / 16;
    if (used + nb > num_blocks) break;
    b.tables.emplace_back(perm.begin() + used, perm.begin() + used + nb);
    used += nb;
    b.reqs.push_back({chunk, ctx, nullptr, nb});
  }
  if (b.reqs.empty()) {
    b.tables.push_back({0});
    b.reqs.push_back({1, 0, nullptr, 1});
  }
  for (size_t r = 0; r < b.reqs.size(); ++r) b.reqs[r].block_table = b.tables[r].data();
  if (malform) {
    hb_request& q = b.reqs[rng() % b.reqs.size()];
    switch (malform) {
      case 1: q.chunk_len = 0; break;
      case 2: q.context_len = -5; break;
      case 3: q.n_blocks = q.n_blocks - 1; break;
      case 4: const_cast<int32_t*>(q.block_table)[0] = num_blocks + 3; break;
      case 5: const_cast<int32_t*>(q.block_table)[0] = -1; break;
      default: b.reqs.push_back(b.reqs[0]); break;  // the same slots written twice
    }
  }
  return b;
}

}  // namespace

int main() {
  std::mt19937_64 rng(20250322);
  const hb_layer_config shapes[] = {
      {256, 4, 2, 64, 688, 16, 5e5f, 1e-5f, 8192, 300},
      {4096, 32, 8, 128, 14336, 16, 5e5f, 1e-5f, 8192, 300},
      {8192, 64, 8, 128, 28672, 16, 5e5f, 1e-5f, 8192, 300},
      {1024, 16, 1, 64, 512, 16, 5e5f, 1e-5f, 8192, 300},
  };
  int ok = 0, rejected = 0;
  for (int iter = 0; iter < 400; ++iter) {
    const hb_layer_config& cfg = shapes[iter % 4];
    hb::Dims d;
    if (hb::check_config(&cfg, &d) != HB_OK) return 10;
    const int num_blocks = 20000;
    const int malform = (iter % 3 == 0) ? 1 + (int)(rng() % 6) : 0;
    Batch b = random_batch(rng, num_blocks, 260, 9000, malform);
    hb_batch_desc desc{(int32_t)b.reqs.size(), b.reqs.data(), (void*)0x1000, (void*)0x80000000, HB_OUT_F32};
    hb::SlotMarks marks;
    const hb_status st = hb::check_batch(d, num_blocks, &desc, &marks);
    if (st != HB_OK) {
      ++rejected;
      continue;
    }
    ++ok;
    hb::Plan p;
    hb::PlanOptions opt;
    if (iter % 5 == 1) opt.split_tile = 1024, opt.split_item = 512;
    hb::build_plan(d, &desc, 256, &p, opt);
    double fl = 0, by = 0;
    hb::iteration_work(d, b.reqs.data(), (int)b.reqs.size(), &fl, &by);
    double f[HB_LAT_FEATURES];
    if (hb_latency_features(&cfg, b.reqs.data(), (int32_t)b.reqs.size(), f) != HB_OK) return 11;
  }
  // latency model: fit on a grid, predict, select
  const hb_layer_config& cfg = shapes[1];
  const int32_t chunks[] = {128, 256, 512, 1024, 2048};
  std::vector<int32_t> dec(256);
  for (auto& c : dec) c = 256 + (int)(rng() % 8000);
  const hb_decode_mix mixes[] = {{0, nullptr, 0}, {32, dec.data(), 0}, {128, dec.data(), 0}, {256, dec.data(), 4096}};
  hb_profile_cell cells[20] = {};
  for (int i = 0; i < 20; ++i) cells[i].median_ms = 0.2f + 0.05f * i + 0.01f * (float)(rng() % 7);
  hb_latency_model m;
  if (hb_fit_latency_model(&cfg, chunks, 5, mixes, 4, cells, &m) != HB_OK) return 12;
  std::vector<double> dl(256);
  for (int t = 0; t < 200; ++t) {
    const int n = (int)(rng() % 257);
    for (int i = 0; i < n; ++i) dl[i] = 100.0 + 0.1 + (double)(rng() % 2000) / 1000.0;
    int32_t chunk = -1;
    double ms = 0;
    const double margin = (double)(rng() % 30) / 100.0;
    if (hb_select_chunk(&m, &cfg, dec.data(), dl.data(), n, 100.0, (int)(rng() % 9000), (int)(rng() % 5000),
                        1 + (int)(rng() % 64), margin, &chunk, &ms) != HB_OK)
      return 13;
    double pred = 0;
    if (hb_predict_latency(&m, &cfg, nullptr, 0, &pred) != HB_OK) return 14;
  }
  // malformed model inputs are rejected, not read past
  if (hb_fit_latency_model(&cfg, chunks, 1, mixes, 1, cells, &m) == HB_OK) return 15;
  std::printf("ok %d rejected %d\n", ok, rejected);
  return (ok > 50 && rejected > 50) ? 0 : 16;
}
