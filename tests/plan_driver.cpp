// Test driver for the host planner: reads a batch from stdin, prints the plan.
// Input: "H nq nkv hd F cu R split_item" then R lines "chunk ctx nblocks id..."
// (split_item 0: the planner's own choice).
#include <cstdio>
#include <vector>

#include "hb_plan.h"

int main() {
  int H, nq, nkv, hd, F, cu, R, split_item;
  if (scanf("%d %d %d %d %d %d %d %d", &H, &nq, &nkv, &hd, &F, &cu, &R, &split_item) != 8) return 2;
  std::vector<hb_request> reqs(R);
  std::vector<std::vector<int32_t>> tables(R);
  int T = 0;
  for (int r = 0; r < R; ++r) {
    int c, x, n;
    if (scanf("%d %d %d", &c, &x, &n) != 3) return 2;
    tables[r].resize(n);
    for (int i = 0; i < n; ++i)
      if (scanf("%d", &tables[r][i]) != 1) return 2;
    reqs[r] = {c, x, tables[r].data(), n};
    T += c;
  }
  hb_layer_config cfg{H, nq, nkv, hd, F, 16, 5e5f, 1e-5f, T > 0 ? T : 1, R > 0 ? R : 1};
  hb::Dims d;
  if (hb::check_config(&cfg, &d) != HB_OK) return 3;
  hb_batch_desc desc{R, reqs.data(), (void*)0x1000, (void*)0x80000000, HB_OUT_F32};
  if (hb::check_batch(d, 1 << 30, &desc, nullptr) != HB_OK) return 4;
  hb::Plan p;
  hb::PlanOptions opt;
  opt.split_item = split_item;
  hb::build_plan(d, &desc, cu, &p, opt);
  const int32_t* m = p.meta.data();
  printf("T %d %d %d %d\n", p.T, p.split_tile, p.split_item, p.n_slots);
  printf("geom %d %d\n", hb::kTileCols, hb::kItemsPerUnit);
  auto dump = [&](const char* tag, int off, int n) {
    for (int i = 0; i < n; ++i) {
      printf("%s", tag);
      for (int j = 0; j < 8; ++j) printf(" %d", m[off + 8 * i + j]);
      printf("\n");
    }
  };
  dump("tile", p.off_tiles, p.n_tiles);
  dump("item", p.off_items, p.n_items);
  dump("group", p.off_groups, p.n_groups);
  for (int i = 0; i < p.n_units; ++i) printf("unit %d\n", m[p.off_units + i]);
  for (int i = 0; i < p.n_merge_units; ++i) printf("merge %d\n", m[p.off_merge + i]);
  for (int t = 0; t < p.T; ++t) printf("tok %d %d\n", m[p.off_tok_pos + t], m[p.off_tok_req + t]);
  for (int r = 0; r < p.R; ++r) printf("reqbt %d\n", m[p.off_req_bt + r]);
  int offs[] = {p.off_tok_pos, p.off_tok_req, p.off_req_bt, p.off_bt, p.off_tiles, p.off_items, p.off_units, p.off_groups, p.off_merge};
  for (int o : offs) printf("off %d\n", o);
  return 0;
}
