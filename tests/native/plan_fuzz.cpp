// Plans random valid batches (every head shape, block size and row kind the
// library supports), for a build with AddressSanitizer and
// UndefinedBehaviorSanitizer (tests/test_native_sanitizers.py).
#include "plan.hpp"
#include <algorithm>
#include <cstdio>
#include <random>
#include <vector>
int main() {
  std::mt19937 g(7);
  cpattn::Plan p;
  cpattn::AppendPlan ap;
  long total_items = 0;
  for (int trial = 0; trial < 3000; ++trial) {
    const int hkv_opts[] = {1, 2, 8}, g_opts[] = {1, 2, 4, 8}, d_opts[] = {64, 128}, b_opts[] = {16, 32};
    cp_attn_desc d{};
    d.num_kv_heads = hkv_opts[g() % 3];
    d.num_q_heads = d.num_kv_heads * g_opts[g() % 4];
    d.head_dim = d_opts[g() % 2];
    d.block_size = b_opts[g() % 2];
    d.max_blocks_per_req = 1 + g() % 200;
    const int nreq = 1 + g() % 64;
    d.num_reqs_in_table = nreq;
    d.num_blocks = nreq * d.max_blocks_per_req;
    d.sm_scale = 0.1f;
    const int cap = d.max_blocks_per_req * d.block_size;
    std::vector<cp_row_meta> rows;
    std::vector<int> perm(nreq);
    for (int i = 0; i < nreq; ++i) perm[i] = i;
    std::shuffle(perm.begin(), perm.end(), g);
    const int nrows = g() % (nreq + 1);
    for (int r = 0; r < nrows; ++r) {
      const int kind = g() % 3;
      int len = kind == 0 ? 1 : kind == 1 ? (int)(g() % 600) : (int)(g() % 8);
      len = std::min(len, cap);
      const int start = (int)(g() % (cap - len + 1));
      rows.push_back({perm[r], start, len, start + len});
    }
    if (cpattn::validate(&d, rows.data(), (int32_t)rows.size()) != CP_OK) { printf("invalid %d\n", trial); return 1; }
    const cpattn::Tuning t = cpattn::tuning_from_env(256);
    cpattn::build_plan(d, rows.data(), (int32_t)rows.size(), t, p);
    cpattn::build_append_plan(d, rows.data(), (int32_t)rows.size(), ap);
    total_items += (long)(p.prefill.size() + p.prefill_wide.size() + p.decode.size()) + (long)ap.items.size();
  }
  printf("ok, %ld items planned\n", total_items);
  return 0;
}
