// Plans random valid batches (every head shape, block size and row kind the
// library supports) under the default tuning and under random tunings, for a
// build with AddressSanitizer and UndefinedBehaviorSanitizer
// (tests/test_native_sanitizers.py).  Every plan is checked against what the
// kernels assume of it: each record and item stays inside the batch, its
// request and the workspace, the key ranges of every (token, kv head)
// partition [0, end) with the token's position below end <= ctx, and every
// decode unit placed in a prefill launch appears there exactly once.
#include "plan.hpp"
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

namespace {

int g_trial = 0;

#define CHECK(c)                                                                  \
  do {                                                                            \
    if (!(c)) {                                                                   \
      std::printf("trial %d: check failed at line %d: %s\n", g_trial, __LINE__, #c); \
      std::exit(1);                                                               \
    }                                                                             \
  } while (0)

cpattn::Tuning random_tuning(std::mt19937& g) {
  cpattn::Tuning t;
  auto pick = [&](int n) { return (int)(g() % (unsigned)n); };
  t.prefill_min_len = 2 + pick(cpattn::kMaxPrefillMinLen - 1);
  if (pick(2)) t.prefill_min_len = 2;
  const int dti[] = {0, 1, 7, 300, 100000};
  t.decode_target_items = dti[pick(5)];
  const int pti[] = {0, 1, 5, 600, 100000};
  t.prefill_target_items = pti[pick(5)];
  t.prefill_min_split = 1 + pick(16);
  const int cus[] = {256, 1, 7, 80};
  t.num_cus = cus[pick(4)];
  const int xcds[] = {8, 1, 3, 64};
  t.num_xcds = xcds[pick(4)];
  const int64_t wmr[] = {129, 1, 100000};
  t.prefill_wide_min_rows = wmr[pick(3)];
  const int64_t wmk[] = {1200, 0, 100000};
  t.prefill_wide_min_keys = wmk[pick(3)];
  t.fuse_decode = pick(5);
  const double spread[] = {1.0, 0.0, 0.3};
  t.fuse_spread = spread[pick(3)];
  const double kps[] = {64.0, 1.0, 1000.0};
  t.fuse_keys_per_step = kps[pick(3)];
  t.fuse_narrow = pick(2) != 0;
  const double upc[] = {0.75, 0.01, 4.0};
  t.fuse_units_per_cu = upc[pick(3)];
  const double fpb[] = {180.0, 0.0, 1e9};
  t.fuse_flops_per_byte = fpb[pick(3)];
  t.xcd_piece_div = pick(10);
  const double tol[] = {0.25, -1.0, 0.0, 10.0};
  t.xcd_balance_tol = tol[pick(4)];
  return t;
}

struct Range {
  int32_t kb, ke, kind;
};

void check_plan(const cp_attn_desc& d, const std::vector<cp_row_meta>& rows,
                const cpattn::Tuning& t, const cpattn::Plan& p) {
  const int Hkv = d.num_kv_heads, G = d.num_q_heads / d.num_kv_heads;
  // token -> (row, position)
  std::vector<int32_t> tok_row, tok_pos;
  for (size_t r = 0; r < rows.size(); ++r)
    for (int j = 0; j < rows[r].chunk_len; ++j) {
      tok_row.push_back((int32_t)r);
      tok_pos.push_back(rows[r].chunk_start + j);
    }
  const int64_t T = (int64_t)tok_row.size();
  std::vector<std::vector<Range>> cov((size_t)T * Hkv);
  const int64_t P = p.partial_rows;

  // ---- prefill records of both launches
  const int64_t n_units = (int64_t)p.decode.size() * Hkv;
  std::vector<int> unit_seen((size_t)n_units, 0);
  for (int w = 0; w < 2; ++w) {
    const auto& recs = w ? p.prefill_wide : p.prefill;
    const int max_tok = (w ? cpattn::kPrefillRowsWide : cpattn::kPrefillRows) / G;
    for (const auto& r : recs) {
      if (r.n_tok == 0) continue;  // idle record
      if (r.n_tok == cpattn::kDecodeBlock) {
        CHECK(p.decode_in_prefill == w + 1);
        CHECK(r.tok0 >= 0 && r.tok0 < n_units);
        ++unit_seen[(size_t)r.tok0];
        if (w == 0) {
          CHECK(r.pos0 == -1);
        } else {
          CHECK(r.pos0 >= -1 && r.pos0 < n_units);
          if (r.pos0 >= 0) ++unit_seen[(size_t)r.pos0];
        }
        continue;
      }
      CHECK(r.n_tok >= 1 && r.n_tok <= max_tok);
      CHECK(r.tok0 >= 0 && r.tok0 + r.n_tok <= T);
      CHECK(r.kvh >= 0 && r.kvh < Hkv);
      CHECK(r.req >= 0 && r.req < d.num_reqs_in_table);
      CHECK(r.kv_begin >= 0 && r.kv_begin < r.kv_end);
      CHECK(r.part == -1 || (r.part >= 0 && r.part + (int64_t)r.n_tok * G <= P));
      const cp_row_meta& m = rows[(size_t)tok_row[(size_t)r.tok0]];
      CHECK(r.req == m.req_id && r.kv_end <= m.ctx_len);
      CHECK(m.chunk_len >= t.prefill_min_len);
      for (int j = 0; j < r.n_tok; ++j) {
        const int64_t tok = r.tok0 + j;
        CHECK(tok_row[(size_t)tok] == tok_row[(size_t)r.tok0]);  // one row per tile
        CHECK(tok_pos[(size_t)tok] == r.pos0 + j);
        cov[(size_t)(tok * Hkv + r.kvh)].push_back({r.kv_begin, r.kv_end, 0});
      }
    }
  }
  if (p.decode_in_prefill != 0)
    for (int64_t u = 0; u < n_units; ++u) CHECK(unit_seen[(size_t)u] == 1);
  else
    CHECK(std::all_of(unit_seen.begin(), unit_seen.end(), [](int c) { return c == 0; }));

  // ---- decode items
  for (const auto& it : p.decode) {
    CHECK(it.tok >= 0 && it.tok < T);
    const cp_row_meta& m = rows[(size_t)tok_row[(size_t)it.tok]];
    CHECK(it.req == m.req_id);
    CHECK(it.kv_begin >= 0 && it.kv_begin < it.kv_end && it.kv_end <= m.ctx_len);
    CHECK(it.kv_begin % d.block_size == 0);
    CHECK(m.chunk_len < t.prefill_min_len);
    if (it.part >= 0)
      CHECK(it.part + (int64_t)(Hkv - 1) * it.part_kvh_stride + G <= P);
    else
      CHECK(it.part == -1);
    for (int h = 0; h < Hkv; ++h) cov[(size_t)(it.tok * Hkv + h)].push_back({it.kv_begin, it.kv_end, 1});
  }

  // ---- merge groups
  for (const auto& mg : p.merge) {
    CHECK(mg.n_split >= 2 && mg.n_tok >= 1 && mg.tok0 >= 0 && mg.tok0 + mg.n_tok <= T);
    CHECK(mg.row0 >= 0 && mg.n_rows >= 1 && mg.row0 + mg.n_rows <= mg.n_tok * G);
    CHECK(mg.part0 >= 0 &&
          mg.part0 + ((int64_t)(Hkv - 1) * mg.n_split + mg.n_split - 1) * mg.n_tok * G +
                  mg.row0 + mg.n_rows <= P);
  }

  // ---- exact coverage of every (token, kv head)
  for (int64_t tok = 0; tok < T; ++tok) {
    const cp_row_meta& m = rows[(size_t)tok_row[(size_t)tok]];
    const int32_t pos = tok_pos[(size_t)tok];
    const bool dec = m.chunk_len < t.prefill_min_len;
    for (int h = 0; h < Hkv; ++h) {
      auto& v = cov[(size_t)(tok * Hkv + h)];
      CHECK(!v.empty());
      std::sort(v.begin(), v.end(), [](const Range& a, const Range& b) { return a.kb < b.kb; });
      CHECK(v.front().kb == 0);
      for (size_t i = 0; i < v.size(); ++i) {
        CHECK(v[i].kind == (dec ? 1 : 0));
        CHECK(v[i].kb <= pos);
        if (i + 1 < v.size()) CHECK(v[i].ke == v[i + 1].kb);
      }
      const int32_t end = v.back().ke;
      CHECK(pos < end && end <= m.ctx_len);
      if (dec) CHECK(end == pos + 1);
    }
  }

  // ---- workspace layout
  CHECK(p.off_prefill == 0);
  CHECK(p.off_prefill_wide >= p.off_prefill + p.prefill.size() * sizeof(cpattn::PrefillRec));
  CHECK(p.off_decode >= p.off_prefill_wide + p.prefill_wide.size() * sizeof(cpattn::PrefillRec));
  CHECK(p.off_merge >= p.off_decode + p.decode.size() * sizeof(cpattn::DecodeItem));
  CHECK(p.plan_bytes >= p.off_merge + p.merge.size() * sizeof(cpattn::MergeGroup));
  CHECK(p.off_part_o >= p.plan_bytes);
  CHECK(p.off_part_lse >= p.off_part_o + (size_t)P * d.head_dim * sizeof(float));
  CHECK(p.ws_bytes >= p.off_part_lse + (size_t)P * sizeof(float));
}

}  // namespace

int main() {
  std::mt19937 g(7);
  cpattn::Plan p;
  cpattn::AppendPlan ap;
  long total_items = 0;
  for (int trial = 0; trial < 3000; ++trial) {
    g_trial = trial;
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
    const cpattn::Tuning t = trial % 3 == 0 ? cpattn::tuning_from_env(256) : random_tuning(g);
    cpattn::build_plan(d, rows.data(), (int32_t)rows.size(), t, p);
    check_plan(d, rows, t, p);
    cpattn::build_append_plan(d, rows.data(), (int32_t)rows.size(), ap);
    total_items += (long)(p.prefill.size() + p.prefill_wide.size() + p.decode.size()) + (long)ap.items.size();
  }
  printf("ok, %ld items planned\n", total_items);
  return 0;
}
