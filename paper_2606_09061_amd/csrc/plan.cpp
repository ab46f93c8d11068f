// Varlen tile planner (host).  See plan.hpp.
#include "plan.hpp"

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <numeric>
#include <unordered_set>

namespace cpattn {

namespace {

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool is_pow2_in(int v, int lo, int hi) {
  if (v < lo || v > hi) return false;
  return (v & (v - 1)) == 0;
}

// Merge items of at most one workgroup's worth of rows (256 threads, each
// combining 4 features of one row).
void add_merge(Plan& p, int32_t tok0, int32_t n_tok, int32_t kvh, int32_t ns, int32_t part0, int G,
               int D) {
  const int32_t rows = n_tok * G;
  const int32_t per = 256 / (D / 4);
  for (int32_t r0 = 0; r0 < rows; r0 += per) {
    MergeGroup g{tok0, n_tok, kvh, ns, part0, r0, std::min(per, rows - r0), 0};
    p.merge.push_back(g);
  }
}

// Orders prefill items so that items sharing a K/V range run on one XCD
// (workgroup i is dispatched to XCD i mod num_xcds) and each XCD runs its
// items longest first.  Groups are dealt to the least-loaded XCD, largest
// group first; missing slots of shorter XCD lists become empty items.
template <class T>
void order_for_xcds(std::vector<T>& pf, int num_xcds, std::vector<PrefillItem>& out) {
  out.clear();
  if (pf.empty()) return;
  const int X = std::max(1, num_xcds);
  std::stable_sort(pf.begin(), pf.end(), [](const T& a, const T& b) {
    return a.group < b.group;
  });
  struct Grp {
    size_t b, e;
    int64_t cost;
  };
  std::vector<Grp> groups;
  for (size_t i = 0; i < pf.size();) {
    size_t j = i;
    int64_t c = 0;
    while (j < pf.size() && pf[j].group == pf[i].group) c += pf[j++].cost;
    groups.push_back({i, j, c});
    i = j;
  }
  std::stable_sort(groups.begin(), groups.end(),
                   [](const Grp& a, const Grp& b) { return a.cost > b.cost; });
  std::vector<int64_t> load(X, 0);
  std::vector<std::vector<const T*>> lists(X);
  for (const Grp& g : groups) {
    const int x = (int)(std::min_element(load.begin(), load.end()) - load.begin());
    load[x] += g.cost;
    for (size_t i = g.b; i < g.e; ++i) lists[x].push_back(&pf[i]);
  }
  size_t longest = 0;
  for (auto& l : lists) {
    std::stable_sort(l.begin(), l.end(), [](const T* a, const T* b) { return a->cost > b->cost; });
    longest = std::max(longest, l.size());
  }
  PrefillItem empty{};
  empty.n_tok = 0;
  empty.part = -1;
  out.reserve(longest * X);
  for (size_t k = 0; k < longest; ++k)
    for (int x = 0; x < X; ++x) out.push_back(k < lists[x].size() ? lists[x][k]->it : empty);
  // drop trailing empty items
  while (!out.empty() && out.back().n_tok == 0) out.pop_back();
}

}  // namespace

int validate(const cp_attn_desc* d, const cp_row_meta* rows, int32_t n_rows) {
  if (!d || n_rows < 0 || (n_rows > 0 && !rows)) return CP_ERR_INVALID_ARG;
  if (d->num_q_heads <= 0 || d->num_kv_heads <= 0 || d->head_dim <= 0 || d->block_size <= 0 ||
      d->num_blocks <= 0 || d->max_blocks_per_req <= 0 || d->num_reqs_in_table <= 0)
    return CP_ERR_INVALID_ARG;
  if (d->num_q_heads % d->num_kv_heads != 0) return CP_ERR_BAD_META;
  if (!std::isfinite(d->sm_scale) || !(d->sm_scale > 0.f)) return CP_ERR_BAD_META;
  if (d->head_dim != 64 && d->head_dim != 128) return CP_ERR_UNSUPPORTED;
  if (d->block_size != 16 && d->block_size != 32) return CP_ERR_UNSUPPORTED;
  if (!is_pow2_in(d->num_q_heads / d->num_kv_heads, 1, 8)) return CP_ERR_UNSUPPORTED;
  // request ids are packed into 24 bits of an append item
  if (d->num_reqs_in_table > (1 << 23)) return CP_ERR_UNSUPPORTED;
  const int64_t cap = (int64_t)d->max_blocks_per_req * d->block_size;
  if (cap > (int64_t)INT32_MAX) return CP_ERR_UNSUPPORTED;
  int64_t total = 0;
  std::unordered_set<int32_t> seen;
  seen.reserve((size_t)n_rows * 2);
  for (int32_t r = 0; r < n_rows; ++r) {
    const cp_row_meta& m = rows[r];
    if (m.chunk_len < 0 || m.chunk_start < 0) return CP_ERR_BAD_META;
    if ((int64_t)m.chunk_start + m.chunk_len != (int64_t)m.ctx_len) return CP_ERR_BAD_META;
    if ((int64_t)m.ctx_len > cap) return CP_ERR_BAD_META;
    if (m.req_id < 0 || m.req_id >= d->num_reqs_in_table) return CP_ERR_BAD_META;
    if (!seen.insert(m.req_id).second) return CP_ERR_BAD_META;
    total += m.chunk_len;
  }
  // token indices and q/out element offsets must fit the kernels' index types
  if (total > (int64_t)INT32_MAX / 2) return CP_ERR_UNSUPPORTED;
  return CP_OK;
}

Tuning tuning_from_env(int num_cus) {
  Tuning t;
  t.num_cus = num_cus > 0 ? num_cus : 256;
  if (const char* s = std::getenv("CP_PREFILL_MIN_LEN")) t.prefill_min_len = std::max(2, atoi(s));
  if (const char* s = std::getenv("CP_DECODE_TARGET_ITEMS")) t.decode_target_items = atoi(s);
  if (const char* s = std::getenv("CP_PREFILL_TARGET_ITEMS")) t.prefill_target_items = atoi(s);
  if (const char* s = std::getenv("CP_PREFILL_MIN_SPLIT")) t.prefill_min_split = std::max(1, atoi(s));
  if (const char* s = std::getenv("CP_NUM_XCDS")) t.num_xcds = std::max(1, atoi(s));
  return t;
}

void build_plan(const cp_attn_desc& d, const cp_row_meta* rows, int32_t n_rows, const Tuning& t,
                Plan& p) {
  p = Plan();
  const int G = d.num_q_heads / d.num_kv_heads;
  const int Hkv = d.num_kv_heads;
  const int B = d.block_size;
  const int tile_tok = kPrefillRows / G;

  // token offsets in row order
  std::vector<int64_t> off((size_t)n_rows + 1, 0);
  for (int32_t r = 0; r < n_rows; ++r) off[r + 1] = off[r] + rows[r].chunk_len;

  // ---- prefill tiles --------------------------------------------------
  struct Tile {
    int32_t tok0, n_tok, pos0, req, kv_end;
    bool wide;
  };
  std::vector<Tile> tiles;
  int64_t pf_cost = 0;  // in kPrefillKeys-key steps, summed over tiles and kv heads
  for (int32_t r = 0; r < n_rows; ++r) {
    const cp_row_meta& m = rows[r];
    if (m.chunk_len < t.prefill_min_len) continue;
    const bool wide = (int64_t)m.chunk_len * G > kPrefillRows;
    const int32_t tt = wide ? kPrefillRowsWide / G : tile_tok;
    for (int32_t j = 0; j < m.chunk_len; j += tt) {
      const int32_t n = std::min<int32_t>(tt, m.chunk_len - j);
      Tile tl{(int32_t)(off[r] + j), n, m.chunk_start + j, m.req_id, m.chunk_start + j + n, wide};
      tiles.push_back(tl);
      pf_cost += ceil_div(tl.kv_end, kPrefillKeys) * Hkv * (wide ? 2 : 1);
    }
  }
  // Key ranges longer than split_keys are cut on a grid of multiples of
  // split_keys, the same grid for every tile, so the tiles of one chunk share
  // their split ranges exactly.  No cut lies past a tile's first query
  // position, so every query of a tile sees at least one key in every split.
  const int64_t pf_target =
      t.prefill_target_items > 0 ? t.prefill_target_items : (int64_t)t.num_cus * 4;
  const int64_t split_steps =
      tiles.empty() ? 1 : std::max<int64_t>(t.prefill_min_split, ceil_div(pf_cost, pf_target));
  const int64_t split_keys = split_steps * kPrefillKeys;
  struct PfTmp {
    PrefillItem it;
    int64_t cost;
    int64_t group;  // items sharing (request, kv head, key range start)
  };
  std::vector<PfTmp> pf, pfw;
  std::vector<int32_t> bounds;
  for (const Tile& tl : tiles) {
    const int64_t last_cut = (tl.pos0 / kPrefillKeys) * (int64_t)kPrefillKeys;
    bounds.assign(1, 0);
    for (int64_t c = split_keys; c <= last_cut && c < tl.kv_end; c += split_keys)
      bounds.push_back((int32_t)c);
    bounds.push_back(tl.kv_end);
    const int64_t ns = (int64_t)bounds.size() - 1;
    for (int kvh = 0; kvh < Hkv; ++kvh) {
      int32_t part0 = -1;
      if (ns > 1) {
        part0 = (int32_t)p.partial_rows;
        p.partial_rows += ns * (int64_t)tl.n_tok * G;
      }
      for (int64_t s = 0; s < ns; ++s) {
        PrefillItem it;
        it.tok0 = tl.tok0;
        it.n_tok = tl.n_tok;
        it.pos0 = tl.pos0;
        it.req = tl.req;
        it.kvh = kvh;
        it.kv_begin = bounds[s];
        it.kv_end = bounds[s + 1];
        it.part = ns > 1 ? part0 + (int32_t)(s * tl.n_tok * G) : -1;
        // group id: request, kv head and split start (split starts are grid points)
        const int64_t gid = (((int64_t)tl.req * Hkv + kvh) << 20) + bounds[s] / split_keys;
        (tl.wide ? pfw : pf).push_back({it, ceil_div(it.kv_end - it.kv_begin, kPrefillKeys), gid});
      }
      if (ns > 1) add_merge(p, tl.tok0, tl.n_tok, kvh, (int32_t)ns, part0, G, d.head_dim);
    }
  }
  order_for_xcds(pf, t.num_xcds, p.prefill);
  order_for_xcds(pfw, t.num_xcds, p.prefill_wide);

  // ---- decode ranges --------------------------------------------------
  int64_t dec_blocks = 0;
  int64_t dec_pairs = 0;
  for (int32_t r = 0; r < n_rows; ++r) {
    const cp_row_meta& m = rows[r];
    if (m.chunk_len <= 0 || m.chunk_len >= t.prefill_min_len) continue;
    dec_blocks += ceil_div(m.ctx_len, B) * Hkv;
    dec_pairs += Hkv;
  }
  if (dec_pairs > 0) {
    const int64_t target =
        t.decode_target_items > 0 ? t.decode_target_items : (int64_t)t.num_cus * 8;
    int64_t sb = ceil_div(dec_blocks, target);
    sb = std::max<int64_t>(sb, 8);
    sb = ceil_div(sb, kDecodeWaves) * kDecodeWaves;
    p.decode_split_blocks = (int32_t)sb;
    struct DcTmp {
      DecodeItem it;
      int64_t cost;
    };
    std::vector<DcTmp> dc;
    for (int32_t r = 0; r < n_rows; ++r) {
      const cp_row_meta& m = rows[r];
      if (m.chunk_len <= 0 || m.chunk_len >= t.prefill_min_len) continue;
      const int64_t nb = ceil_div(m.ctx_len, B);
      const int64_t ns = std::max<int64_t>(1, ceil_div(nb, sb));
      for (int kvh = 0; kvh < Hkv; ++kvh) {
        int32_t part0 = -1;
        if (ns > 1) {
          part0 = (int32_t)p.partial_rows;
          p.partial_rows += ns * (int64_t)G;
          add_merge(p, (int32_t)off[r], 1, kvh, (int32_t)ns, part0, G, d.head_dim);
        }
        for (int64_t s = 0; s < ns; ++s) {
          const int64_t b0 = nb * s / ns, b1 = nb * (s + 1) / ns;
          DecodeItem it;
          it.tok = (int32_t)off[r];
          it.req = m.req_id;
          it.kvh = kvh;
          it.kv_begin = (int32_t)(b0 * B);
          it.kv_end = (int32_t)std::min<int64_t>(b1 * B, m.ctx_len);
          it.part = ns > 1 ? part0 + (int32_t)(s * G) : -1;
          it.pad0 = it.pad1 = 0;
          dc.push_back({it, b1 - b0});
        }
      }
    }
    std::stable_sort(dc.begin(), dc.end(),
                     [](const DcTmp& a, const DcTmp& b) { return a.cost > b.cost; });
    p.decode.reserve(dc.size());
    for (auto& x : dc) p.decode.push_back(x.it);
  }

  // ---- workspace layout ------------------------------------------------
  size_t o = 0;
  p.off_prefill = o;
  o = align_up(o + p.prefill.size() * sizeof(PrefillItem), 256);
  p.off_prefill_wide = o;
  o = align_up(o + p.prefill_wide.size() * sizeof(PrefillItem), 256);
  p.off_decode = o;
  o = align_up(o + p.decode.size() * sizeof(DecodeItem), 256);
  p.off_merge = o;
  o = align_up(o + p.merge.size() * sizeof(MergeGroup), 256);
  p.plan_bytes = o;
  p.off_part_o = o;
  o = align_up(o + (size_t)p.partial_rows * d.head_dim * sizeof(float), 256);
  p.off_part_lse = o;
  o = align_up(o + (size_t)p.partial_rows * sizeof(float), 256);
  p.ws_bytes = std::max<size_t>(o, 256);
}

void build_append_plan(const cp_attn_desc& d, const cp_row_meta* rows, int32_t n_rows,
                       AppendPlan& p) {
  p = AppendPlan();
  const int B = d.block_size;
  int64_t tok = 0;
  for (int32_t r = 0; r < n_rows; ++r) {
    const cp_row_meta& m = rows[r];
    int32_t pos = m.chunk_start;
    const int32_t end = m.chunk_start + m.chunk_len;
    while (pos < end) {
      const int32_t blk = pos / B;
      const int32_t slot = pos % B;
      const int32_t n = std::min<int32_t>(B - slot, end - pos);
      AppendItem it{(int32_t)(tok + (pos - m.chunk_start)), n, blk, (m.req_id << 8) | slot};
      p.items.push_back(it);
      pos += n;
    }
    tok += m.chunk_len;
  }
  p.ws_bytes = align_up(std::max<size_t>(p.items.size() * sizeof(AppendItem), 1), 256);
}

}  // namespace cpattn
