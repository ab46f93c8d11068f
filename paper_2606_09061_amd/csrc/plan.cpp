// Varlen tile planner (host).  See plan.hpp.
#include "plan.hpp"

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <numeric>
#include <stdexcept>

namespace cpattn {

namespace {

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool is_pow2_in(int v, int lo, int hi) {
  if (v < lo || v > hi) return false;
  return (v & (v - 1)) == 0;
}

// Merge items of at most one workgroup's worth of rows (256 threads, each
// combining 4 features of one row); the kernel's grid covers the kv heads.
void add_merge(Plan& p, int32_t tok0, int32_t n_tok, int32_t ns, int32_t part0, int G, int D) {
  const int32_t rows = n_tok * G;
  const int32_t per = 256 / (D / 4);
  for (int32_t r0 = 0; r0 < rows; r0 += per) {
    MergeGroup g{tok0, n_tok, ns, part0, r0, std::min(per, rows - r0), 0, 0};
    p.merge.push_back(g);
  }
}

// Groups the prefill slots (item * Hkv + kv head) of one tile width by XCD
// so that slots sharing a K/V range -- the tiles of one chunk in one split,
// for one kv head -- run on one XCD (a workgroup runs on XCD w mod
// num_xcds), each XCD's slots longest first.  Groups are dealt to the
// least-loaded XCD, largest group first.  When that leaves the busiest XCD
// more than (1 + balance_tol) times the mean load -- few groups (few kv
// heads, few chunks) cannot balance eight XCDs -- every group costlier than
// 1 / (piece_div * num_xcds) of the launch is cut into runs of consecutive
// tiles of about that cost and the pieces are dealt instead; a piece's K/V
// then comes from the shared last-level cache rather than its XCD's L2.
// Result: sc.flat holds XCD 0's slots, then XCD 1's, ...; sc.xcd_len[x] how
// many.
void lists_by_xcd(bool wide, const std::vector<int64_t>& cost, int Hkv, int num_xcds,
                  int piece_div, double balance_tol, PlanScratch& sc) {
  auto& groups = sc.groups;
  groups.clear();
  const int X = std::max(1, num_xcds);
  sc.xcd_len.assign(X, 0);
  sc.flat.clear();
  int64_t max_cost = 0;
  for (int32_t c = 0; c < (int32_t)sc.chunks.size(); ++c) {
    const detail::Chunk& ch = sc.chunks[c];
    if (ch.wide != wide) continue;
    for (int32_t s = 0; s < ch.max_ns; ++s) {
      int64_t gc = 0;
      for (int32_t i = ch.tile0; i < ch.tile0 + ch.n_tiles; ++i)
        if (sc.tiles[i].ns > s) {
          gc += cost[sc.tiles[i].item0 + s];
          max_cost = std::max(max_cost, cost[sc.tiles[i].item0 + s]);
        }
      for (int32_t h = 0; h < Hkv; ++h) groups.push_back({c, h, s, gc, 0, 0, ch.n_tiles});
    }
  }
  if (groups.empty()) return;
  // longest-first dealing to the least-loaded XCD; returns the largest load
  auto deal = [&]() {
    std::stable_sort(groups.begin(), groups.end(),
                     [](const detail::Group& a, const detail::Group& b) { return a.cost > b.cost; });
    sc.load.assign(X, 0);
    for (detail::Group& g : groups) {
      g.xcd = (int32_t)(std::min_element(sc.load.begin(), sc.load.end()) - sc.load.begin());
      sc.load[g.xcd] += g.cost;
    }
    return *std::max_element(sc.load.begin(), sc.load.end());
  };
  int64_t total = 0;
  for (const detail::Group& g : groups) total += g.cost;
  const int64_t busiest = deal();
  if (piece_div > 0 && (double)busiest * X > (1.0 + balance_tol) * (double)total) {
    const int64_t piece = std::max<int64_t>(1, total / ((int64_t)piece_div * X));
    auto& pieces = sc.pieces;
    pieces.clear();
    for (const detail::Group& g : groups) {
      if (g.cost <= piece) {
        pieces.push_back(g);
        continue;
      }
      const detail::Chunk& ch = sc.chunks[g.chunk];
      int32_t a = 0;
      int64_t acc = 0;
      for (int32_t i = 0; i < ch.n_tiles; ++i) {
        const detail::Tile& tl = sc.tiles[ch.tile0 + i];
        if (tl.ns <= g.split) continue;
        acc += cost[tl.item0 + g.split];
        if (acc >= piece) {
          pieces.push_back({g.chunk, g.kvh, g.split, acc, 0, a, i + 1});
          a = i + 1;
          acc = 0;
        }
      }
      if (acc > 0) pieces.push_back({g.chunk, g.kvh, g.split, acc, 0, a, ch.n_tiles});
    }
    groups.swap(pieces);
    deal();
  }
  // Each XCD's slots, longest first, equal costs in the order their groups
  // were dealt: a counting sort keyed on (XCD, max_cost - cost).
  const int64_t K = max_cost + 1;
  auto& pos = sc.count;
  pos.assign((size_t)X * K + 1, 0);
  auto for_each_slot = [&](auto&& f) {
    for (const detail::Group& g : groups) {
      const detail::Chunk& ch = sc.chunks[g.chunk];
      for (int32_t i = ch.tile0 + g.t0; i < ch.tile0 + g.t1; ++i) {
        const detail::Tile& tl = sc.tiles[i];
        if (tl.ns <= g.split) continue;
        const int32_t item = tl.item0 + g.split;
        f((size_t)g.xcd * K + (max_cost - cost[item]), item * Hkv + g.kvh);
      }
    }
  };
  for_each_slot([&](size_t key, int32_t) { ++pos[key + 1]; });
  for (int x = 0; x < X; ++x)
    for (int64_t k = 0; k < K; ++k) sc.xcd_len[x] += pos[(size_t)x * K + k + 1];
  for (size_t k = 1; k < pos.size(); ++k) pos[k] += pos[k - 1];
  sc.flat.resize((size_t)pos.back());
  for_each_slot([&](size_t key, int32_t slot) { sc.flat[(size_t)pos[key]++] = slot; });
}

// Lays the slots out in dispatch order: workgroup i runs on XCD i mod X, so
// position k * X + x takes XCD x's k-th slot (longest first), or an idle
// record when XCD x has fewer; trailing idle records are dropped.
void interleave_by_xcd(const std::vector<detail::PrefillItem>& items, int Hkv, int num_xcds,
                       PlanScratch& sc, std::vector<PrefillRec>& recs) {
  recs.clear();
  if (sc.flat.empty()) return;
  const int X = std::max(1, num_xcds);
  int64_t longest = 0, start[64];
  for (int x = 0, acc = 0; x < X; ++x) {
    start[x] = acc;
    acc += (int)sc.xcd_len[x];
    longest = std::max(longest, sc.xcd_len[x]);
  }
  recs.reserve((size_t)(longest * X));
  for (int64_t k = 0; k < longest; ++k)
    for (int x = 0; x < X; ++x) {
      PrefillRec r{0, 0, 0, 0, 0, 0, -1, 0};
      if (k < sc.xcd_len[x]) {
        const int32_t slot = sc.flat[(size_t)(start[x] + k)];
        const detail::PrefillItem& it = items[(size_t)(slot / Hkv)];
        const int32_t kvh = slot % Hkv;
        r = PrefillRec{it.tok0, it.n_tok, it.pos0, it.req, it.kv_begin, it.kv_end,
                       it.part < 0 ? -1 : it.part + kvh * it.part_kvh_stride, kvh};
      }
      recs.push_back(r);
    }
  while (!recs.empty() && recs.back().n_tok == 0) recs.pop_back();
}

// Adds the decode blocks (n_units units, per_block per workgroup) to a prefill
// record list.  mode 1 appends them after the tiles; modes 2 (before the
// tiles), 3 (spread evenly over the first `spread` fraction of them, the
// longest units first) and 4 (rows of decode blocks and rows of tiles merged
// longest first, a decode unit of k keys costing k / keys_per_step tile
// steps) insert whole rows of X records, so every tile keeps its position
// mod X, i.e. its XCD.  Decode blocks dispatched among tiles stream K/V from
// HBM while the tiles around them keep the matrix cores busy.
void place_decode_blocks(std::vector<PrefillRec>& recs, const std::vector<DecodeItem>& dec,
                         int Hkv, bool wide, const Tuning& t, PlanScratch& sc) {
  const int per_block = wide ? 2 : 1;
  const int64_t n_units = (int64_t)dec.size() * Hkv;
  const int64_t X = std::max(1, t.num_xcds);
  const int64_t n_blk = ceil_div(n_units, per_block);
  const PrefillRec idle{0, 0, 0, 0, 0, 0, -1, 0};
  auto marker = [&](int64_t b) {
    const int64_t u0 = b * per_block;
    const int64_t u1 = per_block > 1 && u0 + 1 < n_units ? u0 + 1 : -1;
    return PrefillRec{(int32_t)u0, kDecodeBlock, (int32_t)u1, 0, 0, 0, -1, 0};
  };
  if (t.fuse_decode == 1) {
    for (int64_t b = 0; b < n_blk; ++b) recs.push_back(marker(b));
    return;
  }
  auto& old = sc.recs_tmp;
  old.swap(recs);
  recs.clear();
  const int64_t R = ceil_div((int64_t)old.size(), X), M = ceil_div(n_blk, X);
  // mode 3: marker rows spread over the first R3 tile rows
  const double spread = std::min(1.0, std::max(0.0, t.fuse_spread));
  const int64_t R3 = std::max<int64_t>(1, (int64_t)std::ceil(spread * (double)R));
  // mode 4: row costs in tile steps (a row's first record is its longest)
  auto tile_row_cost = [&](int64_t r) {
    const PrefillRec& q = old[(size_t)(r * X)];
    return (double)ceil_div(q.kv_end - q.kv_begin, kPrefillKeys) * (wide ? 2.0 : 1.0);
  };
  auto dec_row_cost = [&](int64_t m) {
    const DecodeItem& it = dec[(size_t)(m * X * per_block / Hkv)];
    return (double)(it.kv_end - it.kv_begin) / std::max(1.0, t.fuse_keys_per_step);
  };
  int64_t pi = 0, mi = 0;
  while (pi < R || mi < M) {
    bool take_m = false;
    if (mi < M) {
      if (pi >= R || t.fuse_decode == 2) take_m = true;
      else if (t.fuse_decode == 3)  // midpoints as fractions of their spans
        take_m = pi >= R3 || (2 * mi + 1) * R3 <= (2 * pi + 1) * M;
      else
        take_m = dec_row_cost(mi) > tile_row_cost(pi);
    }
    for (int64_t x = 0; x < X; ++x) {
      if (take_m) {
        const int64_t b = mi * X + x;
        recs.push_back(b < n_blk ? marker(b) : idle);
      } else {
        const int64_t k = pi * X + x;
        recs.push_back(k < (int64_t)old.size() ? old[(size_t)k] : idle);
      }
    }
    (take_m ? mi : pi) += 1;
  }
  while (!recs.empty() && recs.back().n_tok == 0) recs.pop_back();
}

// Makespan, in steps, of longest-first list scheduling of `groups` (cost,
// count) on `slots` identical slots.  Slot loads are kept as a histogram
// (load, slots) sorted by load, so equal items are placed in bulk.
int64_t lpt_makespan(std::vector<std::pair<int64_t, int64_t>>& groups, int64_t slots,
                     std::vector<std::pair<int64_t, int64_t>>& load) {
  if (groups.empty()) return 0;
  std::sort(groups.begin(), groups.end(),
            [](const std::pair<int64_t, int64_t>& a, const std::pair<int64_t, int64_t>& b) {
              return a.first > b.first;
            });
  load.assign(1, {0, slots});
  size_t head = 0;  // load[head] is the least-loaded bucket; earlier ones are empty
  for (const auto& g : groups) {
    int64_t k = g.second;
    if (head + 1 == load.size() && k >= slots) {  // all slots level: whole rounds at once
      load[head].first += (k / slots) * g.first;
      k %= slots;
    }
    while (k > 0) {
      const int64_t l = load[head].first, take = std::min(k, load[head].second);
      if ((load[head].second -= take) == 0) ++head;
      // insert `take` slots at load l + g.first, keeping the order
      const int64_t nl = l + g.first;
      auto pos = std::lower_bound(
          load.begin() + head, load.end(), nl,
          [](const std::pair<int64_t, int64_t>& a, int64_t v) { return a.first < v; });
      if (pos != load.end() && pos->first == nl)
        pos->second += take;
      else
        load.insert(pos, {nl, take});
      k -= take;
    }
  }
  return load.back().first;
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
  int32_t r = 0;
  for (; r < n_rows; ++r) {
    const cp_row_meta& m = rows[r];
    if (m.chunk_len < 0 || m.chunk_start < 0) break;
    if ((int64_t)m.chunk_start + m.chunk_len != (int64_t)m.ctx_len) break;
    if ((int64_t)m.ctx_len > cap) break;
    if (m.req_id < 0 || m.req_id >= d->num_reqs_in_table) break;
    total += m.chunk_len;
  }
  if (r < n_rows) return CP_ERR_BAD_META;
  // duplicate request ids: one bit per block-table row, cleared again after
  thread_local std::vector<uint64_t> seen;
  const size_t words = ((size_t)d->num_reqs_in_table + 63) / 64;
  if (seen.size() < words) seen.resize(words, 0);
  bool dup = false;
  int32_t marked = 0;
  for (; marked < n_rows; ++marked) {
    const uint32_t id = (uint32_t)rows[marked].req_id;
    const uint64_t bit = 1ull << (id & 63);
    if (seen[id >> 6] & bit) {
      dup = true;
      break;
    }
    seen[id >> 6] |= bit;
  }
  for (int32_t i = 0; i < marked; ++i) seen[(uint32_t)rows[i].req_id >> 6] = 0;
  if (dup) return CP_ERR_BAD_META;
  // token indices and q/out element offsets must fit the kernels' index types
  if (total > (int64_t)INT32_MAX / 2) return CP_ERR_UNSUPPORTED;
  return CP_OK;
}

Tuning tuning_from_env(int num_cus) {
  Tuning t;
  t.num_cus = num_cus > 0 ? num_cus : 256;
  // Rows shorter than this run on the decode kernel, token by token (any
  // value >= 2 is exact; 2 sends every multi-token chunk to the MFMA kernel).
  if (const char* s = std::getenv("CP_PREFILL_MIN_LEN"))
    t.prefill_min_len = std::min(kMaxPrefillMinLen, std::max(2, atoi(s)));
  if (const char* s = std::getenv("CP_DECODE_TARGET_ITEMS")) t.decode_target_items = atoi(s);
  if (const char* s = std::getenv("CP_PREFILL_TARGET_ITEMS")) t.prefill_target_items = atoi(s);
  if (const char* s = std::getenv("CP_PREFILL_MIN_SPLIT")) t.prefill_min_split = std::max(1, atoi(s));
  if (const char* s = std::getenv("CP_FUSE_DECODE")) t.fuse_decode = std::min(4, std::max(0, atoi(s)));
  if (const char* s = std::getenv("CP_FUSE_SPREAD")) t.fuse_spread = atof(s);
  if (const char* s = std::getenv("CP_FUSE_KEYS_PER_STEP")) t.fuse_keys_per_step = atof(s);
  if (const char* s = std::getenv("CP_FUSE_NARROW")) t.fuse_narrow = atoi(s) != 0;
  if (const char* s = std::getenv("CP_FUSE_UNITS_PER_CU")) t.fuse_units_per_cu = atof(s);
  if (const char* s = std::getenv("CP_FUSE_FLOPS_PER_BYTE")) t.fuse_flops_per_byte = atof(s);
  if (const char* s = std::getenv("CP_NUM_XCDS")) t.num_xcds = std::min(64, std::max(1, atoi(s)));
  if (const char* s = std::getenv("CP_XCD_PIECE_DIV")) t.xcd_piece_div = std::max(0, atoi(s));
  if (const char* s = std::getenv("CP_XCD_BALANCE_TOL")) t.xcd_balance_tol = std::max(-1.0, atof(s));
  if (const char* s = std::getenv("CP_PREFILL_WIDE_MIN_ROWS"))
    t.prefill_wide_min_rows = std::max<int64_t>(1, atoll(s));
  if (const char* s = std::getenv("CP_PREFILL_WIDE_MIN_KEYS"))
    t.prefill_wide_min_keys = std::max<int64_t>(0, atoll(s));
  return t;
}

// Split length, in steps, for the prefill tiles.  Candidates are a 2^(1/8)
// grid from prefill_min_split up to the longest tile, plus the lengths that
// cut the longest tile into k equal parts; each is scored by the estimated
// run time of the two prefill launches -- wide tiles one workgroup per CU,
// 128-row tiles two -- under longest-first placement, plus the merge traffic
// its partial rows cause, and the best wins.  A tile's splits are all
// split_steps long except its last, so a candidate reduces to a few
// (cost, count) groups.  prefill_target_items > 0 instead fixes the split at
// the work of one slot when the total is spread over that many slots.
static int64_t choose_split_steps(const cp_attn_desc& d, const Tuning& t,
                                  const std::vector<detail::Tile>& tiles, PlanScratch& sc) {
  const int Hkv = d.num_kv_heads;
  const int G = d.num_q_heads / d.num_kv_heads;
  int64_t max_steps = 1;
  bool has[2] = {false, false};  // narrow, wide tiles present
  for (const detail::Tile& tl : tiles) {
    max_steps = std::max<int64_t>(max_steps, ceil_div(tl.kv_end, kPrefillKeys));
    has[tl.wide ? 1 : 0] = true;
  }
  // decode units that join the last prefill launch (sc.dec_groups, in tile
  // steps): they fill its slots too, so they weigh in the estimate
  const int wdec = has[0] ? 0 : 1;
  int64_t dec_total = 0, dec_longest = 0;
  for (const auto& g : sc.dec_groups) {
    dec_total += g.first * g.second;
    dec_longest = std::max(dec_longest, g.first);
  }
  const int64_t min_split = std::max(1, t.prefill_min_split);
  if (t.prefill_target_items > 0) {
    int64_t cost = 0;
    for (const detail::Tile& tl : tiles)
      cost += ceil_div(tl.kv_end, kPrefillKeys) * Hkv * (tl.wide ? 2 : 1);
    return std::max(min_split, ceil_div(cost, t.prefill_target_items));
  }
  auto& cand = sc.candidates;
  cand.clear();
  for (double sf = (double)min_split; sf < (double)max_steps; sf *= 1.09050773)
    cand.push_back((int64_t)sf);
  for (int64_t k = 1; k <= 32; ++k) {
    const int64_t c = ceil_div(max_steps, k);
    if (c < min_split) break;
    cand.push_back(c);
  }
  cand.push_back(max_steps);
  std::sort(cand.begin(), cand.end());
  cand.erase(std::unique(cand.begin(), cand.end()), cand.end());
  constexpr int64_t kItemOverhead = 2;  // steps: query load, first gather, output
  // merge: one step of a wide tile is ~2 us at the kernel's rate, in which
  // HBM moves ~10 MB; a partial row is written and read once, (D + 1) fp32
  const double merge_bytes_per_step = 10.0e6 * d.head_dim / 128.0;
  // Each candidate reduces to (cost, count) groups per tile width: a tile's
  // splits are all S steps long except its last.  The unsplit grid goes
  // first; a candidate whose lower bound -- per width, the larger of the
  // longest item and the average slot load, plus its merge traffic --
  // cannot beat the best estimate so far is not simulated.
  // cuts of a tile are the multiples of split_keys in (0, cut_lim], with
  // cut_lim = min(its first query's step start, kv_end - 1)
  auto& cut_lim = sc.cut_lim;
  cut_lim.resize(tiles.size());
  for (size_t i = 0; i < tiles.size(); ++i)
    cut_lim[i] = (uint32_t)std::min<int64_t>((tiles[i].pos0 / kPrefillKeys) * (int64_t)kPrefillKeys,
                                             tiles[i].kv_end - 1);
  auto cuts_of = [&](size_t i, uint32_t split_keys) -> int64_t {
    return cut_lim[i] < split_keys ? 0 : cut_lim[i] / split_keys;
  };
  auto evaluate = [&](int64_t S, double best) -> double {
    const int64_t split_keys = S * kPrefillKeys;
    const uint32_t sk32 = (uint32_t)std::min<int64_t>(split_keys, UINT32_MAX);
    auto& groups = sc.groups2;
    double lb = 0.0;
    int64_t partial_rows = 0;
    int64_t total[2] = {0, 0}, longest[2] = {0, 0}, full[2] = {0, 0};
    for (size_t i = 0; i < tiles.size(); ++i) {
      const detail::Tile& tl = tiles[i];
      const int w = tl.wide ? 1 : 0;
      const int64_t cuts = cuts_of(i, sk32);
      const int64_t tail = ceil_div(tl.kv_end - cuts * split_keys, kPrefillKeys) + kItemOverhead;
      full[w] += cuts;
      total[w] += (tail + cuts * (S + kItemOverhead)) * Hkv;
      longest[w] = std::max(longest[w], cuts > 0 ? std::max(tail, S + kItemOverhead) : tail);
      if (cuts > 0) partial_rows += Hkv * (1 + cuts) * tl.n_tok * G;
    }
    const double merge = (double)partial_rows * (d.head_dim + 1) * 8 / merge_bytes_per_step;
    total[wdec] += dec_total;
    longest[wdec] = std::max(longest[wdec], dec_longest);
    for (int w = 0; w < 2; ++w) {
      if (!has[w]) continue;
      const int64_t slots = (int64_t)t.num_cus * (w ? 1 : 2);
      lb += (double)std::max(longest[w], ceil_div(total[w], slots));
    }
    if (best >= 0 && lb + merge > best) return -1.0;  // cannot win (ties still can)
    double est = merge;
    for (int w = 0; w < 2; ++w) {
      if (!has[w]) continue;
      groups.clear();
      for (size_t i = 0; i < tiles.size(); ++i) {
        const detail::Tile& tl = tiles[i];
        if ((int)tl.wide != w) continue;
        const int64_t cuts = cuts_of(i, sk32);
        groups.push_back({ceil_div(tl.kv_end - cuts * split_keys, kPrefillKeys) + kItemOverhead, Hkv});
      }
      if (full[w] > 0) groups.push_back({S + kItemOverhead, full[w] * Hkv});
      if (w == wdec) groups.insert(groups.end(), sc.dec_groups.begin(), sc.dec_groups.end());
      const int64_t slots = (int64_t)t.num_cus * (w ? 1 : 2);
      est += (double)lpt_makespan(groups, slots, sc.load_hist);
    }
    return est;
  };
  // the smallest S among those with the least estimate (candidates ascend)
  int64_t best_s = max_steps;
  double best = evaluate(max_steps, -1.0);
  for (const int64_t S : cand) {
    if (S == max_steps) break;
    const double est = evaluate(S, best);
    if (est >= 0 && (est < best || (est == best && best_s == max_steps))) {
      best = est;
      best_s = S;
    }
  }
  return best_s;
}

void build_plan(const cp_attn_desc& d, const cp_row_meta* rows, int32_t n_rows, const Tuning& t,
                Plan& p) {
  PlanScratch& sc = p.scratch;
  p.prefill.clear();
  p.prefill_wide.clear();
  p.decode.clear();
  p.merge.clear();
  p.partial_rows = 0;
  p.decode_split_blocks = 0;
  const int G = d.num_q_heads / d.num_kv_heads;
  const int Hkv = d.num_kv_heads;
  const int B = d.block_size;
  const int tile_tok = kPrefillRows / G;

  // token offsets in row order
  auto& off = sc.off;
  off.assign((size_t)n_rows + 1, 0);
  for (int32_t r = 0; r < n_rows; ++r) off[r + 1] = off[r] + rows[r].chunk_len;

  // ---- prefill tiles --------------------------------------------------
  auto& tiles = sc.tiles;
  auto& chunks = sc.chunks;
  tiles.clear();
  chunks.clear();
  // 256-row tiles halve the K/V reads per flop but leave a CU one workgroup,
  // whose start-up and drain nothing overlaps: they pay only when the step's
  // queries see long key ranges (token-weighted mean of chunk_start + len / 2).
  // The choice is per step, so that all prefill tiles share one launch.
  // When the step's decode rows run inside the prefill launch, 128-row tiles
  // leave each CU a second workgroup slot, which a decode block can take
  // beside a tile (measured: the prefill-heavy 2k-token mix runs 6 % faster
  // fused on 128-row tiles than fused on 256-row ones).
  double pf_tok = 0, pf_keys = 0;
  bool has_decode = false;
  for (int32_t r = 0; r < n_rows; ++r) {
    const cp_row_meta& m = rows[r];
    if (m.chunk_len > 0 && m.chunk_len < t.prefill_min_len) has_decode = true;
    if (m.chunk_len < t.prefill_min_len) continue;
    pf_tok += m.chunk_len;
    pf_keys += (double)m.chunk_len * ((double)m.chunk_start + 0.5 * m.chunk_len);
  }
  const bool fused = t.fuse_decode > 0 && has_decode && pf_tok > 0;
  const bool long_keys = !(fused && t.fuse_narrow) && pf_tok > 0 &&
                         pf_keys >= (double)t.prefill_wide_min_keys * pf_tok;
  for (int32_t r = 0; r < n_rows; ++r) {
    const cp_row_meta& m = rows[r];
    if (m.chunk_len < t.prefill_min_len) continue;
    const bool wide = long_keys && (int64_t)m.chunk_len * G >= t.prefill_wide_min_rows;
    const int32_t tt = wide ? kPrefillRowsWide / G : tile_tok;
    detail::Chunk ch{(int32_t)tiles.size(), 0, 0, wide};
    for (int32_t j = 0; j < m.chunk_len; j += tt) {
      const int32_t n = std::min<int32_t>(tt, m.chunk_len - j);
      detail::Tile tl{(int32_t)(off[r] + j), n, m.chunk_start + j, m.req_id,
                      m.chunk_start + j + n, wide, 0, 0};
      tiles.push_back(tl);
      ++ch.n_tiles;
    }
    chunks.push_back(ch);
  }
  // ---- decode sizing ----------------------------------------------------
  // Rows shorter than prefill_min_len run on the split-K decode kernel, one
  // item list per query token: token j of a row sits at position
  // chunk_start + j and sees keys [0, chunk_start + j + 1), so each token is
  // its own "decode row" with its own causal limit (a one-token row is the
  // usual case; few-token chunks read their request's K/V once per token).
  auto each_decode_token = [&](auto&& f) {
    for (int32_t r = 0; r < n_rows; ++r) {
      const cp_row_meta& m = rows[r];
      if (m.chunk_len <= 0 || m.chunk_len >= t.prefill_min_len) continue;
      for (int32_t j = 0; j < m.chunk_len; ++j)
        f(m, (int32_t)(off[r] + j), m.chunk_start + j + 1);
    }
  };
  sc.dec_groups.clear();
  int64_t dec_blocks = 0;
  each_decode_token([&](const cp_row_meta&, int32_t, int32_t kv_end) {
    dec_blocks += ceil_div(kv_end, B) * Hkv;
  });
  if (dec_blocks > 0) {
    // Items per CU grow with the decode bytes: ~3 per CU (the kernel keeps
    // three workgroups resident) for small loads, where every extra item costs
    // plan upload, partial rows for the merge and a workgroup's start-up,
    // rising to 6 per CU at 4 GB and above, where finer items balance the
    // tail better (measured on the 0.1, 0.8, 1.8 and 5.5 GB mixes).
    const double dec_bytes = (double)dec_blocks * B * d.head_dim * 4.0;
    double per_cu = 3.0 + 3.0 * std::min(1.0, dec_bytes / 4.0e9);
    // Inside a prefill-dominated launch, longer decode ranges: each unit
    // streams beside the tiles for much of the launch.  Only rows longer than
    // the cut are split, so this sets the longest unit (measured best at
    // 0.5-1 ranges per CU on the 2k-token prefill-heavy mix and the 70B
    // replay, with a cliff below 0.5 where whole long rows outlast the tiles;
    // decode-dominated steps keep the rule above).
    const double pf_flops = 4.0 * d.head_dim * d.num_q_heads * pf_keys;
    if (fused && pf_flops > t.fuse_flops_per_byte * dec_bytes) per_cu = t.fuse_units_per_cu;
    const int64_t target = t.decode_target_items > 0
                               ? t.decode_target_items
                               : std::max<int64_t>(1, (int64_t)(t.num_cus * per_cu));
    int64_t sb = ceil_div(dec_blocks, target);
    sb = std::max<int64_t>(sb, 8);
    sb = ceil_div(sb, kDecodeWaves) * kDecodeWaves;
    p.decode_split_blocks = (int32_t)sb;
    // with the decode rows inside the prefill launch, their units (in tile
    // steps) join the split estimate of that launch
    if (fused) {
      auto& hist = sc.dec_hist;
      hist.assign((size_t)sb + 2, 0);
      each_decode_token([&](const cp_row_meta&, int32_t, int32_t kv_end) {
        const int64_t nb = ceil_div(kv_end, B);
        const int64_t ns = std::max<int64_t>(1, ceil_div(nb, sb));
        for (int64_t s = 0; s < ns; ++s) ++hist[nb * (s + 1) / ns - nb * s / ns];
      });
      for (int64_t b = 1; b < (int64_t)hist.size(); ++b)
        if (hist[b] > 0)
          sc.dec_groups.push_back(
              {(int64_t)std::ceil((double)(b * B) / std::max(1.0, t.fuse_keys_per_step)) + 1,
               hist[b] * Hkv});
    }
  }

  // Key ranges longer than split_keys are cut on a grid of multiples of
  // split_keys, the same grid for every tile, so the tiles of one chunk share
  // their split ranges exactly.  No cut lies past a tile's first query
  // position, so every query of a tile sees at least one key in every split.
  const int64_t split_steps = tiles.empty() ? 1 : choose_split_steps(d, t, tiles, sc);
  const int64_t split_keys = split_steps * kPrefillKeys;
  auto& bounds = sc.bounds;
  sc.item_cost[0].clear();
  sc.item_cost[1].clear();
  sc.items[0].clear();
  sc.items[1].clear();
  for (detail::Chunk& ch : chunks) {
    auto& items = sc.items[ch.wide ? 1 : 0];
    auto& cost = sc.item_cost[ch.wide ? 1 : 0];
    for (int32_t i = ch.tile0; i < ch.tile0 + ch.n_tiles; ++i) {
      detail::Tile& tl = tiles[i];
      const int64_t last_cut = (tl.pos0 / kPrefillKeys) * (int64_t)kPrefillKeys;
      bounds.assign(1, 0);
      for (int64_t c = split_keys; c <= last_cut && c < tl.kv_end; c += split_keys)
        bounds.push_back((int32_t)c);
      bounds.push_back(tl.kv_end);
      const int32_t ns = (int32_t)bounds.size() - 1;
      const int32_t stride = ns * tl.n_tok * G;  // partial rows per kv head
      int32_t part0 = -1;
      if (ns > 1) {
        part0 = (int32_t)p.partial_rows;
        p.partial_rows += (int64_t)Hkv * stride;
        add_merge(p, tl.tok0, tl.n_tok, ns, part0, G, d.head_dim);
      }
      tl.item0 = (int32_t)items.size();
      tl.ns = ns;
      ch.max_ns = std::max(ch.max_ns, ns);
      for (int32_t s = 0; s < ns; ++s) {
        detail::PrefillItem it;
        it.tok0 = tl.tok0;
        it.n_tok = tl.n_tok;
        it.pos0 = tl.pos0;
        it.req = tl.req;
        it.kv_begin = bounds[s];
        it.kv_end = bounds[s + 1];
        it.part = ns > 1 ? part0 + s * tl.n_tok * G : -1;
        it.part_kvh_stride = ns > 1 ? stride : 0;
        items.push_back(it);
        cost.push_back(ceil_div(it.kv_end - it.kv_begin, kPrefillKeys));
      }
    }
  }
  if ((int64_t)std::max(sc.items[0].size(), sc.items[1].size()) * Hkv > INT32_MAX)
    throw std::length_error("prefill slot index overflows int32");
  for (int w = 0; w < 2; ++w) {
    lists_by_xcd(w == 1, sc.item_cost[w], Hkv, t.num_xcds, t.xcd_piece_div, t.xcd_balance_tol,
                 sc);
    interleave_by_xcd(sc.items[w], Hkv, t.num_xcds, sc, w ? p.prefill_wide : p.prefill);
  }

  // ---- decode ranges (sized above) ------------------------------------
  if (dec_blocks > 0) {
    const int64_t sb = p.decode_split_blocks;
    // Items are placed longest first (a stable counting sort on their block
    // count, which is at most sb): first count, then place.
    auto& count = sc.count;
    count.assign((size_t)sb + 2, 0);
    each_decode_token([&](const cp_row_meta&, int32_t, int32_t kv_end) {
      const int64_t nb = ceil_div(kv_end, B);
      const int64_t ns = std::max<int64_t>(1, ceil_div(nb, sb));
      for (int64_t s = 0; s < ns; ++s) ++count[nb * (s + 1) / ns - nb * s / ns];
    });
    int64_t n_items = 0;
    for (int64_t c = sb + 1; c >= 0; --c) {  // count[c] becomes the first slot of cost c
      const int64_t k = count[c];
      count[c] = n_items;
      n_items += k;
    }
    p.decode.resize((size_t)n_items);
    each_decode_token([&](const cp_row_meta& m, int32_t tok, int32_t kv_end) {
      const int64_t nb = ceil_div(kv_end, B);
      const int64_t ns = std::max<int64_t>(1, ceil_div(nb, sb));
      int32_t part0 = -1;
      if (ns > 1) {
        part0 = (int32_t)p.partial_rows;
        p.partial_rows += (int64_t)Hkv * ns * G;
        add_merge(p, tok, 1, (int32_t)ns, part0, G, d.head_dim);
      }
      for (int64_t s = 0; s < ns; ++s) {
        const int64_t b0 = nb * s / ns, b1 = nb * (s + 1) / ns;
        DecodeItem& it = p.decode[(size_t)count[b1 - b0]++];
        it.tok = tok;
        it.req = m.req_id;
        it.kv_begin = (int32_t)(b0 * B);
        it.kv_end = (int32_t)std::min<int64_t>(b1 * B, kv_end);
        it.part = ns > 1 ? part0 + (int32_t)(s * G) : -1;
        it.part_kvh_stride = ns > 1 ? (int32_t)(ns * G) : 0;
        it.pad0 = it.pad1 = 0;
      }
    });
  }

  // ---- decode blocks inside the prefill launch ----------------------------
  // The launch that runs last (128-row tiles when there are any) takes the
  // decode units: one per 4-wave workgroup, two per 8-wave one.
  p.decode_in_prefill = 0;
  if (t.fuse_decode > 0 && !p.decode.empty() && !(p.prefill.empty() && p.prefill_wide.empty())) {
    const bool wide = p.prefill.empty();
    const int64_t n_units = (int64_t)p.decode.size() * Hkv;
    if (n_units > INT32_MAX) throw std::length_error("decode unit index overflows int32");
    place_decode_blocks(wide ? p.prefill_wide : p.prefill, p.decode, Hkv, wide, t, sc);
    p.decode_in_prefill = wide ? 2 : 1;
  }

  // ---- workspace layout ------------------------------------------------
  size_t o = 0;
  p.off_prefill = o;
  o = align_up(o + p.prefill.size() * sizeof(PrefillRec), 256);
  p.off_prefill_wide = o;
  o = align_up(o + p.prefill_wide.size() * sizeof(PrefillRec), 256);
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
  p.items.clear();
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
