// Varlen tile planner for one mixed prefill/decode batch (host side, no HIP).
//
// The scheduler packs rows of very different shapes into one iteration:
// single-token decode rows over contexts of 16..32k keys, and prefill chunks
// of a few to thousands of tokens over prior contexts of 0..32k keys (the
// intra-batch heterogeneity of Sec. 1; micro-chunks of Sec. 3.3.1).  The
// planner turns that ragged mix into three flat work lists of near-equal
// cost: prefill tiles for the MFMA kernel, decode ranges for the split-K
// kernel, and merge groups for rows whose key range was split.
#pragma once

#include <cstddef>
#include <cstdint>
#include <utility>
#include <vector>

#include "cp_attn.h"

namespace cpattn {

// Query rows per prefill workgroup: 4 waves x 32 rows, or 8 waves x 32 rows
// for chunks with more rows than that.  A row is one (query token, q head)
// pair of a single kv-head group, so a tile holds rows / G tokens of a chunk.
constexpr int kPrefillRows = 128;
constexpr int kPrefillRowsWide = 256;
// Keys per prefill main-loop iteration.
constexpr int kPrefillKeys = 64;
// Waves per decode workgroup (each wave walks every kDecodeWaves-th block).
constexpr int kDecodeWaves = 4;
// Upper bound of Tuning::prefill_min_len: rows shorter than it become one
// decode item list per token, which only pays for few-token chunks.
constexpr int kMaxPrefillMinLen = 64;

// A decode or merge item describes the work of every kv head; those kernels
// run on a grid of (items, num_kv_heads), and a split item's partial rows for
// kv head h start at part + h * part_kvh_stride.  A prefill workgroup runs
// one record, a (tile, key split, kv head), the one its index names: the
// planner lays the records out in the order the workgroups are dispatched to
// the XCDs, padded with idle records (n_tok == 0).
//
// When a step's decode rows run inside its prefill launch, that launch's
// record list also holds decode blocks (n_tok == kDecodeBlock): a workgroup of
// NW waves runs NW / 4 decode units, unit u being decode item u / num_kv_heads
// for kv head u % num_kv_heads; tok0 names the unit of waves 0-3 and pos0 the
// unit of waves 4-7 (-1: none).
constexpr int32_t kDecodeBlock = -1;

struct PrefillRec {   // 32 bytes
  int32_t tok0;       // first query token (index into q / out)
  int32_t n_tok;      // tokens in the tile, 1 .. kPrefillRows / G (or kPrefillRowsWide / G);
                      // 0: an idle record
  int32_t pos0;       // absolute position of tok0 inside its request
  int32_t req;        // block-table row
  int32_t kv_begin;   // keys [kv_begin, kv_end) of the request
  int32_t kv_end;
  int32_t part;       // -1: final output; else the first partial row of this split and kv head
  int32_t kvh;        // kv head
};

namespace detail {
struct PrefillItem {  // a tile's key split, for every kv head (planner only)
  int32_t tok0, n_tok, pos0, req, kv_begin, kv_end;
  int32_t part;       // -1, or the first partial row of kv head 0
  int32_t part_kvh_stride;
};
}  // namespace detail

struct DecodeItem {   // 32 bytes
  int32_t tok;        // query token
  int32_t req;
  int32_t kv_begin;
  int32_t kv_end;
  int32_t part;       // -1: final output; else first partial row (G rows, kv head 0)
  int32_t part_kvh_stride;
  int32_t pad0, pad1;
};

struct MergeGroup {   // 32 bytes: rows [row0, row0 + n_rows) of one split group
  int32_t tok0;       // first token of the group
  int32_t n_tok;      // tokens of the group (its rows = n_tok * G per kv head)
  int32_t n_split;    // partials to combine per row
  int32_t part0;      // kv head h, split s, row r: part0 + (h * n_split + s) * n_tok * G + r
  int32_t row0;       // first row this item merges
  int32_t n_rows;     // rows this item merges
  int32_t pad0, pad1;
};

struct AppendItem {   // 16 bytes: one request's new tokens inside one block
  int32_t tok0;       // first new token (index into k_new / v_new)
  int32_t n_tok;      // tokens, 1 .. block_size
  int32_t block;      // logical block index of the request
  int32_t req_slot0;  // req << 8 | first slot inside the block
};

struct Tuning {
  int prefill_min_len = 2;      // rows with chunk_len >= this go to the MFMA kernel, shorter
                                // rows to the decode kernel token by token (2..kMaxPrefillMinLen)
  int decode_target_items = 0;  // 0: derived from the CU count and the decode bytes
  int prefill_target_items = 0; // 0: split length chosen by the run-time estimate
  int prefill_min_split = 10;   // shortest prefill split, in kPrefillKeys steps
  int num_cus = 256;
  int num_xcds = 8;             // workgroups are dealt round-robin over the XCDs
  int64_t prefill_wide_min_rows = 129;  // chunks with chunk_len * G >= this use 256-row tiles,
  int64_t prefill_wide_min_keys = 1200; // ... when the step's mean key range per query is this
  int fuse_decode = 4;          // decode units in the (last) prefill launch: 0 no (own launch),
                                // 1 after its tiles, 2 before them, 3 spread among them,
                                // 4 longest first with them
  double fuse_spread = 1.0;     // mode 3: decode blocks spread over this fraction of the tiles
  double fuse_keys_per_step = 64.0;  // mode 4: decode keys worth one 64-key step of a tile
  bool fuse_narrow = true;      // a step with decode blocks in its prefill launch: 128-row tiles
  double fuse_units_per_cu = 0.75;   // decode ranges per CU that set the split length when
                                     // prefill dominates a fused step
  double fuse_flops_per_byte = 180.0;  // prefill dominates: its flops > this x decode bytes
  int xcd_piece_div = 4;        // K/V groups costlier than 1/(this x XCDs) of a launch's work
                                // are cut into runs of tiles of about that cost (0: never) ...
  double xcd_balance_tol = 0.25;  // ... when whole groups leave the busiest XCD more than
                                  // this fraction above the mean (negative: always)
};

namespace detail {
struct Tile {
  int32_t tok0, n_tok, pos0, req, kv_end;
  bool wide;
  int32_t item0, ns;  // its items: item0 .. item0 + ns - 1, one per split
};
struct Chunk {        // the tiles of one chunk, cut on one split grid
  int32_t tile0, n_tiles, max_ns;
  bool wide;
};
struct Group {        // items sharing one kv head's K/V range: (chunk, kv head, split),
  int32_t chunk, kvh, split;  // tiles [t0, t1) of the chunk
  int64_t cost;
  int32_t xcd;        // the XCD it is dealt to
  int32_t t0, t1;
};
}  // namespace detail

// Temporaries of build_plan, kept between calls so that a steady stream of
// batches plans without touching the allocator.
struct PlanScratch {
  std::vector<int64_t> off;
  std::vector<detail::Tile> tiles;
  std::vector<detail::Chunk> chunks;
  std::vector<int32_t> bounds;
  std::vector<int64_t> item_cost[2];
  std::vector<detail::Group> groups, pieces;
  std::vector<int64_t> load;
  std::vector<int64_t> count;
  std::vector<int32_t> flat;                          // slots grouped by XCD, longest first
  std::vector<int64_t> xcd_len;                       // slots per XCD in flat
  std::vector<detail::PrefillItem> items[2];          // 128- and 256-row tiles' key splits
  std::vector<int64_t> candidates;                    // split lengths to score
  std::vector<uint32_t> cut_lim;                      // per tile: last key a split may start at
  std::vector<std::pair<int64_t, int64_t>> groups2;  // (cost, count) of one split candidate
  std::vector<std::pair<int64_t, int64_t>> load_hist; // (slot load, slots), by load
  std::vector<PrefillRec> recs_tmp;                   // a record list being re-laid out
  std::vector<int64_t> dec_hist;                      // decode units per block count
  std::vector<std::pair<int64_t, int64_t>> dec_groups; // (cost, count) of fused decode units
};

struct Plan {
  // prefill records in dispatch order, 128-row tiles and 256-row tiles
  std::vector<PrefillRec> prefill;
  std::vector<PrefillRec> prefill_wide;
  std::vector<DecodeItem> decode;
  std::vector<MergeGroup> merge;
  int64_t partial_rows = 0;
  int32_t decode_split_blocks = 0;
  // 0: the decode items have their own launch; 1 / 2: their units run as decode
  // blocks inside the 128-row / 256-row prefill launch
  int32_t decode_in_prefill = 0;
  // workspace layout (byte offsets from the workspace base)
  size_t off_prefill = 0, off_prefill_wide = 0, off_decode = 0, off_merge = 0, off_part_o = 0,
         off_part_lse = 0;
  size_t plan_bytes = 0;   // bytes of the uploaded item lists
  size_t ws_bytes = 0;     // total workspace
  PlanScratch scratch;
};

struct AppendPlan {
  std::vector<AppendItem> items;
  size_t ws_bytes = 0;
};

// Host validation shared by every entry point.  Returns CP_OK or a CP_ERR_*.
// Thread-safe; duplicate request ids are found with a per-thread bitmap.
int validate(const cp_attn_desc* d, const cp_row_meta* rows, int32_t n_rows);

// Builds the attention plan; assumes validate() passed.  Reuses the capacity
// of every vector in `p`, so callers keep one Plan per thread.
void build_plan(const cp_attn_desc& d, const cp_row_meta* rows, int32_t n_rows, const Tuning& t,
                Plan& p);

void build_append_plan(const cp_attn_desc& d, const cp_row_meta* rows, int32_t n_rows,
                       AppendPlan& p);

// Tuning from the CP_* environment variables, read on every call.
Tuning tuning_from_env(int num_cus);

}  // namespace cpattn
