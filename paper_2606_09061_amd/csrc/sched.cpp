// Host-side chunked-prefill scheduler: Aging ordering (Sec. 3.1), LPRS
// chunk selection (Sec. 3.2, Algorithm 1) and Active Prefill Control
// (Sec. 3.3).  The C ABI and the round semantics are documented in
// include/cp_sched.h.

#include "cp_sched.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <functional>
#include <limits>
#include <new>
#include <unordered_map>
#include <vector>

namespace {

constexpr int NF = CPS_NUM_FEATURES;

struct Request {
  int64_t id;
  double arrival;
  int32_t prompt_len, max_new, processed = 0, generated = 0, chunks = 0, slot = -1;
  int32_t remaining = 0;  // r_i: prompt tokens not yet scheduled
  double first_token = -1.0, finish = -1.0;
};

// Rows of the MLP evaluated together: each weight row loaded from cache
// feeds this many accumulators.
constexpr int kRowBlock = 4;

// One affine layer for kRowBlock rows: z[r][o] = b[o] + sum_i a[r][i] * wt[i][o].
// Built for several x86-64 levels (ifunc-dispatched at load time) so that the
// inner loop runs as 4- or 8-wide double FMAs where the CPU has them.
__attribute__((target_clones("avx512f", "avx2,fma", "default"))) void affine_block(
    const double* __restrict a, int lda, int din, const double* __restrict wt, int dout,
    const double* __restrict bias, double* __restrict z, int ldz) {
  for (int r = 0; r < kRowBlock; ++r)
    for (int o = 0; o < dout; ++o) z[r * ldz + o] = bias[o];
  for (int i = 0; i < din; ++i) {
    const double* __restrict w = wt + (size_t)i * dout;
    const double a0 = a[0 * lda + i], a1 = a[1 * lda + i], a2 = a[2 * lda + i],
                 a3 = a[3 * lda + i];
    for (int o = 0; o < dout; ++o) {
      const double wo = w[o];
      z[0 * ldz + o] += a0 * wo;
      z[1 * ldz + o] += a1 * wo;
      z[2 * ldz + o] += a2 * wo;
      z[3 * ldz + o] += a3 * wo;
    }
  }
}

struct Mlp {
  std::vector<int32_t> dims;
  std::vector<double> wt, b, mean, inv_std;  // wt: per layer [din][dout] (transposed)
  double y_scale = 1.0;
  bool loaded() const { return !dims.empty(); }

  // Forward pass over n rows of x[n][NF]; out[n].  Rows go through the
  // layers kRowBlock at a time (a short last block is padded with zeros).
  void forward(const double* x, int n, double* out) const {
    const int L = (int)dims.size() - 1;
    int widest = 0;
    for (int d : dims) widest = std::max(widest, d);
    std::vector<double> a((size_t)kRowBlock * widest), z((size_t)kRowBlock * widest);
    for (int r0 = 0; r0 < n; r0 += kRowBlock) {
      const int nr = std::min(kRowBlock, n - r0);
      for (int r = 0; r < kRowBlock; ++r)
        for (int k = 0; k < NF; ++k)
          a[(size_t)r * widest + k] =
              r < nr ? (x[(size_t)(r0 + r) * NF + k] - mean[k]) * inv_std[k] : 0.0;
      size_t wo = 0, bo = 0;
      for (int l = 0; l < L; ++l) {
        const int din = dims[l], dout = dims[l + 1];
        affine_block(a.data(), widest, din, &wt[wo], dout, &b[bo], z.data(), widest);
        const bool relu = l + 1 < L;
        for (int r = 0; r < kRowBlock; ++r)
          for (int o = 0; o < dout; ++o) {
            const double v = z[(size_t)r * widest + o];
            a[(size_t)r * widest + o] = relu ? std::max(v, 0.0) : v;
          }
        wo += (size_t)din * dout;
        bo += dout;
      }
      for (int r = 0; r < nr; ++r) out[r0 + r] = a[(size_t)r * widest] * y_scale;
    }
  }
};

bool valid_config(const cps_config& c) {
  return (c.policy == CPS_POLICY_FCFS || c.policy == CPS_POLICY_AGING) &&
         (c.policy == CPS_POLICY_FCFS || (c.alpha > 0.0 && c.beta < 0.0)) &&
         std::isfinite(c.alpha) && std::isfinite(c.beta) && c.max_tokens >= 1 &&
         c.max_seqs >= 1 && c.max_seq_len >= 2 &&
         (c.chunking == CPS_CHUNK_TOKEN_BUDGET || c.chunking == CPS_CHUNK_LPRS) &&
         std::isfinite(c.target_us) && c.delta >= 1 && c.lambda_u >= 0.0 &&
         c.lambda_o >= c.lambda_u && std::isfinite(c.lambda_o) && (c.apc == 0 || c.apc == 1) &&
         c.max_active >= 1 && c.min_chunk >= 1;
}

// Raw batch statistics of Table 1 (all but the memory state), accumulated row by row.
struct Agg {
  double pf_tok = 0, dec_tok = 0, count = 0, sum_dctx = 0, max_dctx = 0, proc = 0, max_proc = 0;
  void add(const cp_row_meta& r) {
    if (r.chunk_len > 0) count += 1;
    if (r.chunk_len == 1) {
      dec_tok += 1;
      sum_dctx += r.ctx_len;
      max_dctx = std::max(max_dctx, (double)r.ctx_len);
    } else if (r.chunk_len >= 2) {
      pf_tok += r.chunk_len;
      proc += r.chunk_start;
      max_proc = std::max(max_proc, (double)r.chunk_start);
    }
  }
  // Table 1 followed by the derived features of Table 2.
  void emit(const double* mem, double* f) const {
    const double avg = sum_dctx / std::max(dec_tok, 1.0);
    const double v[NF] = {pf_tok,  dec_tok, count,  sum_dctx, max_dctx,      proc,
                          max_proc, mem[0], mem[1], mem[2],   mem[3],        1.0,
                          dec_tok + pf_tok, avg, dec_tok * avg, pf_tok * proc};
    std::memcpy(f, v, sizeof(v));
  }
};

void features(const cp_row_meta* rows, int n, const double* mem, double* f) {
  Agg g;
  for (int i = 0; i < n; ++i) g.add(rows[i]);
  g.emit(mem, f);
}

// Eq. 8: {1, h} together with the positive multiples of delta up to h, ascending.
void candidates(int32_t h, int32_t delta, std::vector<int32_t>& c) {
  c.clear();
  c.push_back(1);
  for (int64_t k = delta; k <= h; k += delta)
    if (k > 1) c.push_back((int32_t)k);
  if (h > 1 && c.back() != h) c.push_back(h);
}

// C_t of Eq. 12.
int64_t activity_cap(const cps_config& cfg, int32_t n_decode, int64_t committed) {
  const int64_t by_budget = ((int64_t)cfg.max_tokens - committed) / cfg.min_chunk;
  return std::min<int64_t>({(int64_t)cfg.max_active, (int64_t)cfg.max_seqs - n_decode, by_budget});
}

// Eq. 12–14.  Returns the chunk; *reason as documented in the header.
int32_t apc_rule(const cps_config& cfg, int32_t c_star, int32_t h, int32_t remaining,
                 int32_t n_decode, int32_t n_active, int32_t committed, int32_t* reason) {
  const int64_t cap = activity_cap(cfg, n_decode, committed);
  const int32_t m = std::min(remaining, cfg.min_chunk);  // Eq. 13
  if (n_active < cap && c_star >= m) {
    *reason = 0;
    return c_star;
  }
  if (c_star < m && n_active == 0) {
    *reason = 1;
    return std::min(h, m);
  }
  *reason = c_star >= m ? 2 : 3;
  return 0;
}

// Scratch buffers of Algorithm 1, reused across calls, and the predictions
// already made against the current committed rows: the features of a
// candidate depend only on the committed rows, its processed tokens and c
// (not on the request), so within a round, until another row is committed,
// requests at the same prefill progress (every new arrival has 0) share them.
struct SelectScratch {
  std::vector<int32_t> cand, miss;
  std::vector<double> feat, pred;
  std::unordered_map<int64_t, double> seen;  // (processed << 32 | c) -> T_hat
  // (processed << 32 | h) -> (c*, T_hat(c*)): the whole decision is shared too
  std::unordered_map<int64_t, std::pair<int32_t, double>> decided;
  Agg base;  // statistics of the committed rows
  int64_t base_tokens = 0;
  bool base_valid = false;
  void forget() {
    seen.clear();
    decided.clear();
    base_valid = false;
  }
};

// Algorithm 1 over the rows committed so far (U_t = their tokens): the
// candidate set of Eq. 8 scored by Eq. 10 on the predictions of Eq. 9, argmin
// with ties to the larger chunk (Eq. 11), then the empty-batch guard.
int32_t select_chunk(const cps_config& cfg, const Mlp& mlp, const double* mem,
                     const cp_row_meta* committed, int32_t n, int32_t slot, int32_t processed,
                     int32_t remaining, SelectScratch& sc, double* predicted,
                     int64_t* rows_scored) {
  if (!sc.base_valid) {
    sc.base = Agg();
    sc.base_tokens = 0;
    for (int32_t i = 0; i < n; ++i) {
      sc.base.add(committed[i]);
      sc.base_tokens += committed[i].chunk_len;
    }
    sc.base_valid = true;
  }
  const int64_t u = sc.base_tokens;
  const int64_t h64 = std::min<int64_t>(remaining, (int64_t)cfg.max_tokens - u);  // Eq. 6
  *predicted = std::numeric_limits<double>::quiet_NaN();
  if (h64 <= 0) return 0;
  const int32_t h = (int32_t)h64;
  const int64_t dkey = ((int64_t)processed << 32) | h;
  auto dit = sc.decided.find(dkey);
  if (dit != sc.decided.end()) {
    *predicted = dit->second.second;
    return dit->second.first;
  }
  candidates(h, cfg.delta, sc.cand);
  const int nc = (int)sc.cand.size();
  const Agg& base = sc.base;
  sc.feat.resize((size_t)nc * NF);
  sc.pred.resize(nc);
  sc.miss.clear();
  for (int k = 0; k < nc; ++k) {
    auto it = sc.seen.find(((int64_t)processed << 32) | sc.cand[k]);
    if (it != sc.seen.end()) {
      sc.pred[k] = it->second;
      continue;
    }
    Agg g = base;
    g.add({slot, processed, sc.cand[k], processed + sc.cand[k]});
    g.emit(mem, &sc.feat[sc.miss.size() * NF]);
    sc.miss.push_back(k);
  }
  if (!sc.miss.empty()) {
    std::vector<double> t(sc.miss.size());
    mlp.forward(sc.feat.data(), (int)sc.miss.size(), t.data());  // Eq. 9
    for (size_t j = 0; j < sc.miss.size(); ++j) {
      const int k = sc.miss[j];
      sc.pred[k] = t[j];
      sc.seen.emplace(((int64_t)processed << 32) | sc.cand[k], t[j]);
    }
    *rows_scored += (int64_t)sc.miss.size();
  }
  double best = std::numeric_limits<double>::infinity();
  int32_t c_star = 0;
  for (int k = 0; k < nc; ++k) {  // ascending c
    const double t = sc.pred[k];
    const double score = t <= cfg.target_us ? cfg.lambda_u * (cfg.target_us - t)
                                            : cfg.lambda_o * (t - cfg.target_us);  // Eq. 10
    if (score < best || (score == best && sc.cand[k] > c_star)) {  // Eq. 11
      best = score;
      c_star = sc.cand[k];
      *predicted = t;
    }
  }
  if (c_star == 0 && u == 0 && h >= 1) c_star = 1;  // starvation guard
  sc.decided.emplace(dkey, std::make_pair(c_star, *predicted));
  return c_star;
}

// Runs an entry point's body; a failed host allocation becomes an error code
// instead of an exception crossing the C ABI.
template <class F>
int guarded(F&& body) {
  try {
    return body();
  } catch (...) {
    return CPS_ERR_NO_MEMORY;
  }
}

// Room for `extra` more elements without a reallocation later (amortised growth).
template <class V>
void make_room(V& v, size_t extra) {
  if (v.capacity() - v.size() < extra) v.reserve(std::max(v.size() + extra, 2 * v.capacity()));
}

}  // namespace

struct cps_sched {
  cps_config cfg;
  Mlp mlp;
  double mem[4] = {0, 0, 0, 0};
  std::vector<Request> reqs;                 // by internal index
  std::unordered_map<int64_t, int32_t> by_id;
  // Waiting prefills (remaining > 0): max-heap of (key, arrival, index).
  struct Entry {
    double key, arrival;
    int32_t idx;
  };
  std::vector<Entry> heap;
  std::vector<int32_t> decoding;              // internal indices, admission order
  std::vector<int32_t> free_slots;            // stack, lowest slot on top
  // The scheduled batch awaiting cps_complete.
  std::vector<int32_t> batch_idx;
  std::vector<int32_t> batch_len;
  bool pending_batch = false;
  cps_stats stats{};
  SelectScratch scratch;

  static bool heap_less(const Entry& a, const Entry& b) {
    // max-heap on key; equal keys: earlier arrival, then lower index first
    if (a.key != b.key) return a.key < b.key;
    if (a.arrival != b.arrival) return a.arrival > b.arrival;
    return a.idx > b.idx;
  }
  double key_of(const Request& r) const {
    if (cfg.policy == CPS_POLICY_FCFS) return -r.arrival;
    return -cfg.alpha * r.arrival + cfg.beta * (double)r.remaining;  // Eq. 4
  }
  void push(int32_t idx) {
    heap.push_back({key_of(reqs[idx]), reqs[idx].arrival, idx});
    std::push_heap(heap.begin(), heap.end(), heap_less);
  }
  int32_t pop() {
    std::pop_heap(heap.begin(), heap.end(), heap_less);
    const int32_t idx = heap.back().idx;
    heap.pop_back();
    return idx;
  }

  int32_t select(const cp_row_meta* committed, int32_t n, int32_t slot, int32_t processed,
                 int32_t remaining, double* predicted) {
    stats.lprs_calls += 1;
    return select_chunk(cfg, mlp, mem, committed, n, slot, processed, remaining, scratch,
                        predicted, &stats.predictor_rows);
  }
};

extern "C" {

cps_sched* cps_create(const cps_config* cfg, int* err) {
  int dummy;
  if (!err) err = &dummy;
  if (!cfg || !valid_config(*cfg)) {
    *err = CPS_ERR_INVALID_ARG;
    return nullptr;
  }
  cps_sched* s = nullptr;
  const int rc = guarded([&] {
    s = new cps_sched();
    s->cfg = *cfg;
    s->free_slots.reserve(cfg->max_seqs);
    for (int32_t i = cfg->max_seqs - 1; i >= 0; --i) s->free_slots.push_back(i);
    return CPS_OK;
  });
  if (rc != CPS_OK) {
    delete s;
    *err = rc;
    return nullptr;
  }
  *err = CPS_OK;
  return s;
}

void cps_destroy(cps_sched* s) { delete s; }

int cps_set_predictor(cps_sched* s, int32_t n_layers, const int32_t* dims, const double* weights,
                      const double* biases, const double* x_mean, const double* x_std,
                      double y_scale) {
  if (!s || n_layers < 1 || n_layers > 16 || !dims || !weights || !biases || !x_mean || !x_std ||
      !std::isfinite(y_scale))
    return CPS_ERR_INVALID_ARG;
  if (dims[0] != NF || dims[n_layers] != 1) return CPS_ERR_INVALID_ARG;
  size_t nw = 0, nb = 0;
  for (int32_t l = 0; l < n_layers; ++l) {
    if (dims[l + 1] < 1 || dims[l + 1] > 4096) return CPS_ERR_INVALID_ARG;
    nw += (size_t)dims[l] * dims[l + 1];
    nb += dims[l + 1];
  }
  for (int k = 0; k < NF; ++k)
    if (!(x_std[k] > 0.0) || !std::isfinite(x_mean[k])) return CPS_ERR_INVALID_ARG;
  return guarded([&] {
  Mlp m;
  m.dims.assign(dims, dims + n_layers + 1);
  m.wt.resize(nw);
  for (int32_t l = 0, off = 0; l < n_layers; off += dims[l] * dims[l + 1], ++l)
    for (int32_t o = 0; o < dims[l + 1]; ++o)
      for (int32_t i = 0; i < dims[l]; ++i)
        m.wt[(size_t)off + (size_t)i * dims[l + 1] + o] = weights[(size_t)off + (size_t)o * dims[l] + i];
  m.b.assign(biases, biases + nb);
  m.mean.assign(x_mean, x_mean + NF);
  m.inv_std.resize(NF);
  for (int k = 0; k < NF; ++k) m.inv_std[k] = 1.0 / x_std[k];
  m.y_scale = y_scale;
  s->mlp = std::move(m);
  return CPS_OK;
  });
}

int cps_set_memory_state(cps_sched* s, const double mem_mb[4]) {
  if (!s || !mem_mb) return CPS_ERR_INVALID_ARG;
  for (int k = 0; k < 4; ++k)
    if (!std::isfinite(mem_mb[k])) return CPS_ERR_INVALID_ARG;
  std::memcpy(s->mem, mem_mb, sizeof(s->mem));
  return CPS_OK;
}

int cps_add_request(cps_sched* s, int64_t id, double arrival, int32_t prompt_len,
                    int32_t max_new_tokens) {
  if (!s || id < 0 || !std::isfinite(arrival) || prompt_len < 1 || max_new_tokens < 1 ||
      (int64_t)prompt_len + max_new_tokens > s->cfg.max_seq_len)
    return CPS_ERR_INVALID_ARG;
  if (s->by_id.count(id)) return CPS_ERR_STATE;
  return guarded([&] {
    // every allocation happens before the first change of state
    make_room(s->reqs, 1);
    make_room(s->heap, 1);
    const int32_t idx = (int32_t)s->reqs.size();
    s->by_id.emplace(id, idx);
    Request r;
    r.id = id;
    r.arrival = arrival;
    r.prompt_len = prompt_len;
    r.max_new = max_new_tokens;
    r.remaining = prompt_len;
    s->reqs.push_back(r);
    s->push(idx);
    return CPS_OK;
  });
}

int cps_schedule(cps_sched* s, double now, cp_row_meta* rows, int64_t* ids, int32_t cap,
                 int32_t* n_rows, int32_t* n_decode_out) {
  if (!s || !rows || !ids || !n_rows || !n_decode_out || cap < 0 || !std::isfinite(now))
    return CPS_ERR_INVALID_ARG;
  if (s->pending_batch) return CPS_ERR_STATE;
  if (s->cfg.chunking == CPS_CHUNK_LPRS && !s->mlp.loaded()) return CPS_ERR_NO_PREDICTOR;
  // Every row holds a distinct slot, so max_seqs rows always fit.
  if (cap < std::min<int64_t>(s->cfg.max_seqs, (int64_t)s->decoding.size() + (int64_t)s->heap.size()))
    return CPS_ERR_CAPACITY;
  return guarded([&] {
  const cps_config& cfg = s->cfg;
  make_room(s->batch_idx, (size_t)cap);
  make_room(s->batch_len, (size_t)cap);
  int32_t n = 0;
  int64_t u = 0;
  s->batch_idx.clear();
  s->batch_len.clear();
  // Decode-first admission.
  for (int32_t idx : s->decoding) {
    if (u >= cfg.max_tokens) break;
    Request& r = s->reqs[idx];
    const int32_t pos = r.prompt_len + r.generated - 1;
    rows[n] = {r.slot, pos, 1, pos + 1};
    ids[n] = r.id;
    s->batch_idx.push_back(idx);
    s->batch_len.push_back(1);
    ++n;
    ++u;
  }
  const int32_t n_decode = n;
  int32_t n_active = 0;
  s->scratch.forget();
  std::vector<int32_t> popped;
  popped.reserve(s->heap.size());
  while (!s->heap.empty() && u < cfg.max_tokens && n < cap) {
    if (cfg.apc && n_active > 0 && n_active >= activity_cap(cfg, n_decode, u)) {
      s->stats.apc_not_scored += (int64_t)s->heap.size();
      break;
    }
    const int32_t idx = s->pop();
    popped.push_back(idx);
    Request& r = s->reqs[idx];
    if (r.slot < 0 && s->free_slots.empty()) {
      s->stats.skipped_no_slot += 1;
      continue;
    }
    const int32_t h = (int32_t)std::min<int64_t>(r.remaining, cfg.max_tokens - u);  // Eq. 6
    int32_t c;
    double t_hat;
    const int32_t slot_for_features = r.slot >= 0 ? r.slot : s->free_slots.back();
    if (cfg.chunking == CPS_CHUNK_LPRS)
      c = s->select(rows, n, slot_for_features, r.processed, r.remaining, &t_hat);
    else
      c = h;  // Eq. 7
    if (cfg.apc) {
      int32_t reason;
      const int32_t c_apc = apc_rule(cfg, c, h, r.remaining, n_decode, n_active, (int32_t)u, &reason);
      if (reason == 2) s->stats.apc_blocked_cap += 1;
      if (reason == 3) s->stats.apc_blocked_min += 1;
      if (reason == 1 && c_apc != c) s->stats.apc_warm_starts += 1;
      c = c_apc;
    }
    if (c <= 0) continue;
    if (r.slot < 0) {
      r.slot = s->free_slots.back();
      s->free_slots.pop_back();
    }
    rows[n] = {r.slot, r.processed, c, r.processed + c};
    s->scratch.forget();  // the committed rows changed
    ids[n] = r.id;
    s->batch_idx.push_back(idx);
    s->batch_len.push_back(c);
    ++n;
    ++n_active;
    u += c;
    r.remaining -= c;  // Eq. 2
    r.chunks += 1;
    s->stats.prefill_rows += 1;
    s->stats.prefill_tokens += c;
  }
  for (int32_t idx : popped)
    if (s->reqs[idx].remaining > 0) s->push(idx);
  s->stats.rounds += 1;
  s->stats.decode_rows += n_decode;
  s->pending_batch = true;
  *n_rows = n;
  *n_decode_out = n_decode;
  return CPS_OK;
  });
}

int cps_complete(cps_sched* s, double now) {
  if (!s || !std::isfinite(now)) return CPS_ERR_INVALID_ARG;
  if (!s->pending_batch) return CPS_ERR_STATE;
  return guarded([&] {
  // every allocation happens before the first change of state
  std::vector<int32_t> still;
  still.reserve(s->decoding.size() + s->batch_idx.size());
  std::vector<char> done(s->reqs.size(), 0);
  make_room(s->decoding, s->batch_idx.size());
  make_room(s->free_slots, s->batch_idx.size());
  for (size_t k = 0; k < s->batch_idx.size(); ++k) {
    Request& r = s->reqs[s->batch_idx[k]];
    if (r.processed < r.prompt_len) {  // a prefill chunk
      r.processed += s->batch_len[k];
      if (r.processed == r.prompt_len) {
        r.first_token = now;
        r.generated = 1;
        if (r.generated < r.max_new) {
          s->decoding.push_back(s->batch_idx[k]);
          continue;
        }
      } else {
        continue;
      }
    } else {
      r.generated += 1;
      if (r.generated < r.max_new) continue;
    }
    r.finish = now;
    done[s->batch_idx[k]] = 1;
    s->free_slots.push_back(r.slot);
    s->stats.finished += 1;
  }
  for (int32_t idx : s->decoding)
    if (!done[idx]) still.push_back(idx);
  s->decoding.swap(still);
  // Keep the lowest free slot on top of the stack.
  std::sort(s->free_slots.begin(), s->free_slots.end(), std::greater<int32_t>());
  s->pending_batch = false;
  return CPS_OK;
  });
}

int cps_get_stats(const cps_sched* s, cps_stats* out) {
  if (!s || !out) return CPS_ERR_INVALID_ARG;
  *out = s->stats;
  return CPS_OK;
}

int cps_request(const cps_sched* s, int64_t id, cps_request_info* out) {
  if (!s || !out) return CPS_ERR_INVALID_ARG;
  auto it = s->by_id.find(id);
  if (it == s->by_id.end()) return CPS_ERR_INVALID_ARG;
  const Request& r = s->reqs[it->second];
  *out = {r.arrival, r.first_token, r.finish, r.prompt_len, r.max_new,
          r.processed, r.generated, r.chunks, r.slot};
  return CPS_OK;
}

int64_t cps_pending(const cps_sched* s) {
  if (!s) return CPS_ERR_INVALID_ARG;
  return (int64_t)s->reqs.size() - s->stats.finished;
}

int cps_batch_features(const cp_row_meta* rows, int32_t n_rows, const double mem_mb[4],
                       double* out) {
  if ((!rows && n_rows > 0) || n_rows < 0 || !mem_mb || !out) return CPS_ERR_INVALID_ARG;
  return guarded([&] {
    features(rows, n_rows, mem_mb, out);
    return CPS_OK;
  });
}

int cps_predict(const cps_sched* s, const double* x, int32_t n, double* out) {
  if (!s || (!x && n > 0) || (!out && n > 0) || n < 0) return CPS_ERR_INVALID_ARG;
  if (!s->mlp.loaded()) return CPS_ERR_NO_PREDICTOR;
  return guarded([&] {
    s->mlp.forward(x, n, out);
    return CPS_OK;
  });
}

int cps_select_chunk(const cps_sched* s, const cp_row_meta* committed, int32_t n_committed,
                     int32_t slot, int32_t processed, int32_t remaining, int32_t* chunk,
                     double* predicted) {
  if (!s || (!committed && n_committed > 0) || n_committed < 0 || processed < 0 ||
      remaining < 0 || !chunk || !predicted)
    return CPS_ERR_INVALID_ARG;
  if (!s->mlp.loaded()) return CPS_ERR_NO_PREDICTOR;
  // Own scratch and counter: the scheduler's state is left unchanged.
  return guarded([&] {
    SelectScratch sc;
    int64_t scored = 0;
    *chunk = select_chunk(s->cfg, s->mlp, s->mem, committed, n_committed, slot, processed,
                          remaining, sc, predicted, &scored);
    return CPS_OK;
  });
}

int cps_apc_decide(const cps_config* cfg, int32_t c_star, int32_t h, int32_t remaining,
                   int32_t n_decode, int32_t n_active, int32_t committed, int32_t* chunk,
                   int32_t* reason) {
  if (!cfg || !valid_config(*cfg) || !chunk || !reason || c_star < 0 || h < 0 || remaining < 1 ||
      n_decode < 0 || n_active < 0 || committed < 0 || committed > cfg->max_tokens)
    return CPS_ERR_INVALID_ARG;
  *chunk = apc_rule(*cfg, c_star, h, remaining, n_decode, n_active, committed, reason);
  return CPS_OK;
}

}  // extern "C"
