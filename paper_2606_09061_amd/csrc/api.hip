// C ABI of libcpattn: validation, planning, plan upload and launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "cp_attn.h"
#include "copy_body.hpp"
#include "kernels.hpp"
#include "plan.hpp"

using namespace cpattn;

namespace {

constexpr int kRingSlots = 8;

// Device scratch of the allocation-free entry point, one copy per GPU (each
// device holds it from the library's load until the process ends).  Host code
// never passes `scratch` itself: it stands for the array only on the host
// side; the per-device address comes from hipGetSymbolAddress at set-up.
static __device__ __align__(256) uint8_t scratch[CP_NOALLOC_SCRATCH_BYTES];
constexpr int kNoallocSlots = 2;  // pinned plan-staging slots of that path

// Pinned host staging for plan uploads: fine-grained (coherent) host memory
// that the plan-copy kernel reads directly.  Each workgroup of that kernel,
// once it has read its part of the slot, writes the call's sequence number
// into the slot's completion words (fine-grained host memory too); a slot is
// rewritten only after all of them show its last sequence number.  So a host
// write never races a GPU read, whatever the stream, and no event sits
// between the kernels (an event record costs the GPU 5-10 us of idle time).
constexpr int kCopyBlocksMax = 16;      // workgroups of one plan copy
constexpr size_t kStageHeader = 256;    // completion words ahead of the data
struct Stage {
  void* base = nullptr;                 // allocation: [completion words][data]
  uint8_t* host = nullptr;              // data, as the host writes it
  const void* dev = nullptr;            // data, as the GPU addresses it
  uint32_t* done_host = nullptr;        // kCopyBlocksMax completion words
  uint32_t* done_dev = nullptr;
  size_t cap = 0;
  uint32_t seq = 0;                     // sequence number of its last copy (0: none)
  int blocks = 0;                       // workgroups of that copy
  bool busy = false;
};
constexpr size_t kStageMinBytes = 1u << 20;

// Copies n16 16-byte words of a staged plan from pinned host memory into the
// workspace: each workgroup takes 128 KiB pieces (8 words per thread, all
// loads in flight before the stores: one host round trip per piece), then
// marks its part done with `seq`.  Replaces hipMemcpyAsync, which sends
// copies above 16 KB to the DMA engine and leaves the GPU idle ~24 us.
constexpr int kCopyPer = 8;
constexpr int kCopyPiece = kCopyPer * 1024;
__global__ __launch_bounds__(1024) void plan_copy_kernel(const uint4* __restrict__ src,
                                                         uint4* __restrict__ dst, int n16,
                                                         uint32_t* __restrict__ done,
                                                         uint32_t seq) {
  plan_copy_body<1024, kCopyPer>(src, dst, n16, done, seq, (int)blockIdx.x, (int)gridDim.x,
                                 (int)threadIdx.x);
}

// Waits until the slot's last copy has read it (normally long done: a slot
// comes round again only several calls later).
int wait_copied(const Stage& st) {
  if (st.seq == 0) return CP_OK;
  const auto t0 = std::chrono::steady_clock::now();
  for (int b = 0; b < st.blocks; ++b) {
    long spins = 0;
    while (__atomic_load_n(&st.done_host[b], __ATOMIC_ACQUIRE) != st.seq) {
      if (++spins % 256 == 0) {
        std::this_thread::yield();
        if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(60)) return CP_ERR_HIP;
      }
    }
  }
  return CP_OK;
}

// Allocates (or grows) a slot's pinned buffer; its last copy must be done.
int stage_reserve(Stage& st, size_t bytes) {
  if (st.cap >= bytes) return CP_OK;
  if (st.base) (void)hipHostFree(st.base);
  st = Stage{};
  size_t cap = kStageMinBytes;
  while (cap < bytes) cap *= 2;
  void* b = nullptr;
  if (hipHostMalloc(&b, cap + kStageHeader, hipHostMallocMapped | hipHostMallocCoherent) !=
      hipSuccess)
    return CP_ERR_HIP;
  void* d = nullptr;
  if (hipHostGetDevicePointer(&d, b, 0) != hipSuccess || !d) {
    (void)hipHostFree(b);
    return CP_ERR_HIP;
  }
  std::memset(b, 0, kStageHeader);
  st.base = b;
  st.done_host = static_cast<uint32_t*>(b);
  st.done_dev = static_cast<uint32_t*>(d);
  st.host = static_cast<uint8_t*>(b) + kStageHeader;
  st.dev = static_cast<const uint8_t*>(d) + kStageHeader;
  st.cap = cap;
  return CP_OK;
}

// Enqueues the copy of a staged slot's first `bytes` (a multiple of 16) into
// dst under the next sequence number `seq` (never 0).
int launch_plan_copy(Stage& st, void* dst, size_t bytes, uint32_t seq, hipStream_t s) {
  const int n16 = (int)(bytes / 16);
  const int grid = std::min(kCopyBlocksMax, (n16 + kCopyPiece - 1) / kCopyPiece);
  hipLaunchKernelGGL(plan_copy_kernel, dim3(grid), dim3(1024), 0, s,
                     static_cast<const uint4*>(st.dev), static_cast<uint4*>(dst), n16, st.done_dev,
                     seq);
  if (hipGetLastError() != hipSuccess) return CP_ERR_HIP;
  st.seq = seq;
  st.blocks = grid;
  return CP_OK;
}

// Per-device state: the staging ring; for the allocation-free path the
// device address of `scratch` and its fixed-size staging slots (set up by
// cp_noalloc_init).
struct DeviceCtx {
  Stage ring[kRingSlots];
  int next = 0;
  uint32_t seq = 0;  // sequence numbers of plan copies on this device
  uint8_t* scratch_dev = nullptr;
  Stage noalloc_ring[kNoallocSlots];
  int noalloc_next = 0;
};

std::mutex g_mu;
std::vector<DeviceCtx*> g_devs;

int num_cus_setting() {
  static const int n = [] {
    const char* s = std::getenv("CP_NUM_CUS");
    const int v = s ? std::atoi(s) : 0;
    return v > 0 ? v : 256;  // MI355X
  }();
  return n;
}

// CP_DEBUG=1: check block-table entries on the host before enqueueing and
// synchronise after every launch (read on every call).
bool debug_mode() {
  const char* s = std::getenv("CP_DEBUG");
  return s && s[0] == '1';
}

int check_tables_host(const cp_attn_desc* d, const int32_t* bt, const cp_row_meta* rows,
                      int32_t n_rows) {
  const int64_t mbr = d->max_blocks_per_req;
  for (int32_t r = 0; r < n_rows; ++r) {
    const int64_t nb = ((int64_t)rows[r].ctx_len + d->block_size - 1) / d->block_size;
    const int32_t* e = bt + (int64_t)rows[r].req_id * mbr;
    for (int64_t i = 0; i < nb; ++i)
      if (e[i] < 0 || e[i] >= d->num_blocks) return CP_ERR_BAD_META;
  }
  return CP_OK;
}

// Debug path: waits for the stream (earlier work may still write the table),
// copies the entries the batch reads to the host and checks them.
int debug_check_tables(const cp_attn_desc* d, const int32_t* bt_dev, const cp_row_meta* rows,
                       int32_t n_rows, hipStream_t s) {
  if (hipStreamSynchronize(s) != hipSuccess) return CP_ERR_HIP;
  const int64_t mbr = d->max_blocks_per_req;
  std::vector<int32_t> host((size_t)d->num_reqs_in_table * mbr, 0);
  for (int32_t r = 0; r < n_rows; ++r) {
    const int64_t nb = ((int64_t)rows[r].ctx_len + d->block_size - 1) / d->block_size;
    if (nb == 0) continue;
    const int64_t off = (int64_t)rows[r].req_id * mbr;
    if (hipMemcpy(host.data() + off, bt_dev + off, (size_t)nb * sizeof(int32_t),
                  hipMemcpyDefault) != hipSuccess)
      return CP_ERR_HIP;
  }
  return check_tables_host(d, host.data(), rows, n_rows);
}

// Requires g_mu held.
uint32_t next_seq(DeviceCtx* c) {
  if (++c->seq == 0) ++c->seq;
  return c->seq;
}

// Requires g_mu held.
DeviceCtx* device_ctx(int* err) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    *err = CP_ERR_HIP;
    return nullptr;
  }
  if ((int)g_devs.size() <= dev) g_devs.resize(dev + 1, nullptr);
  if (!g_devs[dev]) g_devs[dev] = new (std::nothrow) DeviceCtx();
  if (!g_devs[dev]) *err = CP_ERR_HIP;
  return g_devs[dev];
}

// Takes a free ring slot of the current device (waiting for its previous
// copy if that is still pending), fills it through `fill(host)` and draws the
// sequence number of its copy.  The slot stays busy until release_stage.
template <class Fill>
int take_stage(size_t bytes, Stage** taken, uint32_t* seq, Fill&& fill) {
  *taken = nullptr;
  for (;;) {
    std::unique_lock<std::mutex> lk(g_mu);
    int err = CP_OK;
    DeviceCtx* c = device_ctx(&err);
    if (!c) return err;
    Stage* st = nullptr;
    for (int k = 0; k < kRingSlots && !st; ++k) {
      Stage& cand = c->ring[(c->next + k) % kRingSlots];
      if (!cand.busy) {
        st = &cand;
        c->next = (c->next + k + 1) % kRingSlots;
      }
    }
    if (!st) {  // every slot inside another thread's call: let one finish
      lk.unlock();
      std::this_thread::yield();
      continue;
    }
    int rc = wait_copied(*st);
    if (rc == CP_OK) rc = stage_reserve(*st, bytes);
    if (rc != CP_OK) return rc;
    fill(st->host);
    *seq = next_seq(c);
    st->busy = true;
    *taken = st;
    return CP_OK;
  }
}

// take_stage, then the copy of the slot into dst on stream s.
template <class Fill>
int upload(void* dst, size_t bytes, hipStream_t s, Stage** taken, Fill&& fill) {
  *taken = nullptr;
  if (bytes == 0) return CP_OK;
  uint32_t seq = 0;
  const int rc = take_stage(bytes, taken, &seq, fill);
  if (rc != CP_OK) return rc;
  if (launch_plan_copy(**taken, dst, bytes, seq, s) != CP_OK) {
    std::lock_guard<std::mutex> lk(g_mu);
    (*taken)->busy = false;
    *taken = nullptr;
    return CP_ERR_HIP;
  }
  return CP_OK;
}

// After the call's last launch the slot may be taken again (its completion
// words guard the data until the copy has read it).
int release_stage(Stage* st, hipStream_t) {
  if (!st) return CP_OK;
  std::lock_guard<std::mutex> lk(g_mu);
  st->busy = false;
  return CP_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int64_t total_tokens(const cp_row_meta* rows, int32_t n) {
  int64_t t = 0;
  for (int32_t i = 0; i < n; ++i) t += rows[i].chunk_len;
  return t;
}

// ---- per-kernel event timing (diagnostics)
struct ProfPair {
  hipEvent_t a = nullptr, b = nullptr;
  int kind = 0;
};
struct Profiler {
  bool on = false;
  std::vector<ProfPair> pool;
  size_t used = 0;
};
Profiler g_prof;

// Records the opening event of a launch of `kind`; returns the pair index or -1.
long prof_open(int kind, hipStream_t s) {
  if (!g_prof.on) return -1;
  if (g_prof.used == g_prof.pool.size()) {
    ProfPair p;
    if (hipEventCreate(&p.a) != hipSuccess || hipEventCreate(&p.b) != hipSuccess) return -1;
    g_prof.pool.push_back(p);
  }
  ProfPair& p = g_prof.pool[g_prof.used];
  p.kind = kind;
  if (hipEventRecord(p.a, s) != hipSuccess) return -1;
  return (long)g_prof.used++;
}

void prof_close(long idx, hipStream_t s) {
  if (idx >= 0) (void)hipEventRecord(g_prof.pool[idx].b, s);
}

int finish(hipError_t e, hipStream_t s) {
  if (e != hipSuccess) return CP_ERR_HIP;
  if (debug_mode()) {
    if (hipStreamSynchronize(s) != hipSuccess) return CP_ERR_HIP;
    if (hipGetLastError() != hipSuccess) return CP_ERR_HIP;
  }
  return CP_OK;
}

template <class T>
void put(uint8_t* buf, size_t off, const std::vector<T>& v) {
  if (!v.empty()) std::memcpy(buf + off, v.data(), v.size() * sizeof(T));
}

// The plan's item lists at their workspace offsets (p.plan_bytes bytes).
void serialize_into(const Plan& p, uint8_t* buf) {
  put(buf, p.off_prefill, p.prefill);
  put(buf, p.off_prefill_wide, p.prefill_wide);
  put(buf, p.off_decode, p.decode);
  put(buf, p.off_merge, p.merge);
}

// The plan's lists, counts and workspace offsets as the caller-visible struct.
void fill_plan(const Plan& p, cp_attn_plan& pl) {
  pl.ws_bytes = (int64_t)p.ws_bytes;
  pl.n_decode = (int32_t)p.decode.size();
  pl.n_merge = (int32_t)p.merge.size();
  pl.off_prefill = (int64_t)p.off_prefill;
  pl.off_prefill_wide = (int64_t)p.off_prefill_wide;
  pl.off_decode = (int64_t)p.off_decode;
  pl.off_merge = (int64_t)p.off_merge;
  pl.off_part_o = (int64_t)p.off_part_o;
  pl.off_part_lse = (int64_t)p.off_part_lse;
  pl.n_prefill_items = (int32_t)p.prefill.size();
  pl.n_prefill_wide_items = (int32_t)p.prefill_wide.size();
  pl.partial_rows = p.partial_rows;
  pl.decode_in_prefill = p.decode_in_prefill;
  pl.reserved = 0;
}

// Allocation-free upload: writes the plan straight into one of the device's
// fixed pinned slots (after the copy that last read it has completed) and
// enqueues the copy into `dst`; *taken is released by the caller after its
// last launch.  Requires g_mu held and plan_bytes within the slot size.
int upload_noalloc(DeviceCtx* c, void* dst, const Plan& p, hipStream_t s, Stage** taken) {
  Stage& st = c->noalloc_ring[c->noalloc_next];
  c->noalloc_next = (c->noalloc_next + 1) % kNoallocSlots;
  const int rc = wait_copied(st);
  if (rc != CP_OK) return rc;
  serialize_into(p, st.host);
  if (launch_plan_copy(st, dst, p.plan_bytes, next_seq(c), s) != CP_OK) return CP_ERR_HIP;
  st.busy = true;
  *taken = &st;
  return CP_OK;
}

// One plan per thread, reused across calls (its vectors keep their capacity).
Plan& thread_plan() {
  thread_local Plan p;
  return p;
}

AppendPlan& thread_append_plan() {
  thread_local AppendPlan p;
  return p;
}

}  // namespace

extern "C" {

int cp_version(void) { return 1 * 10000 + 0 * 100 + 0; }

const char* cp_strerror(int code) {
  switch (code) {
    case CP_OK: return "success";
    case CP_ERR_INVALID_ARG: return "invalid argument (null pointer, size or alignment)";
    case CP_ERR_BAD_META: return "malformed row metadata";
    case CP_ERR_WORKSPACE: return "workspace too small";
    case CP_ERR_UNSUPPORTED: return "unsupported head_dim, block_size or head group";
    case CP_ERR_HIP: return "HIP runtime error";
  }
  return "unknown error";
}

int cp_check_batch(const cp_attn_desc* desc, const cp_row_meta* rows, int32_t n_rows) {
  return validate(desc, rows, n_rows);
}

int cp_check_block_tables(const cp_attn_desc* desc, const int32_t* block_tables_host,
                          const cp_row_meta* rows, int32_t n_rows) {
  const int v = validate(desc, rows, n_rows);
  if (v != CP_OK) return v;
  if (!block_tables_host) return n_rows > 0 ? CP_ERR_INVALID_ARG : CP_OK;
  return check_tables_host(desc, block_tables_host, rows, n_rows);
}

size_t cp_workspace_bytes(const cp_attn_desc* desc, const cp_row_meta* rows, int32_t n_rows) {
  if (validate(desc, rows, n_rows) != CP_OK) return 0;
  try {
    Plan& p = thread_plan();
    build_plan(*desc, rows, n_rows, tuning_from_env(num_cus_setting()), p);
    AppendPlan& a = thread_append_plan();
    build_append_plan(*desc, rows, n_rows, a);
    return p.ws_bytes > a.ws_bytes ? p.ws_bytes : a.ws_bytes;
  } catch (...) {
    return 0;
  }
}

int cp_plan_summary(const cp_attn_desc* desc, const cp_row_meta* rows, int32_t n_rows,
                    int64_t counts[6]) {
  const int v = validate(desc, rows, n_rows);
  if (v != CP_OK) return v;
  if (!counts) return CP_ERR_INVALID_ARG;
  try {
    Plan& p = thread_plan();
    build_plan(*desc, rows, n_rows, tuning_from_env(num_cus_setting()), p);
    const int64_t hkv = desc->num_kv_heads;
    counts[0] = 0;
    for (const PrefillRec& r : p.prefill) counts[0] += r.n_tok > 0;
    for (const PrefillRec& r : p.prefill_wide) counts[0] += r.n_tok > 0;
    counts[1] = (int64_t)p.decode.size() * hkv;
    counts[2] = (int64_t)p.merge.size() * hkv;
    counts[3] = p.partial_rows;
    counts[5] = p.decode_split_blocks;
    AppendPlan& a = thread_append_plan();
    build_append_plan(*desc, rows, n_rows, a);
    counts[4] = (int64_t)(p.ws_bytes > a.ws_bytes ? p.ws_bytes : a.ws_bytes);
  } catch (...) {
    return CP_ERR_INVALID_ARG;
  }
  return CP_OK;
}

int64_t cp_plan_items(const cp_attn_desc* desc, const cp_row_meta* rows, int32_t n_rows,
                      int32_t* items, int64_t cap) {
  const int v = validate(desc, rows, n_rows);
  if (v != CP_OK) return v;
  if (cap > 0 && !items) return CP_ERR_INVALID_ARG;
  try {
    Plan& p = thread_plan();
    build_plan(*desc, rows, n_rows, tuning_from_env(num_cus_setting()), p);
    const int32_t hkv = desc->num_kv_heads;
    int64_t n = 0;
    auto put_item = [&](int32_t kind, int32_t tok, int32_t ntok, int32_t pos, int32_t req,
                        int32_t kvh, int32_t kb, int32_t ke) {
      if (n < cap) {
        int32_t* o = items + 8 * n;
        o[0] = kind, o[1] = tok, o[2] = ntok, o[3] = pos, o[4] = req, o[5] = kvh, o[6] = kb,
        o[7] = ke;
      }
      ++n;
    };
    // prefill records in dispatch order (idle padding skipped)
    for (int w = 1; w >= 0; --w)
      for (const PrefillRec& r : (w ? p.prefill_wide : p.prefill))
        if (r.n_tok > 0) put_item(0, r.tok0, r.n_tok, r.pos0, r.req, r.kvh, r.kv_begin, r.kv_end);
    // position of a decode query: chunk_start + its index inside the row
    std::vector<int32_t> pos_of_tok;
    {
      int64_t t = 0;
      for (int32_t r = 0; r < n_rows; ++r) t += rows[r].chunk_len;
      pos_of_tok.assign((size_t)t, -1);
      t = 0;
      for (int32_t r = 0; r < n_rows; ++r)
        for (int32_t j = 0; j < rows[r].chunk_len; ++j) pos_of_tok[(size_t)t++] = rows[r].chunk_start + j;
    }
    for (int32_t h = 0; h < hkv; ++h)
      for (const DecodeItem& it : p.decode)
        put_item(1, it.tok, 1, pos_of_tok[(size_t)it.tok], it.req, h, it.kv_begin, it.kv_end);
    return n;
  } catch (...) {
    return CP_ERR_INVALID_ARG;
  }
}

int64_t cp_plan_records(const cp_attn_desc* desc, const cp_row_meta* rows, int32_t n_rows,
                        int32_t which, int32_t* recs, int64_t cap) {
  const int v = validate(desc, rows, n_rows);
  if (v != CP_OK) return v;
  if ((which != 0 && which != 1) || (cap > 0 && !recs)) return CP_ERR_INVALID_ARG;
  try {
    Plan& p = thread_plan();
    build_plan(*desc, rows, n_rows, tuning_from_env(num_cus_setting()), p);
    const std::vector<PrefillRec>& l = which ? p.prefill_wide : p.prefill;
    const int64_t n = (int64_t)l.size();
    if (cap > 0) std::memcpy(recs, l.data(), (size_t)std::min(cap, n) * sizeof(PrefillRec));
    return n;
  } catch (...) {
    return CP_ERR_INVALID_ARG;
  }
}

int cp_kv_append(const cp_attn_desc* desc, const void* k_new, const void* v_new, void* k_cache,
                 void* v_cache, const int32_t* block_tables, const cp_row_meta* rows,
                 int32_t n_rows, void* ws, size_t ws_bytes, void* stream) {
  const int v = validate(desc, rows, n_rows);
  if (v != CP_OK) return v;
  if (total_tokens(rows, n_rows) == 0) return CP_OK;
  if (!k_new || !v_new || !k_cache || !v_cache || !block_tables || !ws) return CP_ERR_INVALID_ARG;
  if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_cache, 16) ||
      !aligned(v_cache, 16) || !aligned(ws, 256) || !aligned(block_tables, 4))
    return CP_ERR_INVALID_ARG;
  try {
    AppendPlan& p = thread_append_plan();
    build_append_plan(*desc, rows, n_rows, p);
    if (ws_bytes < p.ws_bytes) return CP_ERR_WORKSPACE;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (debug_mode()) {
      const int rc = debug_check_tables(desc, block_tables, rows, n_rows, s);
      if (rc != CP_OK) return rc;
    }
    AppendArgs a;
    a.items = reinterpret_cast<const AppendItem*>(ws);
    a.n_items = (int)p.items.size();
    a.k_new = static_cast<const uint16_t*>(k_new);
    a.v_new = static_cast<const uint16_t*>(v_new);
    a.k_cache = static_cast<uint16_t*>(k_cache);
    a.v_cache = static_cast<uint16_t*>(v_cache);
    a.bt = block_tables;
    a.hkv = desc->num_kv_heads;
    a.mbr = desc->max_blocks_per_req;
    const AppendInline* inl = nullptr;
    Stage* st = nullptr;
    if (a.n_items <= kAppendInlineItems) {
      thread_local AppendInline buf;
      std::memcpy(buf.items, p.items.data(), p.items.size() * sizeof(AppendItem));
      inl = &buf;
    } else {
      const size_t bytes = p.items.size() * sizeof(AppendItem);
      const int rc = upload(ws, bytes, s, &st, [&](uint8_t* h) {
        std::memcpy(h, p.items.data(), bytes);
      });
      if (rc != CP_OK) return rc;
    }
    const long pi = prof_open(0, s);
    const hipError_t e = launch_append(desc->head_dim, desc->block_size, a, inl, s);
    prof_close(pi, s);
    const int rs = release_stage(st, s);
    const int rf = finish(e, s);
    return rf != CP_OK ? rf : rs;
  } catch (...) {
    return CP_ERR_INVALID_ARG;
  }
}

}  // extern "C"

namespace {

// cp_attn_prepare, leaving the plan's staging slot busy in *st (released by
// the caller after its last launch, so the slot's event follows the kernels
// rather than sitting between the copy and the first of them).
int prepare_impl(const cp_attn_desc* desc, const cp_row_meta* rows, int32_t n_rows, void* ws,
                 size_t ws_bytes, hipStream_t s, cp_attn_plan* plan, Stage** st) {
  *st = nullptr;
  if (!plan) return CP_ERR_INVALID_ARG;
  const int v = validate(desc, rows, n_rows);
  if (v != CP_OK) return v;
  cp_attn_plan pl{};
  pl.desc = *desc;
  pl.tokens = total_tokens(rows, n_rows);
  if (pl.tokens == 0) {
    *plan = pl;
    return CP_OK;
  }
  if (!ws || !aligned(ws, 256)) return CP_ERR_INVALID_ARG;
  try {
    Plan& p = thread_plan();
    build_plan(*desc, rows, n_rows, tuning_from_env(num_cus_setting()), p);
    if (ws_bytes < p.ws_bytes) return CP_ERR_WORKSPACE;
    const int rc = upload(ws, p.plan_bytes, s, st, [&](uint8_t* h) { serialize_into(p, h); });
    if (rc != CP_OK) return rc;
    fill_plan(p, pl);
    *plan = pl;
    return CP_OK;
  } catch (...) {
    return CP_ERR_INVALID_ARG;
  }
}

}  // namespace

extern "C" {

int cp_attn_prepare(const cp_attn_desc* desc, const cp_row_meta* rows, int32_t n_rows, void* ws,
                    size_t ws_bytes, void* stream, cp_attn_plan* plan) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Stage* st = nullptr;
  const int rc = prepare_impl(desc, rows, n_rows, ws, ws_bytes, s, plan, &st);
  const int rs = release_stage(st, s);
  return rc != CP_OK ? rc : rs;
}

int cp_attn_run(const cp_attn_plan* plan, const void* q, const void* k_cache, const void* v_cache,
                const int32_t* block_tables, void* out, void* ws, size_t ws_bytes, void* stream) {
  if (!plan) return CP_ERR_INVALID_ARG;
  const cp_attn_desc* desc = &plan->desc;
  const int vd = validate(desc, nullptr, 0);
  if (vd != CP_OK) return vd;
  if (plan->tokens == 0) return CP_OK;
  if (plan->ws_bytes <= 0 || plan->n_prefill_items < 0 || plan->n_prefill_wide_items < 0 ||
      plan->n_decode < 0 || plan->n_merge < 0 || plan->partial_rows < 0)
    return CP_ERR_INVALID_ARG;
  // decode items inside a prefill launch need that launch
  if (plan->decode_in_prefill < 0 || plan->decode_in_prefill > 2 ||
      (plan->decode_in_prefill == 1 && plan->n_prefill_items == 0) ||
      (plan->decode_in_prefill == 2 && plan->n_prefill_wide_items == 0) ||
      (int64_t)plan->n_decode * desc->num_kv_heads > INT32_MAX)
    return CP_ERR_INVALID_ARG;
  if ((size_t)plan->ws_bytes > ws_bytes) return CP_ERR_WORKSPACE;
  if (!q || !k_cache || !v_cache || !block_tables || !out || !ws) return CP_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16) ||
      !aligned(ws, 256) || !aligned(block_tables, 4))
    return CP_ERR_INVALID_ARG;
  const int64_t offs[6] = {plan->off_prefill, plan->off_prefill_wide, plan->off_decode,
                           plan->off_merge,   plan->off_part_o,       plan->off_part_lse};
  for (int64_t o : offs)
    if (o < 0 || o > plan->ws_bytes) return CP_ERR_INVALID_ARG;
  // every list the kernels read lies inside the plan's workspace
  const int64_t D64 = desc->head_dim;
  const int64_t ends[6] = {
      plan->off_prefill + (int64_t)plan->n_prefill_items * (int64_t)sizeof(PrefillRec),
      plan->off_prefill_wide + (int64_t)plan->n_prefill_wide_items * (int64_t)sizeof(PrefillRec),
      plan->off_decode + (int64_t)plan->n_decode * (int64_t)sizeof(DecodeItem),
      plan->off_merge + (int64_t)plan->n_merge * (int64_t)sizeof(MergeGroup),
      plan->off_part_o + plan->partial_rows * D64 * 4,
      plan->off_part_lse + plan->partial_rows * 4};
  for (int64_t e : ends)
    if (e > plan->ws_bytes) return CP_ERR_INVALID_ARG;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* base = static_cast<uint8_t*>(ws);
  AttnArgs a;
  a.prefill = reinterpret_cast<const PrefillRec*>(base + plan->off_prefill);
  a.n_prefill_items = plan->n_prefill_items;
  a.prefill_wide = reinterpret_cast<const PrefillRec*>(base + plan->off_prefill_wide);
  a.n_prefill_wide_items = plan->n_prefill_wide_items;
  a.decode = reinterpret_cast<const DecodeItem*>(base + plan->off_decode);
  a.n_decode = plan->n_decode;
  a.decode_in_prefill = plan->decode_in_prefill;
  a.merge = reinterpret_cast<const MergeGroup*>(base + plan->off_merge);
  a.n_merge = plan->n_merge;
  a.q = static_cast<const uint16_t*>(q);
  a.k_cache = static_cast<const uint16_t*>(k_cache);
  a.v_cache = static_cast<const uint16_t*>(v_cache);
  a.bt = block_tables;
  a.out = static_cast<uint16_t*>(out);
  a.part_o = reinterpret_cast<float*>(base + plan->off_part_o);
  a.part_lse = reinterpret_cast<float*>(base + plan->off_part_lse);
  a.hq = desc->num_q_heads;
  a.hkv = desc->num_kv_heads;
  a.block_size = desc->block_size;
  a.mbr = desc->max_blocks_per_req;
  a.scale_log2 = desc->sm_scale * 1.4426950408889634f;
  const int D = desc->head_dim;
  const int G = desc->num_q_heads / desc->num_kv_heads;
  int rc = CP_OK;
  if (a.n_prefill_items > 0 || a.n_prefill_wide_items > 0) {
    const long pi = prof_open(1, s);
    const hipError_t e = launch_prefill(D, G, a, s);
    prof_close(pi, s);
    rc = finish(e, s);
    if (rc != CP_OK) return rc;
  }
  if (a.n_decode > 0 && a.decode_in_prefill == 0) {
    const long pi = prof_open(2, s);
    const hipError_t e = launch_decode(D, desc->block_size, G, a, s);
    prof_close(pi, s);
    rc = finish(e, s);
    if (rc != CP_OK) return rc;
  }
  if (a.n_merge > 0) {
    const long pi = prof_open(3, s);
    const hipError_t e = launch_merge(D, G, a, s);
    prof_close(pi, s);
    rc = finish(e, s);
    if (rc != CP_OK) return rc;
  }
  return CP_OK;
}

int cp_attn_mixed(const cp_attn_desc* desc, const void* q, const void* k_cache,
                  const void* v_cache, const int32_t* block_tables, const cp_row_meta* rows,
                  int32_t n_rows, void* out, void* ws, size_t ws_bytes, void* stream) {
  const int v = validate(desc, rows, n_rows);
  if (v != CP_OK) return v;
  if (total_tokens(rows, n_rows) == 0) return CP_OK;
  if (!q || !k_cache || !v_cache || !block_tables || !out || !ws) return CP_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16) ||
      !aligned(ws, 256) || !aligned(block_tables, 4))
    return CP_ERR_INVALID_ARG;
  if (debug_mode()) {
    const int rc = debug_check_tables(desc, block_tables, rows, n_rows,
                                      reinterpret_cast<hipStream_t>(stream));
    if (rc != CP_OK) return rc;
  }
  cp_attn_plan plan;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Stage* st = nullptr;
  const int rc = prepare_impl(desc, rows, n_rows, ws, ws_bytes, s, &plan, &st);
  if (rc != CP_OK) {
    (void)release_stage(st, s);
    return rc;
  }
  const int rr = cp_attn_run(&plan, q, k_cache, v_cache, block_tables, out, ws, ws_bytes, stream);
  const int rs = release_stage(st, s);
  return rr != CP_OK ? rr : rs;
}

int cp_step_mixed(const cp_attn_desc* desc, const void* q, const void* k_new, const void* v_new,
                  void* k_cache, void* v_cache, const int32_t* block_tables,
                  const cp_row_meta* rows, int32_t n_rows, void* out, void* ws, size_t ws_bytes,
                  void* stream) {
  const int v = validate(desc, rows, n_rows);
  if (v != CP_OK) return v;
  const int64_t tokens = total_tokens(rows, n_rows);
  if (tokens == 0) return CP_OK;
  if (!q || !k_new || !v_new || !k_cache || !v_cache || !block_tables || !out || !ws)
    return CP_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_cache, 16) ||
      !aligned(v_cache, 16) || !aligned(out, 16) || !aligned(ws, 256) || !aligned(block_tables, 4))
    return CP_ERR_INVALID_ARG;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  try {
    AppendPlan& ap = thread_append_plan();
    build_append_plan(*desc, rows, n_rows, ap);
    if (ap.items.size() > (size_t)kAppendInlineItems) {
      // a long span list is uploaded itself: the two calls in turn
      const int ra = cp_kv_append(desc, k_new, v_new, k_cache, v_cache, block_tables, rows,
                                  n_rows, ws, ws_bytes, stream);
      if (ra != CP_OK) return ra;
      return cp_attn_mixed(desc, q, k_cache, v_cache, block_tables, rows, n_rows, out, ws,
                           ws_bytes, stream);
    }
    if (debug_mode()) {
      const int rc = debug_check_tables(desc, block_tables, rows, n_rows, s);
      if (rc != CP_OK) return rc;
    }
    Plan& p = thread_plan();
    build_plan(*desc, rows, n_rows, tuning_from_env(num_cus_setting()), p);
    if (ws_bytes < p.ws_bytes) return CP_ERR_WORKSPACE;
    Stage* st = nullptr;
    uint32_t seq = 0;
    int rc = take_stage(p.plan_bytes, &st, &seq, [&](uint8_t* h) { serialize_into(p, h); });
    if (rc != CP_OK) return rc;
    thread_local AppendInline inl;
    std::memcpy(inl.items, ap.items.data(), ap.items.size() * sizeof(AppendItem));
    AppendArgs a;
    a.items = nullptr;
    a.n_items = (int)ap.items.size();
    a.k_new = static_cast<const uint16_t*>(k_new);
    a.v_new = static_cast<const uint16_t*>(v_new);
    a.k_cache = static_cast<uint16_t*>(k_cache);
    a.v_cache = static_cast<uint16_t*>(v_cache);
    a.bt = block_tables;
    a.hkv = desc->num_kv_heads;
    a.mbr = desc->max_blocks_per_req;
    PlanCopyArgs cpa;
    cpa.src = static_cast<const uint4*>(st->dev);
    cpa.dst = static_cast<uint4*>(ws);
    cpa.n16 = (int)(p.plan_bytes / 16);
    cpa.done = st->done_dev;
    cpa.seq = seq;
    cpa.n_blocks = std::min(kCopyBlocksMax, (cpa.n16 + 8 * 256 - 1) / (8 * 256));
    const long pi = prof_open(0, s);
    const hipError_t e = launch_append_copy(desc->head_dim, desc->block_size, a, inl, cpa, s);
    prof_close(pi, s);
    if (e == hipSuccess) {  // the slot's completion words now belong to this copy
      st->seq = seq;
      st->blocks = cpa.n_blocks;
    }
    rc = finish(e, s);
    if (rc == CP_OK) {
      cp_attn_plan pl{};
      pl.desc = *desc;
      pl.tokens = tokens;
      fill_plan(p, pl);
      rc = cp_attn_run(&pl, q, k_cache, v_cache, block_tables, out, ws, ws_bytes, stream);
    }
    const int rs = release_stage(st, s);
    return rc != CP_OK ? rc : rs;
  } catch (...) {
    return CP_ERR_INVALID_ARG;
  }
}

int cp_noalloc_init(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  int err = CP_OK;
  DeviceCtx* c = device_ctx(&err);
  if (!c) return err;
  if (c->scratch_dev) return CP_OK;
  for (Stage& st : c->noalloc_ring) {
    const int rc = stage_reserve(st, CP_NOALLOC_PLAN_BYTES);
    if (rc != CP_OK) return rc;
  }
  void* addr = nullptr;
  if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || !addr) return CP_ERR_HIP;
  if (!aligned(addr, 256)) return CP_ERR_HIP;
  c->scratch_dev = static_cast<uint8_t*>(addr);
  return CP_OK;
}

int cp_attn_mixed_noalloc(const cp_attn_desc* desc, const void* q, const void* k_cache,
                          const void* v_cache, const int32_t* block_tables,
                          const cp_row_meta* rows, int32_t n_rows, void* out, void* stream) {
  const int v = validate(desc, rows, n_rows);
  if (v != CP_OK) return v;
  cp_attn_plan pl{};
  pl.desc = *desc;
  pl.tokens = total_tokens(rows, n_rows);
  if (pl.tokens == 0) return CP_OK;
  if (!q || !k_cache || !v_cache || !block_tables || !out) return CP_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16) ||
      !aligned(block_tables, 4))
    return CP_ERR_INVALID_ARG;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  try {
    // plan first: the size limits are host-side facts, checked before the
    // device is touched
    Plan& p = thread_plan();
    build_plan(*desc, rows, n_rows, tuning_from_env(num_cus_setting()), p);
    if (p.ws_bytes > CP_NOALLOC_SCRATCH_BYTES || p.plan_bytes > CP_NOALLOC_PLAN_BYTES)
      return CP_ERR_WORKSPACE;
    fill_plan(p, pl);
    uint8_t* ws = nullptr;
    Stage* st = nullptr;
    {
      std::lock_guard<std::mutex> lk(g_mu);
      int err = CP_OK;
      DeviceCtx* c = device_ctx(&err);
      if (!c) return err;
      if (!c->scratch_dev) return CP_ERR_INVALID_ARG;  // cp_noalloc_init not called here
      if (debug_mode()) {
        const int rc = debug_check_tables(desc, block_tables, rows, n_rows, s);
        if (rc != CP_OK) return rc;
      }
      ws = c->scratch_dev;
      const int rc = upload_noalloc(c, ws, p, s, &st);
      if (rc != CP_OK) return rc;
    }
    const int rr = cp_attn_run(&pl, q, k_cache, v_cache, block_tables, out, ws,
                               CP_NOALLOC_SCRATCH_BYTES, stream);
    const int rs = release_stage(st, s);
    return rr != CP_OK ? rr : rs;
  } catch (...) {
    return CP_ERR_INVALID_ARG;
  }
}

int cp_profile_begin(void) {
  g_prof.used = 0;
  g_prof.on = true;
  return CP_OK;
}

int cp_profile_end(double ms[4], int64_t launches[4]) {
  if (!ms || !launches) return CP_ERR_INVALID_ARG;
  for (int k = 0; k < 4; ++k) {
    ms[k] = 0.0;
    launches[k] = 0;
  }
  g_prof.on = false;
  for (size_t i = 0; i < g_prof.used; ++i) {
    ProfPair& p = g_prof.pool[i];
    if (hipEventSynchronize(p.b) != hipSuccess) return CP_ERR_HIP;
    float t = 0.f;
    if (hipEventElapsedTime(&t, p.a, p.b) != hipSuccess) return CP_ERR_HIP;
    ms[p.kind] += t;
    launches[p.kind] += 1;
  }
  g_prof.used = 0;
  return CP_OK;
}

}  // extern "C"
