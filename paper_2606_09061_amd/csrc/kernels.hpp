// Launch interface between the host API and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.hpp"

namespace cpattn {

// Append plans of up to kAppendInlineItems items travel inside the kernel
// arguments (3.2 KB), so a small append needs no plan upload.
constexpr int kAppendInlineItems = 200;
struct AppendInline {
  AppendItem items[kAppendInlineItems];
};

struct AppendArgs {
  const AppendItem* items;
  int n_items;
  const uint16_t* k_new;
  const uint16_t* v_new;
  uint16_t* k_cache;
  uint16_t* v_cache;
  const int32_t* bt;
  int hkv, mbr;
};

struct AttnArgs {
  const PrefillRec* prefill;        // 128-row tiles (4-wave kernel): one record per workgroup
  int n_prefill_items;
  const PrefillRec* prefill_wide;   // 256-row tiles (8-wave kernel)
  int n_prefill_wide_items;
  const DecodeItem* decode;         // grid (n_decode, hkv), or units of a prefill launch
  int n_decode;
  int decode_in_prefill;            // 0: own launch; 1 / 2: inside the 128- / 256-row launch
  const MergeGroup* merge;          // grid (n_merge, hkv)
  int n_merge;
  const uint16_t* q;
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int32_t* bt;
  uint16_t* out;
  float* part_o;
  float* part_lse;
  int hq, hkv, block_size, mbr;
  float scale_log2;  // sm_scale * log2(e)
};

// A staged plan's copy: n16 16-byte words from src (pinned host memory) to
// dst by n_blocks workgroups, each writing seq to done[its index] at the end.
struct PlanCopyArgs {
  const uint4* src;
  uint4* dst;
  int n16;
  uint32_t* done;
  uint32_t seq;
  int n_blocks;
};

// `inl` non-null: the items are taken from it (a.n_items <= kAppendInlineItems)
// and a.items is ignored.
hipError_t launch_append(int D, int B, const AppendArgs& a, const AppendInline* inl,
                         hipStream_t s);
// the inline append and a plan copy in one launch (256-thread workgroups)
hipError_t launch_append_copy(int D, int B, const AppendArgs& a, const AppendInline& inl,
                              const PlanCopyArgs& cp, hipStream_t s);
hipError_t launch_prefill(int D, int G, const AttnArgs& a, hipStream_t s);
hipError_t launch_decode(int D, int B, int G, const AttnArgs& a, hipStream_t s);
hipError_t launch_merge(int D, int G, const AttnArgs& a, hipStream_t s);

}  // namespace cpattn
