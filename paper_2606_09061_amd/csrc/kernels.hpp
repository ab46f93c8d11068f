// Launch interface between the host API and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.hpp"

namespace cpattn {

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
  const PrefillItem* prefill;       // 128-row tiles (4-wave kernel)
  int n_prefill;
  const PrefillItem* prefill_wide;  // 256-row tiles (8-wave kernel)
  int n_prefill_wide;
  const DecodeItem* decode;
  int n_decode;
  const MergeGroup* merge;
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

hipError_t launch_append(int D, int B, const AppendArgs& a, hipStream_t s);
hipError_t launch_prefill(int D, int G, const AttnArgs& a, hipStream_t s);
hipError_t launch_decode(int D, int B, int G, const AttnArgs& a, hipStream_t s);
hipError_t launch_merge(int D, int G, const AttnArgs& a, hipStream_t s);

}  // namespace cpattn
