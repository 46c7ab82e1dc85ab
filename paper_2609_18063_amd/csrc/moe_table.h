// Host object behind moe_slot_table (include/moe_api.h), shared by the C ABI
// and the host-tier stager.
#pragma once

#include <hip/hip_runtime.h>

#include <vector>

#include "../../include/moe_api.h"

struct moe_slot_table {
  int n_layers = 0, n_ids = 0, n_slots = 0;
  std::vector<int32_t> slot_of;      // [L][n_ids], -1 = not resident
  std::vector<int32_t> expert_in;    // [L][n_slots], -1 = free
  std::vector<moe_bundle> bundles;   // [L][n_slots]
  // device copy: [slot_of | pad | bundles] in one allocation
  void* dev = nullptr;
  size_t dev_bytes = 0, bundles_off = 0;
  void* pinned = nullptr;
  hipEvent_t copied = nullptr;
  bool copy_pending = false;
};
