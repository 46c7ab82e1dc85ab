// Batched / prefill expert path (moe_grouped.hip): tokens grouped by expert,
// then MFMA grouped GEMMs over int4 weights streamed through LDS and
// dequantized to fp16 in registers.
#pragma once

#include "moe_device.h"

namespace moe {

constexpr int kGroupRows = 64;   // permuted rows per tile (4 MFMA row blocks of 16)
constexpr int kGroupMaxR = 16;   // LoRA rank the grouped path supports
constexpr int kGroupMaxG = 2048; // experts + shared experts the permutation handles
constexpr int kGroupSlab = 64;   // columns of one partial A_d h (one gate/up workgroup)

// One tile of the grouped GEMMs: rows [row0, row0 + nrows) of the permuted
// list, all routed to group g (expert id g < E, shared expert E + s), whose
// bundle sits in slot `slot` (-1: not resident). The bundle's pointers are
// copied into the record (zero when not resident), so that a GEMM workgroup
// can start its weight copies as soon as it has read its record.
struct GroupTile {
  int32_t g, row0, nrows, slot;
  moe_bundle b;
};

struct GroupedArgs {
  int T, d, I, E, K, S, r, n_list, n_ids;
  float lora_scale;
  const __half* x;              // [T][d]
  const int32_t* idx;           // [T][K]
  const int32_t* slot_of;       // [n_ids] of this layer
  const moe_bundle* bundles;    // [n_slots] of this layer
  uint32_t* status;             // may be null
  // workspace
  int32_t* perm;                // [T * n_list]: y_experts row (t * n_list + k) of each position
  GroupTile* tiles;             // [max_tiles]
  int32_t* tile_tok;            // [max_tiles][kGroupRows]: token of each tile row (unset
                                // past nrows)
  int32_t* n_tiles;             // [1]
  int max_tiles;
  __half* h;                    // [T * n_list][I], by permuted position, pair order
  __half* xp;                   // [T][d]: x in pair order
  float* ax;                    // [T * n_list][4][2][16]: A_g x, A_u x by permuted position,
                                // per quarter of d
  float* adp;                   // [T * n_list][I / kGroupSlab][16]: A_d h over column slabs
  float* y_experts;             // [T][n_list][d]
};

// Upper bound on the tiles of T tokens: sum over groups of ceil(m_g / 64).
inline int grouped_max_tiles(int T, int n_list, int groups) {
  return (T * n_list + kGroupRows - 1) / kGroupRows + groups;
}

bool grouped_shape_supported(int d, int I, int r, int groups);
hipError_t launch_grouped_ffn(const GroupedArgs& a, hipStream_t st);

}  // namespace moe
