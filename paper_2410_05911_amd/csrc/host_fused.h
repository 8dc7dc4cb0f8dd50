// Host packing of the fused path (d = 32, one wavefront per word): token tiles, neighbour
// tables and permuted weight fragments, built at create time from the Tanner-graph lists and the
// model's weights.
#pragma once

#include <cstdint>
#include <vector>

#include "../../include/aecct.h"
#include "aecct_internal.h"

namespace aecct {

// 2-bit code of a ternary value: 00 -> 0, 01 -> +1, 11 -> -1.
inline uint16_t code2(int8_t v) { return v == 1 ? 1u : (v == -1 ? 3u : 0u); }

// Host image of the fused path's tables.  Lane layout (see kernel_fused.hip): lane group g
// of token slot c holds, for maps feeding a LayerNorm, feature 16 o + 4 i + g in register
// v = 4 o + i; the query / key / value maps are unpermuted (row r of output tile o is
// feature 16 o + r); an input step's slot 8 g + e carries the feature the producing lane
// group g keeps in its register e.
struct FusedImage {
  std::vector<uint16_t> frag;
  std::vector<float> vec;
  std::vector<uint16_t> nbr;
  std::vector<uint32_t> slot_tab;
  std::vector<uint32_t> tile_tab;
  std::vector<uint64_t> chk;
  std::vector<int32_t> slot_token;
  std::vector<float> eperm, pperm, w1perm;
};

// Token slots of NT tiles of 16 minimising the padded neighbour-loop steps, given each token's
// loop length per head group; returns the token of each slot (-1 for padding).
std::vector<int32_t> fused_tile_partition(int L, int NT, const std::vector<int> &w0, const std::vector<int> &w1);

// The fused path's tables of model M (its shape, head split and per-map scales already set) for
// parity-check matrix H, weights w and the first- and second-ring lists (CSR).
void build_fused(const Model &M, const uint8_t *H, const aecct_weights *w, const std::vector<int32_t> &m1_ptr,
                 const std::vector<int32_t> &m1_idx, const std::vector<int32_t> &m2_ptr,
                 const std::vector<int32_t> &m2_idx, FusedImage &F);

}  // namespace aecct
