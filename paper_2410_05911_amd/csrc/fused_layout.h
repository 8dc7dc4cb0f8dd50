// Layout of the fused path's per-layer tables (d = 32, one wavefront per word) and the device
// tables a model holds for it; shared by its host packing and its kernel.
#pragma once

#include <cstdint>

namespace aecct {

// Per-layer layout of the fused path's tables (d = 32, d_ff = 128).
namespace fz {
constexpr int D = 32;
constexpr int DFF = 128;
constexpr int FRAGS = 24;      // MFMA A fragments per layer: qkv 6, o 2, ff1 8, ff2 2 x 4
constexpr int F_O = 6, F_FF1 = 8, F_FF2 = 16;
constexpr int VEC = 424;       // floats per layer
constexpr int V_BQKV = 0, V_BO = 96, V_BFF1 = 128, V_BFF2 = 256, V_LN1G = 288, V_LN1B = 320, V_LN2G = 352,
              V_LN2B = 384, V_SQ = 416;
// wavefronts (words in flight) per block: 12 of 168 registers each fill the register file; blocks
// of 8 or 10 waves were measured 18 % slower on BCH(31,16)
constexpr int kWaves = 12;
constexpr int kLdsMax = 160 * 1024;   // the kernel's design limit: gfx950's LDS per workgroup
}  // namespace fz

// Tables of the fused path (one wavefront per word), built at create time when the
// shape allows it; see kernel_fused.hip for the lane layout they encode.
struct FusedTables {
  bool ready;
  const uint16_t *frag;        // [N][24][64] 2-bit MFMA A-operand fragments, permuted rows / inputs
  const float *vec;            // [N][424] biases, LayerNorm parameters and scales in lane order
  const uint32_t *nbr;         // neighbour entries (uint16 byte offsets into a wave's key buffer)
  int nbr_words;               // 32-bit words of nbr (a multiple of 4)
  const uint32_t *slot_tab;    // [16 NT][2] start | count << 16 per slot, first / second ring
  const uint32_t *tile_tab;    // [NT][2] longest list T of the tile, per head group
  const uint64_t *chk;         // [m] bitmask of the variables of each check
  const int32_t *slot_token;   // [16 NT] token in each slot, -1 for padding
  const float *eperm, *pperm;  // [16 NT][4][8] embedding / positional rows in lane order
  const float *w1perm;         // [4][8] W_{d->1} in lane order
};

}  // namespace aecct
