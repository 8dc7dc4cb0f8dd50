// Fused path: one wavefront decodes one whole word, every layer, in one launch.
//
// Shapes: d = 32, 8 heads of 4, d_ff = 128, L = n + m <= 64 tokens, n <= 64.  A word's
// tokens fill NT = ceil(L / 16) tiles of 16 token "slots"; the host orders tokens by
// attention work so that the 16 lanes of a tile run neighbour loops of similar length.
//
// The linear maps run transposed on v_mfma_i32_16x16x32_i8: the ternary weights are the A
// operand (16 output features x 32 inputs) and 16 tokens are the columns, so lane
// (c = lane & 15, g = lane >> 4) owns token slot c of a tile and, for every map, a fixed
// set of 4 (per 16-feature output tile) of that token's features.  The host permutes the
// rows and input slots of every packed weight fragment so that
//   - the outputs feeding a LayerNorm (attention output projection, second FFN map) land
//     with feature 4 v + g in register v (v = 0..7): the pairwise feature sum is three
//     in-lane levels (v strides 4, 2, 1) then lane xor 32 and lane xor 16;
//   - the int8 codes a lane produces are exactly the B-operand bytes of the next map
//     (input slot 8 g + e of a 32-input step), so activations never leave registers;
//   - the query, key and value outputs of lane group g are the 4 dims of head g (first
//     16 features) or head 4 + g (second 16).
// Queries stay in registers; keys and values of one head group (4 heads) at a time go to
// a per-wave LDS buffer that the neighbour loops gather from.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "aecct_internal.h"
#include "device_common.h"

namespace aecct {



struct FusedArgs {
  const uint16_t *frag;        // [N][FRAGS][64] 2-bit codes
  const float *vec;            // [N][VEC]
  const uint32_t *nbr;         // neighbour entries, uint16 byte offsets, four per lane and group
  int nbr_words;
  const uint32_t *slot_tab;    // [16 NT][2]: start | count << 16, first / second ring
  const uint32_t *tile_tab;    // [NT][2]: longest list T of the tile, per head group
  const uint64_t *chk;         // [m] variable bitmask of each check
  const int32_t *slot_token;   // [16 NT] token of each slot or -1
  const float *eperm, *pperm;  // [16 NT][4][8] embedding (and positional) rows in lane order
  const float *w1perm;         // [4][8]
  float b1;
  const float *wo, *bo;        // [L][n], [n]
  const float *y;
  uint8_t *bits;
  float *logits;
  int64_t words;
  int n, m, L, N, hf;
  float eps;
  int off_vec, off_nbr, off_slot, off_chk, off_tok, off_kv, kv_bytes;
};

namespace {

// Butterfly steps across lane xor 32 and lane xor 16 through ds_bpermute (the LDS crossbar;
// measured faster here than the gfx950 lane-swap instructions).  Sum and maximum commute, so
// both lanes of a pair get the same bits.
// v of lane (this lane xor M), M = 16 or 32: a whole-wave permute, byte address 4 (lane ^ M)
template <int M>
__device__ __forceinline__ uint32_t lane_xor(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_ds_bpermute((int)(((__builtin_amdgcn_workitem_id_x() & 63u) ^ M) << 2), (int)v);
}
__device__ __forceinline__ float pair_sum32(float v) {
  return v + __builtin_bit_cast(float, lane_xor<32>(__builtin_bit_cast(uint32_t, v)));
}
__device__ __forceinline__ float pair_sum16(float v) {
  return v + __builtin_bit_cast(float, lane_xor<16>(__builtin_bit_cast(uint32_t, v)));
}
__device__ __forceinline__ uint32_t pair_max32(uint32_t v) { return max(v, lane_xor<32>(v)); }
__device__ __forceinline__ uint32_t pair_max16(uint32_t v) { return max(v, lane_xor<16>(v)); }

// Pairwise sum over a token's 32 features held as x[v] = feature 4 v + g.
__device__ __forceinline__ float token_sum(const float (&x)[8]) {
  float u[8];
#pragma unroll
  for (int v = 0; v < 8; ++v) u[v] = x[v];
  return pair_sum16(pair_sum32(lane_tree<8>(u)));
}

// Maximum of non-negative values across lane xor 32 and lane xor 16: for non-negative
// floats the bit patterns order like unsigned integers.
__device__ __forceinline__ float cross_max_nonneg(float a) {
  return __builtin_bit_cast(float, pair_max16(pair_max32(__builtin_bit_cast(uint32_t, a))));
}

__device__ __forceinline__ float token_max_abs(const float (&x)[8]) {
  float a = fabsf(x[0]);
#pragma unroll
  for (int v = 1; v < 8; ++v) a = fmaxf(a, fabsf(x[v]));
  return cross_max_nonneg(a);
}

// Byte 0 of four Eq. 2 code patterns into one dword (byte i from b[i]).
__device__ __forceinline__ uint32_t pack4(uint32_t b0, uint32_t b1, uint32_t b2, uint32_t b3) {
  const uint32_t lo = __builtin_amdgcn_perm(b1, b0, 0x0c0c0400u);
  const uint32_t hi = __builtin_amdgcn_perm(b3, b2, 0x0c0c0400u);
  return __builtin_amdgcn_perm(hi, lo, 0x05040100u);
}

// Eq. 2 over a token's 32 values held 8 per lane; returns alpha, writes the 8 codes
// (value v in byte v) to two dwords.
__device__ __forceinline__ float quant8(const float (&x)[8], uint32_t &lo, uint32_t &hi) {
  const float a = token_max_abs(x);
  const float inv = inv127(a);
  lo = pack4(quant_bits(x[0], inv), quant_bits(x[1], inv), quant_bits(x[2], inv), quant_bits(x[3], inv));
  hi = pack4(quant_bits(x[4], inv), quant_bits(x[5], inv), quant_bits(x[6], inv), quant_bits(x[7], inv));
  return a;
}

// LayerNorm of a token's 32 features (x[v] = feature 4 v + g), gain / offset in lane order.
__device__ __forceinline__ void token_layernorm(float (&x)[8], const float *gp, const float *bp, float eps) {
  const float mean = token_sum(x) / 32.0f;
  float e[8], sq[8];
#pragma unroll
  for (int v = 0; v < 8; ++v) {
    e[v] = x[v] - mean;
    sq[v] = e[v] * e[v];
  }
  const float var = token_sum(sq) / 32.0f;
  const float rho = ln_rsqrt(var + eps);
#pragma unroll
  for (int v = 0; v < 8; ++v) x[v] = __builtin_fmaf(e[v] * rho, gp[v], bp[v]);
}

__device__ __forceinline__ long as_long(uint32_t lo, uint32_t hi) { return (long)(((uint64_t)hi << 32) | lo); }

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Neighbour lists: q is the lane's scaled query; ent its entries (byte offsets of the
// neighbours' key rows in ascending token order), four to a lane per 8-byte group: entry e
// at ent[64 (e / 4) + e % 4], so the 16 lanes of a head read 128 consecutive bytes per
// group; kbase is this lane's head in the key buffer, values vofs bytes after the keys.
__device__ __forceinline__ float4 lds_row(const unsigned char *p) { return *(const float4 *)p; }

// One neighbour of the base-2 softmax (Section 4.2): score DOT(q', k), its weight
// 2^(s - shift), and the running sums S and acc (ascending neighbours).
__device__ __forceinline__ void attend_step(const float (&q)[4], float4 k, float4 vv, float shift, float &S,
                                            float (&acc)[4]) {
  const float kk[4] = {k.x, k.y, k.z, k.w};
  const float ex = softmax_exp2(head_dot<4>(q, kk) - shift);
  S = S + ex;
  acc[0] = __builtin_fmaf(ex, vv.x, acc[0]);
  acc[1] = __builtin_fmaf(ex, vv.y, acc[1]);
  acc[2] = __builtin_fmaf(ex, vv.z, acc[2]);
  acc[3] = __builtin_fmaf(ex, vv.w, acc[3]);
}

// Attention of one lane's (token, head) row over its cnt neighbours, all lanes of the tile
// running T (the tile's longest list) steps, a group of four entries at a time with the
// next group's entries read ahead.  Entries past a lane's list point at the head's pad row
// (key NaN, value 0): its weight is 2^-125 (the clamp maps the NaN score to -125) and its
// value 0, so acc is unchanged and S too whenever S >= 2^-64, the only case in which the
// unshifted sums are kept; a row whose sum leaves [2^-64, 2^64] is redone over its real
// entries with the scores shifted by their maximum.
// The first neighbour starts the sums: S = e and acc = e v (the same values as 0 + e and
// fma(e, v, 0), up to the sign of a zero acc, which no later step or Eq. 2 code can observe).
__device__ __forceinline__ void attend_first(const float (&q)[4], float4 k, float4 vv, float &S, float (&acc)[4]) {
  const float kk[4] = {k.x, k.y, k.z, k.w};
  const float ex = softmax_exp2(head_dot<4>(q, kk));
  S = ex;
  acc[0] = ex * vv.x;
  acc[1] = ex * vv.y;
  acc[2] = ex * vv.z;
  acc[3] = ex * vv.w;
}

__device__ __forceinline__ void attend_tile(const float (&q)[4], const uint16_t *ent, int cnt, int T,
                                            const unsigned char *kbase, int vofs, float (&o)[4]) {
  float S, acc[4];
  const uint2 *eg = (const uint2 *)ent;
  const int G = T >> 2;
  uint2 nx = eg[0];
  if (G > 0) {                        // the first group, its first entry starting the sums
    const uint32_t e0 = nx.x & 0xffffu, e1 = nx.x >> 16, e2 = nx.y & 0xffffu, e3 = nx.y >> 16;
    const float4 k0 = lds_row(kbase + e0), v0 = lds_row(kbase + vofs + e0);
    const float4 k1 = lds_row(kbase + e1), v1 = lds_row(kbase + vofs + e1);
    const float4 k2 = lds_row(kbase + e2), v2 = lds_row(kbase + vofs + e2);
    const float4 k3 = lds_row(kbase + e3), v3 = lds_row(kbase + vofs + e3);
    nx = eg[16];
    attend_first(q, k0, v0, S, acc);
    attend_step(q, k1, v1, 0.0f, S, acc);
    attend_step(q, k2, v2, 0.0f, S, acc);
    attend_step(q, k3, v3, 0.0f, S, acc);
  } else {                            // T = 1..3 (T >= 1): the first remainder entry starts them
    const uint32_t e0 = nx.x & 0xffffu;
    attend_first(q, lds_row(kbase + e0), lds_row(kbase + vofs + e0), S, acc);
  }
  for (int u = 1; u < G; ++u) {
    const uint32_t e0 = nx.x & 0xffffu, e1 = nx.x >> 16, e2 = nx.y & 0xffffu, e3 = nx.y >> 16;
    const float4 k0 = lds_row(kbase + e0), v0 = lds_row(kbase + vofs + e0);
    const float4 k1 = lds_row(kbase + e1), v1 = lds_row(kbase + vofs + e1);
    const float4 k2 = lds_row(kbase + e2), v2 = lds_row(kbase + vofs + e2);
    const float4 k3 = lds_row(kbase + e3), v3 = lds_row(kbase + vofs + e3);
    nx = eg[16 * (u + 1)];          // in the table: every list has a group past its end
    attend_step(q, k0, v0, 0.0f, S, acc);
    attend_step(q, k1, v1, 0.0f, S, acc);
    attend_step(q, k2, v2, 0.0f, S, acc);
    attend_step(q, k3, v3, 0.0f, S, acc);
  }
  const int rem = T & 3;              // the last, partial group is already in nx
  if (rem > 0 && G > 0) {             // (with no full group, its first entry started the sums)
    const uint32_t e0 = nx.x & 0xffffu;
    attend_step(q, lds_row(kbase + e0), lds_row(kbase + vofs + e0), 0.0f, S, acc);
  }
  if (rem > 1) {
    const uint32_t e1 = nx.x >> 16;
    attend_step(q, lds_row(kbase + e1), lds_row(kbase + vofs + e1), 0.0f, S, acc);
  }
  if (rem > 2) {
    const uint32_t e2 = nx.y & 0xffffu;
    attend_step(q, lds_row(kbase + e2), lds_row(kbase + vofs + e2), 0.0f, S, acc);
  }
  if (cnt > 0 && !(S >= 0x1p-64f && S <= 0x1p64f)) {
    float mu = -INFINITY;
    for (int i = 0; i < cnt; ++i) {
      const float4 k = lds_row(kbase + ent[64 * (i >> 2) + (i & 3)]);
      const float kk[4] = {k.x, k.y, k.z, k.w};
      mu = fmaxf(mu, head_dot<4>(q, kk));
    }
    S = 0.0f;
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = 0.0f;
    for (int i = 0; i < cnt; ++i) {
      const uint32_t e = ent[64 * (i >> 2) + (i & 3)];
      attend_step(q, lds_row(kbase + e), lds_row(kbase + vofs + e), mu, S, acc);
    }
  }
  const float rS = cnt > 0 ? recip_softmax_sum(S) : 0.0f;
#pragma unroll
  for (int t = 0; t < 4; ++t) o[t] = acc[t] * rS;
}

}  // namespace

template <int NT, int WAVES>
__global__ __launch_bounds__(WAVES * 64, 1) void k_fused_decode(FusedArgs p) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  // ---- one-time staging: packed ternary fragments -> int8, per-layer vectors, tables ----
  {
    uint64_t *sf = (uint64_t *)smem;
    const int nf = p.N * fz::FRAGS * 64;
    for (int u = tid; u < nf; u += nthr) sf[u] = unpack_ternary8(p.frag[u]);
    float *sv = (float *)(smem + p.off_vec);
    for (int u = tid; u < p.N * fz::VEC; u += nthr) sv[u] = p.vec[u];
    uint32_t *sn = (uint32_t *)(smem + p.off_nbr);
    for (int u = tid; u < p.nbr_words; u += nthr) sn[u] = p.nbr[u];
    uint32_t *ss = (uint32_t *)(smem + p.off_slot);
    for (int u = tid; u < 32 * NT; u += nthr) ss[u] = p.slot_tab[u];
    uint64_t *sc = (uint64_t *)(smem + p.off_chk);
    for (int u = tid; u < p.m; u += nthr) sc[u] = p.chk[u];
    int32_t *st = (int32_t *)(smem + p.off_tok);
    for (int u = tid; u < 16 * NT; u += nthr) st[u] = p.slot_token[u];
  }
  __syncthreads();

  const int lane = tid & 63, c = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), nw = nthr >> 6;   // uniform: scalar
  const uint64_t *sfrag = (const uint64_t *)smem;
  const float *svec = (const float *)(smem + p.off_vec);
  const uint16_t *snbr = (const uint16_t *)(smem + p.off_nbr);
  const uint32_t *sslot = (const uint32_t *)(smem + p.off_slot);
  const uint64_t *schk = (const uint64_t *)(smem + p.off_chk);
  const int32_t *stok = (const int32_t *)(smem + p.off_tok);
  // Keys (then values) of the current head group, head-major: head h of slot s at
  // (h * 16 NT + s) * 16 bytes, so the 16 lanes of one head gather from all banks.
  unsigned char *kv = smem + p.off_kv + wave * p.kv_bytes;
  constexpr int HS = (16 * NT + 1) * 16;   // one head: 16 NT slot rows and the pad row
  const int vofs = 4 * HS;                 // values follow the keys of all four heads
  unsigned char *kbase = kv + g * HS;
  if (lane < 4) {                          // pad rows of the four heads: key NaN, value 0
    *(float4 *)(kv + lane * HS + 16 * NT * 16) = make_float4(__builtin_nanf(""), __builtin_nanf(""),
                                                             __builtin_nanf(""), __builtin_nanf(""));
    *(float4 *)(kv + vofs + lane * HS + 16 * NT * 16) = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  }
  const int mask1 = g < p.hf ? 0 : 1, mask2 = 4 + g < p.hf ? 0 : 1;

  // Words in rounds of one per wave, consecutive words to the waves of one block (their y rows and
  // outputs adjacent in memory).  The last, partial round goes to the lowest-numbered waves of
  // every block (q or q + 1 per block), one per SIMD, rather than to every wave of the first
  // blocks: no SIMD then runs more than one word above the others.  v runs over the rounds
  // wave-major, which selects exactly those waves for the last round; w is the word it stands for.
  // (32-bit indices: the launcher passes at most 2^31 - 1 words per launch.)
  const uint32_t words = (uint32_t)p.words, wt = gridDim.x * (uint32_t)nw, full = words / wt;
  const uint32_t rq = (words - full * wt) / gridDim.x, rr = words - full * wt - rq * gridDim.x;
  const uint32_t last_w = full * wt + blockIdx.x * rq + min(blockIdx.x, rr) + (uint32_t)wave;
  uint32_t base = blockIdx.x * (uint32_t)nw + (uint32_t)wave;
  for (uint32_t v = (uint32_t)wave * gridDim.x + blockIdx.x; v < words; v += wt, base += wt) {
    const int64_t w = base < full * wt ? base : last_w;
    // Per-word copy of the lane index: the addresses of the embedding and head steps derive
    // from it, so they are recomputed per word rather than held through the layers.
    int lw = lane;
    asm volatile("" : "+v"(lw));
    const int cw = lw & 15, gw = lw >> 4;
    int tok[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) tok[t] = stok[16 * t + cw];
    // ---- pre-processing h(y) (Section 3) and embedding ----
    const float *yw = p.y + w * p.n;
    const float ylane = lw < p.n ? yw[lw] : 0.0f;
    const uint64_t neg = __ballot(ylane < 0.0f);
    float X[NT][8], al[NT];
    uint32_t xb[NT][2];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int tk = tok[t];
      const float yv = __builtin_bit_cast(
          float, __builtin_amdgcn_ds_bpermute(((tk >= 0 && tk < p.n) ? tk : 0) << 2, __builtin_bit_cast(int, ylane)));
      float tv = 0.0f;
      if (tk >= 0) {
        if (tk < p.n) {
          tv = fabsf(yv);
        } else {
          const int s = __builtin_popcountll(neg & schk[tk - p.n]) & 1;
          tv = s ? -1.0f : 1.0f;
        }
      }
      const float4 *er = (const float4 *)(p.eperm + ((16 * t + cw) * 4 + gw) * 8);
      const float4 e0 = er[0], e1 = er[1];
      const float ev[8] = {e0.x, e0.y, e0.z, e0.w, e1.x, e1.y, e1.z, e1.w};
      float pv[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      if (p.pperm) {
        const float4 *pr = (const float4 *)(p.pperm + ((16 * t + cw) * 4 + gw) * 8);
        const float4 p0 = pr[0], p1 = pr[1];
        pv[0] = p0.x; pv[1] = p0.y; pv[2] = p0.z; pv[3] = p0.w;
        pv[4] = p1.x; pv[5] = p1.y; pv[6] = p1.z; pv[7] = p1.w;
      }
#pragma unroll
      for (int v = 0; v < 8; ++v) X[t][v] = __builtin_fmaf(tv, ev[v], pv[v]);
      al[t] = quant8(X[t], xb[t][0], xb[t][1]);
    }

    for (int l = 0; l < p.N; ++l) {
      const uint64_t *F = sfrag + l * fz::FRAGS * 64 + lane;
      const float *V = svec + l * fz::VEC;
      const float sq_q = V[fz::V_SQ + 0], sq_k = V[fz::V_SQ + 1], sq_v = V[fz::V_SQ + 2];
      const float sq_o = V[fz::V_SQ + 3], sq_1 = V[fz::V_SQ + 4], sq_2 = V[fz::V_SQ + 5];
      // ---- per head group (heads g, then 4 + g): queries, keys, values (Eq. 3) of that
      // group, keys and values to LDS, then head-partitioned attention (Section 4.2) ----
      float ob[NT][8];
#pragma unroll
      for (int grp = 0; grp < 2; ++grp) {
        // keys and values of every tile to LDS; queries are made per tile just before use
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const long bop = as_long(xb[t][0], xb[t][1]);
          const v4i ak = mfma_i8_16x16x32((long)F[(2 + grp) * 64], bop, v4i{0, 0, 0, 0});
          const v4i av = mfma_i8_16x16x32((long)F[(4 + grp) * 64], bop, v4i{0, 0, 0, 0});
          const float sck = al[t] * sq_k, scv = al[t] * sq_v;
          const float *bq = V + fz::V_BQKV + 16 * grp + 4 * g;
          float kk[4], vv[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            kk[i] = __builtin_fmaf((float)ak[i], sck, bq[32 + i]);
            vv[i] = __builtin_fmaf((float)av[i], scv, bq[64 + i]);
          }
          *(float4 *)(kbase + (16 * t + c) * 16) = make_float4(kk[0], kk[1], kk[2], kk[3]);
          *(float4 *)(kbase + vofs + (16 * t + c) * 16) = make_float4(vv[0], vv[1], vv[2], vv[3]);
        }
        wave_sync_lds();
        const int mask = grp == 0 ? mask1 : mask2;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const v4i aq =
              mfma_i8_16x16x32((long)F[(0 + grp) * 64], as_long(xb[t][0], xb[t][1]), v4i{0, 0, 0, 0});
          const float scq = al[t] * sq_q;
          const float *bq = V + fz::V_BQKV + 16 * grp + 4 * g;
          float q[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) q[i] = __builtin_fmaf((float)aq[i], scq, bq[i]);
          const uint32_t st = sslot[(16 * t + c) * 2 + mask];
          const int T = (int)__builtin_amdgcn_readfirstlane(p.tile_tab[2 * t + grp]);
          float o[4];
          attend_tile(q, snbr + (st & 0xffff), (int)(st >> 16), T, kbase, vofs, o);
#pragma unroll
          for (int i = 0; i < 4; ++i) ob[t][4 * grp + i] = o[i];
        }
        wave_sync_lds();
      }
      // ---- output projection, residual, LN1 (Section 6), Eq. 2 ----
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        uint32_t lo, hi;
        const float ao = quant8(ob[t], lo, hi);
        const long bop = as_long(lo, hi);
        const v4i a0 = mfma_i8_16x16x32((long)F[fz::F_O * 64], bop, v4i{0, 0, 0, 0});
        const v4i a1 = mfma_i8_16x16x32((long)F[(fz::F_O + 1) * 64], bop, v4i{0, 0, 0, 0});
        const float sc = ao * sq_o;
        const float *bo = V + fz::V_BO + 4 * g;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          X[t][i] = X[t][i] + __builtin_fmaf((float)a0[i], sc, bo[i]);
          X[t][4 + i] = X[t][4 + i] + __builtin_fmaf((float)a1[i], sc, bo[16 + i]);
        }
        token_layernorm(X[t], V + fz::V_LN1G + 8 * g, V + fz::V_LN1B + 8 * g, p.eps);
        al[t] = quant8(X[t], xb[t][0], xb[t][1]);
      }
      // ---- feed-forward block with ReLU, residual, LN2, Eq. 2 ----
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const long bop = as_long(xb[t][0], xb[t][1]);
        v4i acc[8];
#pragma unroll
        for (int o = 0; o < 8; ++o) acc[o] = mfma_i8_16x16x32((long)F[(fz::F_FF1 + o) * 64], bop, v4i{0, 0, 0, 0});
        const float sc = al[t] * sq_1;
        // F1 pre-activations; the ReLU is applied to the maximum (max(0, F...)) and to the codes
        float G[8][4];
        float amax = 0.0f;
#pragma unroll
        for (int o = 0; o < 8; ++o)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            G[o][i] = __builtin_fmaf((float)acc[o][i], sc, V[fz::V_BFF1 + 16 * o + 4 * g + i]);
            amax = fmaxf(amax, G[o][i]);
          }
        amax = cross_max_nonneg(amax + 0.0f);   // + 0 turns a -0 maximum into +0
        const float inv = inv127(amax);
        uint32_t gb[8];
#pragma unroll
        for (int o = 0; o < 8; ++o)
          gb[o] = pack4_relu(quant_bits(G[o][0], inv), quant_bits(G[o][1], inv), quant_bits(G[o][2], inv),
                             quant_bits(G[o][3], inv));
        const auto gop = [&](int s) { return as_long(gb[2 * s], gb[2 * s + 1]); };
        const v4i b0 = mfma_i8_steps<4>([&](int s) { return (long)F[(fz::F_FF2 + s) * 64]; }, gop, v4i{0, 0, 0, 0});
        const v4i b1 = mfma_i8_steps<4>([&](int s) { return (long)F[(fz::F_FF2 + 4 + s) * 64]; }, gop, v4i{0, 0, 0, 0});
        const float sc2 = amax * sq_2;
        const float *b2 = V + fz::V_BFF2 + 4 * g;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          X[t][i] = X[t][i] + __builtin_fmaf((float)b0[i], sc2, b2[i]);
          X[t][4 + i] = X[t][4 + i] + __builtin_fmaf((float)b1[i], sc2, b2[16 + i]);
        }
        token_layernorm(X[t], V + fz::V_LN2G + 8 * g, V + fz::V_LN2B + 8 * g, p.eps);
        al[t] = quant8(X[t], xb[t][0], xb[t][1]);
      }
    }

    // ---- output head and hard decision (Section 3) ----
    float *zbuf = (float *)kv;
    int lh = lane;
    asm volatile("" : "+v"(lh));
    {
      const float4 *wr = (const float4 *)(p.w1perm + 8 * (lh >> 4));
      const float4 w0 = wr[0], w1 = wr[1];
      const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        float pr[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) pr[v] = X[t][v] * wv[v];
        const float z = token_sum(pr) + p.b1;
        const int tk = stok[16 * t + (lh & 15)];
        if (lh < 16 && tk >= 0) zbuf[tk] = z;
      }
    }
    wave_sync_lds();
    if (lh < p.n) {
      float acc = 0.0f;
      for (int i = 0; i < p.L; ++i) acc = __builtin_fmaf(zbuf[i], p.wo[(int64_t)i * p.n + lh], acc);
      const float f = acc + p.bo[lh];
      p.bits[w * p.n + lh] = (uint8_t)((ylane < 0.0f) != (f < 0.0f));
      if (p.logits) p.logits[w * p.n + lh] = f;
    }
    wave_sync_lds();
  }
}

// ------------------------------------------------------------------------------------------
// host-side launcher
// ------------------------------------------------------------------------------------------

int fused_tiles(const Model &M) { return (M.L + 15) / 16; }

// LDS layout of one block: fragments, vectors, neighbour entries, slot table, check
// masks, slot tokens (all shared), then one key/value buffer per wave.
struct FusedLds {
  int off_vec, off_nbr, off_slot, off_chk, off_tok, off_kv, kv_bytes;
};

FusedLds fused_lds(const Model &M, int nbr_words) {
  const int NT = fused_tiles(M);
  FusedLds L{};
  size_t off = (size_t)M.n_layers * fz::FRAGS * 64 * 8;
  L.off_vec = (int)off;
  off += (size_t)M.n_layers * fz::VEC * 4;
  off = (off + 7) / 8 * 8;                    // 8-byte entry groups
  L.off_nbr = (int)off;
  off += (size_t)nbr_words * 4;
  L.off_slot = (int)off;
  off += (size_t)32 * NT * 4;
  off = (off + 7) / 8 * 8;
  L.off_chk = (int)off;
  off += (size_t)M.m * 8;
  L.off_tok = (int)off;
  off += (size_t)16 * NT * 4;
  off = (off + 15) / 16 * 16;
  L.off_kv = (int)off;
  L.kv_bytes = 2 * 4 * (16 * NT + 1) * 16;   // keys and values, 4 heads, 16 NT slots + pad row
  return L;
}

bool fused_supported(const Model &M) {
  return M.d == 32 && M.heads == 8 && M.dff == 128 && M.L <= 64 && M.n <= 64;
}

// Words in flight per block: kWaves, or as many as the LDS holds when the tables are larger
// (at least 4, one per SIMD); 0 if not even that fits.  The kernel is compiled for kWaves
// wavefronts (its register budget), and runs with any smaller count.
int fused_waves(const Model &M, int nbr_words) {
  const FusedLds L = fused_lds(M, nbr_words);
  const size_t lds_max = std::min<size_t>(M.lds_max, fz::kLdsMax);
  if ((size_t)L.off_kv >= lds_max) return 0;
  const int fit = (int)((lds_max - (size_t)L.off_kv) / (size_t)L.kv_bytes);
  const int w = fit < fz::kWaves ? fit : fz::kWaves;
  return w >= 4 ? w : 0;
}

bool fused_fits(const Model &M, int nbr_words) { return fused_waves(M, nbr_words) > 0; }

// The largest dynamic LDS the fused kernel may use on the model's device, set once per model at
// create time (the launches only choose a size within it).
hipError_t set_fused_kernel_attributes(const Model &M) {
  const void *fns[] = {(const void *)k_fused_decode<1, fz::kWaves>, (const void *)k_fused_decode<2, fz::kWaves>,
                       (const void *)k_fused_decode<3, fz::kWaves>, (const void *)k_fused_decode<4, fz::kWaves>};
  const int lds = (int)std::min<size_t>(M.lds_max, fz::kLdsMax);
  for (const void *f : fns) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <int NT, int WAVES>
static hipError_t launch_nt(const FusedArgs &a, size_t lds, int grid, int waves, hipStream_t s) {
  hipLaunchKernelGGL((k_fused_decode<NT, WAVES>), dim3(grid), dim3(waves * 64), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_fused(const Model &M, const float *y, int64_t words, uint8_t *bits, float *logits,
                        hipStream_t s) {
  if (words <= 0) return hipSuccess;
  constexpr int64_t kMaxWords = INT32_MAX;   // the kernel's word indices are 32-bit
  if (words > kMaxWords) {
    for (int64_t w0 = 0; w0 < words; w0 += kMaxWords) {
      const int64_t nw = std::min(kMaxWords, words - w0);
      const hipError_t e = launch_fused(M, y + w0 * M.n, nw, bits + w0 * M.n, logits ? logits + w0 * M.n : nullptr, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  const FusedTables &T = M.fused;
  const int NT = fused_tiles(M);
  FusedArgs a{};
  a.frag = T.frag;
  a.vec = T.vec;
  a.nbr = T.nbr;
  a.nbr_words = T.nbr_words;
  a.slot_tab = T.slot_tab;
  a.tile_tab = T.tile_tab;
  a.chk = T.chk;
  a.slot_token = T.slot_token;
  a.eperm = T.eperm;
  a.pperm = T.pperm;
  a.w1perm = T.w1perm;
  a.b1 = M.head_b1;
  a.wo = M.head_wo;
  a.bo = M.head_bo;
  a.y = y;
  a.bits = bits;
  a.logits = logits;
  a.words = words;
  a.n = M.n;
  a.m = M.m;
  a.L = M.L;
  a.N = M.n_layers;
  a.hf = M.hf;
  a.eps = M.eps;
  const FusedLds Ld = fused_lds(M, T.nbr_words);
  a.off_vec = Ld.off_vec;
  a.off_nbr = Ld.off_nbr;
  a.off_slot = Ld.off_slot;
  a.off_chk = Ld.off_chk;
  a.off_tok = Ld.off_tok;
  a.off_kv = Ld.off_kv;
  a.kv_bytes = Ld.kv_bytes;
  const size_t off = (size_t)Ld.off_kv;
  const int waves = fused_waves(M, T.nbr_words);
  const size_t lds_max = std::min<size_t>(M.lds_max, fz::kLdsMax);
  if (waves < 1 || waves > fz::kWaves || off + (size_t)waves * a.kv_bytes > lds_max)
    return hipErrorInvalidConfiguration;
  const size_t lds = off + (size_t)waves * a.kv_bytes;
  int64_t blocks = (words + waves - 1) / waves;
  const int64_t per_cu = (int64_t)(lds_max / lds) > 0 ? (int64_t)(lds_max / lds) : 1;
  const int64_t cap = (int64_t)M.cu_count * per_cu;
  const int grid = (int)(blocks < cap ? blocks : cap);
  switch (NT) {
    case 1: return launch_nt<1, fz::kWaves>(a, lds, grid, waves, s);
    case 2: return launch_nt<2, fz::kWaves>(a, lds, grid, waves, s);
    case 3: return launch_nt<3, fz::kWaves>(a, lds, grid, waves, s);
    case 4: return launch_nt<4, fz::kWaves>(a, lds, grid, waves, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace aecct
