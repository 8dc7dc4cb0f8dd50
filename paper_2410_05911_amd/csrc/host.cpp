// Host side of the C ABI: argument validation, Tanner-graph neighbour lists, packing
// of the ternary weights into MFMA B fragments, the single device allocation of a
// model, workspace layout, and the launch sequence of a decode.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <iterator>
#include <mutex>
#include <new>
#include <vector>

#include <hip/hip_runtime.h>

#include "../../include/aecct.h"
#include "aecct_internal.h"
#include "host_fused.h"

using aecct::Model;
using aecct::code2;
using aecct::FusedImage;
using aecct::build_fused;

struct aecct_model {
  Model M;
};

// ---- static scratch of aecct_decode_static -----------------------------------------------
// The layered decode's workspace for callers that cannot allocate: one array per GPU the library
// runs on, held until the process ends.  In host code `scratch` only names the array; its device
// address comes from hipGetSymbolAddress, once per device (each GPU holds its own copy at its own
// address), and is the only form in which it reaches a kernel or a copy.
constexpr size_t kStaticScratchBytes = size_t(256) << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mutex;
unsigned char *g_scratch_ptr[kMaxScratchDevices];   // per device; null until first looked up

// The static scratch's address on device `dev`, which must be current.  Null if it cannot be had
// (a device index beyond the table, or a HIP error); aecct_decode_static then refuses.
unsigned char *static_scratch_address(int dev) {
  if (dev < 0 || dev >= kMaxScratchDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = (unsigned char *)p;
  }
  return g_scratch_ptr[dev];
}
}  // namespace

namespace {

constexpr size_t kAlign = 256;
constexpr size_t kChunkCapBytes = size_t(4) << 30;   // layered workspace per chunk of words

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool finite_all(const float *p, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!std::isfinite(p[i])) return false;
  return true;
}

bool ternary_all(const int8_t *p, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (p[i] < -1 || p[i] > 1) return false;
  return true;
}

// Packs a [K][N] ternary map given by get(k, j) into 16x32 MFMA B-fragment blocks:
// block (t, s) at index t * (K/32) + s, lane l holds column 16t + (l & 15) and inputs
// 32s + 8(l >> 4) + e in bits 2e..2e+1.
template <class Get>
void pack_map(int K, int N, Get get, uint16_t *out) {
  const int S = K / 32, T = N / 16;
  for (int t = 0; t < T; ++t)
    for (int s = 0; s < S; ++s)
      for (int l = 0; l < 64; ++l) {
        uint16_t v = 0;
        const int j = 16 * t + (l & 15);
        for (int e = 0; e < 8; ++e) v |= (uint16_t)(code2(get(32 * s + 8 * (l >> 4) + e, j)) << (2 * e));
        out[((size_t)t * S + s) * 64 + l] = v;
      }
}

size_t packed_words(int K, int N) { return (size_t)(K / 32) * (N / 16) * 64; }

// Device memory plan: byte offsets inside the model's single allocation.
struct Plan {
  size_t chk_ptr, chk_idx, m1_ptr, m1_idx, m2_ptr, m2_idx, embed, pos, embed_lo, pos_lo, w1, w1lo, wo, bo, total;
  size_t g1_meta, g1_tab, g2_meta, g2_tab;   // grouped neighbour lists (layered attention)
  size_t g1s_tab, g2s_tab;                    // the same, counted within each node type
  size_t f_frag, f_vec, f_nbr, f_slot, f_tile, f_chk, f_tok, f_e, f_p, f_w1;
  struct Layer {
    size_t qkv, o, ff1, ff2, b_qkv, b_o, b_ff1, b_ff2, ln1_g, ln1_b, ln2_g, ln2_b;
    size_t tb_o, tb_1, tb_2, tb_vec;   // token-block fragments and lane-order vectors (d = 64, 128), or 0
    size_t qkv_tb;                     // the QKV map reading lane-order codes (d = 64, 128), or 0
  };
  std::vector<Layer> layer;
};

Plan make_plan(int n, int m, int d, int N, int dff, size_t E, size_t nnz1, size_t nnz2, bool has_pos) {
  const int L = n + m;
  Plan p{};
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes); return o; };
  p.chk_ptr = take(sizeof(int32_t) * (m + 1));
  p.chk_idx = take(sizeof(int32_t) * E);
  p.m1_ptr = take(sizeof(int32_t) * (L + 1));
  p.m1_idx = take(sizeof(int32_t) * nnz1);
  p.m2_ptr = take(sizeof(int32_t) * (L + 1));
  p.m2_idx = take(sizeof(int32_t) * nnz2);
  p.embed = take(sizeof(float) * L * d);
  p.pos = has_pos ? take(sizeof(float) * L * d) : 0;
  p.embed_lo = take(sizeof(float) * L * d);
  p.pos_lo = has_pos ? take(sizeof(float) * L * d) : 0;
  p.w1 = take(sizeof(float) * d);
  p.w1lo = take(sizeof(float) * d);
  p.wo = take(sizeof(float) * (size_t)L * n);
  p.bo = take(sizeof(float) * n);
  p.layer.resize(N);
  for (int l = 0; l < N; ++l) {
    auto &q = p.layer[l];
    q.qkv = take(2 * packed_words(d, 3 * d));
    q.o = take(2 * packed_words(d, d));
    q.ff1 = take(2 * packed_words(d, dff));
    q.ff2 = take(2 * packed_words(dff, d));
    q.b_qkv = take(sizeof(float) * 3 * d);
    q.b_o = take(sizeof(float) * d);
    q.b_ff1 = take(sizeof(float) * dff);
    q.b_ff2 = take(sizeof(float) * d);
    q.ln1_g = take(sizeof(float) * d);
    q.ln1_b = take(sizeof(float) * d);
    q.ln2_g = take(sizeof(float) * d);
    q.ln2_b = take(sizeof(float) * d);
    if ((d == 64 || d == 128) && dff == 4 * d) {   // the token block's int8 A fragments
      q.tb_o = take((size_t)d * d);
      q.tb_1 = take((size_t)d * dff);
      q.tb_2 = take((size_t)dff * d);
      q.tb_vec = take(sizeof(float) * 6 * d);
      q.qkv_tb = take(2 * packed_words(d, 3 * d));
    }
  }
  p.total = off;
  return p;
}

// Layered-path workspace for `words` words: region offsets.
struct WsPlan {
  size_t x, xq, ax, qkv, oq, ao, x1, x1q, a1, gq, ag;
  size_t o32, h32;   // fp32 attention output and hidden row (one alpha per word only), or 0
  size_t total;
};

WsPlan ws_plan(const Model &M, int64_t words) {
  const size_t R = (size_t)words * M.L, d = M.d, dff = M.dff;
  // With the token block a layer needs X, its codes, the attention output (fp32 in the qkv region,
  // d wide, from the fused forms that leave it so; the separate GEMM's Q, K, V there, 3 d wide;
  // codes in oq otherwise) and per-token scalars (the head's z in a1, the embedding's t in ag);
  // X1, its codes and the hidden codes stay in the token block's registers.
  const bool tb = !M.act_word && aecct::token_block_supported(M);
  const bool unf = M.lattn == AECCT_LAYERED_ATTN_UNFUSED;
  WsPlan w{};
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes); return o; };
  w.x = take(4 * R * d);
  w.xq = take(R * d);
  w.ax = take(4 * R);
  w.qkv = take(4 * R * (tb && !unf ? 1 : 3) * d);
  w.oq = take(R * d);
  w.ao = take(4 * R);
  w.x1 = take(tb ? 0 : 4 * R * d);
  w.x1q = take(tb ? 0 : R * d);
  w.a1 = take(4 * R);
  w.gq = take(tb ? 0 : R * dff);
  w.ag = take(4 * R);
  if (M.act_word) {
    w.o32 = take(4 * R * d);
    w.h32 = take(4 * R * dff);
  }
  w.total = off;
  return w;
}

// Words per chunk of a layered decode within `cap_bytes` of workspace: the batch in as few
// chunks as fit, as even as possible, each a multiple of the words the attention kernel runs at
// once (one word per block), so that no chunk ends in a round of mostly idle blocks.
int64_t chunk_words_within(const Model &M, int64_t batch, size_t cap_bytes) {
  const size_t per_word = ws_plan(M, 1).total;
  int64_t cap = (int64_t)(cap_bytes / (per_word ? per_word : 1));
  if (cap < 1) cap = 1;
  while (cap > 1 && ws_plan(M, cap).total > cap_bytes) --cap;
  if (batch <= cap) return batch;
  const int64_t slots = aecct::attention_word_slots(M, M.lattn);
  const int64_t nchunks = (batch + cap - 1) / cap;
  int64_t cw = (batch + nchunks - 1) / nchunks;
  if (slots > 1 && cw >= slots) {
    const int64_t up = (cw + slots - 1) / slots * slots;
    cw = up <= cap ? up : cap / slots * slots;
  }
  return std::max<int64_t>(1, std::min<int64_t>(cw, cap));
}

int64_t chunk_words(const Model &M, int64_t batch) { return chunk_words_within(M, batch, kChunkCapBytes); }

// The layered decode's projection + attention form: the requested one if the shape allows it, or
// (AUTO) fused with fp32 keys and values in LDS when a word's fit, else (with the token block,
// which takes O in fp32) int16 accumulators, else rows one node type at a time with that type's
// keys and values in LDS as fp32 (measured no faster than the int16 form on LDPC(1024,512): its
// two phases per head take 3 + 2 row passes of the block where one pass over all rows takes 4),
// else the separate GEMM and attention kernels; the unfused form with one alpha per word.  -1 if
// the requested form does not fit the shape.
int32_t resolve_layered_attention(const Model &M, int requested) {
  const bool tb = aecct::token_block_supported(M);
  const bool f32 = aecct::qkv_attention_supported(M);
  const bool split = tb && aecct::qkv_attention_split_supported(M);
  const bool i16 = tb && aecct::qkv_attention_i16_supported(M);
  switch (requested) {
    case AECCT_LAYERED_ATTN_UNFUSED: return AECCT_LAYERED_ATTN_UNFUSED;
    case AECCT_LAYERED_ATTN_LDS_F32: return f32 && !M.act_word ? AECCT_LAYERED_ATTN_LDS_F32 : -1;
    case AECCT_LAYERED_ATTN_LDS_I16: return i16 && !M.act_word ? AECCT_LAYERED_ATTN_LDS_I16 : -1;
    case AECCT_LAYERED_ATTN_LDS_SPLIT: return split && !M.act_word ? AECCT_LAYERED_ATTN_LDS_SPLIT : -1;
  }
  if (M.act_word) return AECCT_LAYERED_ATTN_UNFUSED;
  if (f32) return AECCT_LAYERED_ATTN_LDS_F32;
  if (i16) return AECCT_LAYERED_ATTN_LDS_I16;
  return split ? AECCT_LAYERED_ATTN_LDS_SPLIT : AECCT_LAYERED_ATTN_UNFUSED;
}

aecct_status from_hip(hipError_t e) {
  if (e == hipSuccess) return AECCT_OK;
  return e == hipErrorOutOfMemory ? AECCT_ERR_OUT_OF_MEMORY : AECCT_ERR_DEVICE;
}

}  // namespace

namespace aecct {

// Tanner graph lists and HPSA masks (Section 4.2): M1 = neighbours, M2 = nodes two steps away
// plus the node itself; each list ascending.
TannerLists tanner_lists(const uint8_t *H, int m, int n) {
  const int L = n + m;
  TannerLists T;
  std::vector<std::vector<int>> adj(L);
  T.chk_ptr.assign(m + 1, 0);
  for (int j = 0; j < m; ++j) {
    for (int i = 0; i < n; ++i)
      if (H[(size_t)j * n + i]) {
        T.chk_idx.push_back(i);
        adj[i].push_back(n + j);
        adj[n + j].push_back(i);
      }
    T.chk_ptr[j + 1] = (int32_t)T.chk_idx.size();
  }
  T.m1_ptr.assign(L + 1, 0);
  T.m2_ptr.assign(L + 1, 0);
  std::vector<int> mark(L, -1);
  for (int a = 0; a < L; ++a) {
    std::vector<int> nb = adj[a];
    std::sort(nb.begin(), nb.end());
    for (int v : nb) T.m1_idx.push_back(v);
    T.m1_ptr[a + 1] = (int32_t)T.m1_idx.size();
    for (int k : adj[a])
      for (int b : adj[k]) mark[b] = a;
    for (int b = 0; b < L; ++b)
      if (mark[b] == a) T.m2_idx.push_back(b);
    T.m2_ptr[a + 1] = (int32_t)T.m2_idx.size();
  }
  return T;
}

// The ECCT mask of every head under CASA (Section 3): the second-ring lists become the merged,
// ascending union of both rings.
void casa_union(TannerLists &T) {
  const int L = (int)T.m1_ptr.size() - 1;
  std::vector<int32_t> u_ptr(L + 1, 0), u_idx;
  u_idx.reserve(T.m1_idx.size() + T.m2_idx.size());
  for (int a = 0; a < L; ++a) {
    std::merge(T.m1_idx.begin() + T.m1_ptr[a], T.m1_idx.begin() + T.m1_ptr[a + 1], T.m2_idx.begin() + T.m2_ptr[a],
               T.m2_idx.begin() + T.m2_ptr[a + 1], std::back_inserter(u_idx));
    u_ptr[a + 1] = (int32_t)u_idx.size();
  }
  T.m2_ptr.swap(u_ptr);
  T.m2_idx.swap(u_idx);
}

}  // namespace aecct

extern "C" {

const char *aecct_status_string(aecct_status s) {
  switch (s) {
    case AECCT_OK: return "ok";
    case AECCT_ERR_INVALID_ARG: return "invalid argument";
    case AECCT_ERR_UNSUPPORTED: return "unsupported model shape";
    case AECCT_ERR_OUT_OF_MEMORY: return "out of memory";
    case AECCT_ERR_DEVICE: return "device error";
    case AECCT_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
  }
  return "unknown status";
}

aecct_status aecct_create(const uint8_t *H, int32_t m, int32_t n, const aecct_weights *w, int32_t d,
                          int32_t n_layers, int32_t heads, const aecct_options *opt, aecct_model **out) {
  if (!out) return AECCT_ERR_INVALID_ARG;
  *out = nullptr;
  if (!H || !w || m <= 0 || n <= 0 || d <= 0 || n_layers <= 0 || heads <= 0 || d % heads) return AECCT_ERR_INVALID_ARG;
  const int hf = (opt && opt->first_ring_heads >= 0) ? opt->first_ring_heads : heads / 2;
  if (opt && opt->first_ring_heads < -1) return AECCT_ERR_INVALID_ARG;
  if (hf > heads) return AECCT_ERR_INVALID_ARG;
  const int dff = (opt && opt->d_ff > 0) ? opt->d_ff : 4 * d;
  if (opt && opt->d_ff < -1) return AECCT_ERR_INVALID_ARG;
  const float eps = (opt && opt->ln_eps > 0.0f) ? opt->ln_eps : 1e-5f;
  if (opt && !std::isfinite(opt->ln_eps)) return AECCT_ERR_INVALID_ARG;
  const int path_req = opt ? opt->path : AECCT_PATH_AUTO;
  if (path_req < AECCT_PATH_AUTO || path_req > AECCT_PATH_FUSED) return AECCT_ERR_INVALID_ARG;
  const int attention = opt ? opt->attention : AECCT_ATTN_HPSA;
  if (attention != AECCT_ATTN_HPSA && attention != AECCT_ATTN_CASA) return AECCT_ERR_INVALID_ARG;
  const int lattn_req = opt ? opt->layered_attention : AECCT_LAYERED_ATTN_AUTO;
  if (lattn_req < AECCT_LAYERED_ATTN_AUTO || lattn_req > AECCT_LAYERED_ATTN_LDS_SPLIT) return AECCT_ERR_INVALID_ARG;
  const int act_mode = opt ? opt->act_scale_mode : AECCT_ACT_SCALE_TOKEN;
  if (act_mode != AECCT_ACT_SCALE_TOKEN && act_mode != AECCT_ACT_SCALE_WORD) return AECCT_ERR_INVALID_ARG;
  const int64_t L64 = (int64_t)n + m;
  if (L64 > (1 << 20)) return AECCT_ERR_UNSUPPORTED;
  const int L = (int)L64;
  // parity-check matrix: 0/1, no empty row or column
  std::vector<int> rowdeg(m, 0), coldeg(n, 0);
  size_t E = 0;
  for (int j = 0; j < m; ++j)
    for (int i = 0; i < n; ++i) {
      const uint8_t h = H[(size_t)j * n + i];
      if (h > 1) return AECCT_ERR_INVALID_ARG;
      if (h) { ++rowdeg[j]; ++coldeg[i]; ++E; }
    }
  for (int j = 0; j < m; ++j) if (!rowdeg[j]) return AECCT_ERR_INVALID_ARG;
  for (int i = 0; i < n; ++i) if (!coldeg[i]) return AECCT_ERR_INVALID_ARG;
  // weights
  const size_t N = (size_t)n_layers, D = (size_t)d, F = (size_t)dff;
  const int8_t *wts[6] = {w->w_q, w->w_k, w->w_v, w->w_o, w->w_ff1, w->w_ff2};
  const float *bs[6] = {w->b_q, w->b_k, w->b_v, w->b_o, w->b_ff1, w->b_ff2};
  const size_t wsz[6] = {D * D, D * D, D * D, D * D, D * F, F * D};
  const size_t bsz[6] = {D, D, D, D, F, D};
  if (!w->embed || !w->scale || !w->ln1_g || !w->ln1_b || !w->ln2_g || !w->ln2_b || !w->head_w1 || !w->head_wo ||
      !w->head_bo)
    return AECCT_ERR_INVALID_ARG;
  for (int k = 0; k < 6; ++k) {
    if (!wts[k] || !bs[k]) return AECCT_ERR_INVALID_ARG;
    if (!ternary_all(wts[k], N * wsz[k])) return AECCT_ERR_INVALID_ARG;
    if (!finite_all(bs[k], N * bsz[k])) return AECCT_ERR_INVALID_ARG;
  }
  if (!finite_all(w->embed, (size_t)L * D) || (w->pos && !finite_all(w->pos, (size_t)L * D)) ||
      !finite_all(w->scale, N * 6) || !finite_all(w->ln1_g, N * D) || !finite_all(w->ln1_b, N * D) ||
      !finite_all(w->ln2_g, N * D) || !finite_all(w->ln2_b, N * D) || !finite_all(w->head_w1, D) ||
      !std::isfinite(w->head_b1) || !finite_all(w->head_wo, (size_t)L * n) || !finite_all(w->head_bo, (size_t)n))
    return AECCT_ERR_INVALID_ARG;
  // shapes the kernels implement
  const int dh = d / heads;
  if (!(d == 32 || d == 64 || d == 128) || !(dh == 4 || dh == 8 || dh == 16) || dff != 4 * d || L > 4096 ||
      n_layers > aecct::kMaxLayers)
    return AECCT_ERR_UNSUPPORTED;
  // one alpha per word: the unfused layered form with natural layouts only
  if (act_mode == AECCT_ACT_SCALE_WORD &&
      (path_req == AECCT_PATH_FUSED || lattn_req == AECCT_LAYERED_ATTN_LDS_F32 || lattn_req == AECCT_LAYERED_ATTN_LDS_I16 ||
       lattn_req == AECCT_LAYERED_ATTN_LDS_SPLIT))
    return AECCT_ERR_UNSUPPORTED;

  aecct::TannerLists TL = aecct::tanner_lists(H, m, n);
  std::vector<int32_t> &chk_ptr = TL.chk_ptr, &chk_idx = TL.chk_idx, &m1_ptr = TL.m1_ptr, &m1_idx = TL.m1_idx,
                       &m2_ptr = TL.m2_ptr, &m2_idx = TL.m2_idx;

  Model M{};
  M.n = n; M.m = m; M.L = L; M.d = d; M.n_layers = n_layers; M.heads = heads; M.hf = hf; M.dff = dff;
  M.dh = dh; M.eps = eps;
  M.kq = (float)(1.4426950408889634074 / std::sqrt((double)dh));
  M.nnz1 = (int64_t)m1_idx.size();
  M.nnz2 = (int64_t)m2_idx.size();
  M.attention = attention;
  if (attention == AECCT_ATTN_CASA) {
    // every head reads the union of the two rings: it takes the second-ring list slot, h_f = 0
    aecct::casa_union(TL);
    M.hf = 0;
  }
  M.head_b1 = w->head_b1;
  for (int l = 0; l < n_layers; ++l) {
    for (int k = 0; k < 6; ++k) M.layer[l].sq[k] = w->scale[(size_t)l * 6 + k] / 127.0f;
    M.layer[l].sq_qs = M.layer[l].sq[0] * M.kq;
  }
  M.path = path_req;
  M.act_word = act_mode == AECCT_ACT_SCALE_WORD ? 1 : 0;
  M.grouped = L <= 65535;

  // the device: every table and launch below is sized for its compute units and LDS
  int dev = 0, cus = 0, lds = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || cus <= 0 ||
      lds <= 0)
    return AECCT_ERR_DEVICE;
  M.device = dev;
  M.cu_count = cus;
  M.lds_max = (size_t)lds;
  if (aecct::set_layered_kernel_attributes(M) != hipSuccess || aecct::set_fused_kernel_attributes(M) != hipSuccess)
    return AECCT_ERR_DEVICE;
  M.static_scratch = static_scratch_address(dev);

  // fused-path tables (built whenever the shape allows the fused kernel)
  FusedImage FI;
  bool fused_ok = path_req != AECCT_PATH_LAYERED && !M.act_word && aecct::fused_supported(M);
  if (fused_ok) {
    build_fused(M, H, w, m1_ptr, m1_idx, m2_ptr, m2_idx, FI);
    // list starts are 16-bit entry indices
    fused_ok = FI.nbr.size() <= 65536 && aecct::fused_fits(M, (int)(FI.nbr.size() / 2));
    if (!fused_ok) FI = FusedImage();
  }
  if (M.path == AECCT_PATH_AUTO) M.path = fused_ok ? AECCT_PATH_FUSED : AECCT_PATH_LAYERED;
  if (M.path == AECCT_PATH_FUSED && !fused_ok) return AECCT_ERR_UNSUPPORTED;

  // Neighbour lists in groups of four 16-bit token indices for the layered attention: token a's
  // list starts at group meta[2a] and has meta[2a + 1] entries; floor(cnt / 4) + 1 groups are
  // stored, so the group after the last full one can always be read (its unused slots hold 0).
  std::vector<int32_t> G1m, G2m;
  std::vector<uint16_t> G1, G2;
  auto group_lists = [&](const std::vector<int32_t> &ptr, const std::vector<int32_t> &idx,
                         std::vector<int32_t> &meta, std::vector<uint16_t> &tab) {
    meta.assign(2 * (size_t)L, 0);
    for (int a = 0; a < L; ++a) {
      const int cnt = ptr[a + 1] - ptr[a];
      meta[2 * a] = (int32_t)(tab.size() / 4);
      meta[2 * a + 1] = cnt;
      const int slots = 4 * (cnt / 4 + 1);
      for (int e = 0; e < slots; ++e) tab.push_back(e < cnt ? (uint16_t)idx[ptr[a] + e] : 0);
    }
  };
  if (M.grouped) {
    group_lists(m1_ptr, m1_idx, G1m, G1);
    group_lists(m2_ptr, m2_idx, G2m, G2);
  }
  // Under head partitioning every list holds one node type (first ring: the other type; second
  // ring: its own): the same lists counted from the first token of that type.
  std::vector<uint16_t> G1s, G2s;
  if (M.grouped && attention == AECCT_ATTN_HPSA) {
    auto rebase = [&](const std::vector<uint16_t> &tab) {
      std::vector<uint16_t> r(tab.size());
      for (size_t e = 0; e < tab.size(); ++e) r[e] = tab[e] >= n ? (uint16_t)(tab[e] - n) : tab[e];
      return r;
    };
    // every entry of a token's list must be of the node type that list reads (the Tanner graph is
    // bipartite: first-ring neighbours are of the other type, second-ring ones of the same type)
    bool one_type = true;
    for (int a = 0; a < L; ++a) {
      const bool var = a < n;
      for (int32_t e = m1_ptr[a]; e < m1_ptr[a + 1]; ++e) one_type &= (m1_idx[e] < n) != var;
      for (int32_t e = m2_ptr[a]; e < m2_ptr[a + 1]; ++e) one_type &= (m2_idx[e] < n) == var;
    }
    if (one_type) {
      G1s = rebase(G1);
      G2s = rebase(G2);
    }
  }

  // host image of the device block
  Plan P = make_plan(n, m, d, n_layers, dff, E, m1_idx.size(), m2_idx.size(), w->pos != nullptr);
  {
    size_t off = P.total;
    auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes); return o; };
    P.f_frag = take(2 * FI.frag.size());
    P.f_vec = take(4 * FI.vec.size());
    P.f_nbr = take(2 * FI.nbr.size());
    P.f_slot = take(4 * FI.slot_tab.size());
    P.f_tile = take(4 * FI.tile_tab.size());
    P.f_chk = take(8 * FI.chk.size());
    P.f_tok = take(4 * FI.slot_token.size());
    P.f_e = take(4 * FI.eperm.size());
    P.f_p = take(4 * FI.pperm.size());
    P.f_w1 = take(4 * FI.w1perm.size());
    P.g1_meta = take(8 * (size_t)L);
    P.g1_tab = take(2 * G1.size());
    P.g2_meta = take(8 * (size_t)L);
    P.g2_tab = take(2 * G2.size());
    P.g1s_tab = take(2 * G1s.size());
    P.g2s_tab = take(2 * G2s.size());
    P.total = off;
  }
  std::vector<unsigned char> img;
  try {
    img.assign(P.total, 0);
  } catch (const std::bad_alloc &) {
    return AECCT_ERR_OUT_OF_MEMORY;
  }
  auto put = [&](size_t off, const void *src, size_t bytes) { if (bytes) std::memcpy(img.data() + off, src, bytes); };
  put(P.chk_ptr, chk_ptr.data(), 4 * chk_ptr.size());
  put(P.chk_idx, chk_idx.data(), 4 * chk_idx.size());
  put(P.m1_ptr, m1_ptr.data(), 4 * m1_ptr.size());
  put(P.m1_idx, m1_idx.data(), 4 * m1_idx.size());
  put(P.m2_ptr, m2_ptr.data(), 4 * m2_ptr.size());
  put(P.m2_idx, m2_idx.data(), 4 * m2_idx.size());
  put(P.embed, w->embed, 4 * (size_t)L * D);
  if (w->pos) put(P.pos, w->pos, 4 * (size_t)L * D);
  put(P.w1, w->head_w1, 4 * D);
  {
    // the token block's lane order: [i][g][v] = row_i[4 v + g]
    std::vector<float> lo((size_t)L * D);
    auto to_lo = [&](const float *src, size_t off) {
      for (size_t i = 0; i < (size_t)L; ++i)
        for (size_t g = 0; g < 4; ++g)
          for (size_t v = 0; v < D / 4; ++v) lo[i * D + g * (D / 4) + v] = src[i * D + 4 * v + g];
      put(off, lo.data(), 4 * (size_t)L * D);
    };
    to_lo(w->embed, P.embed_lo);
    if (w->pos) to_lo(w->pos, P.pos_lo);
  }
  {
    std::vector<float> w1lo(D);   // [g][v] = W_{d->1}[4 v + g]
    for (size_t g = 0; g < 4; ++g)
      for (size_t v = 0; v < D / 4; ++v) w1lo[g * (D / 4) + v] = w->head_w1[4 * v + g];
    put(P.w1lo, w1lo.data(), 4 * D);
  }
  put(P.wo, w->head_wo, 4 * (size_t)L * n);
  put(P.bo, w->head_bo, 4 * (size_t)n);
  put(P.f_frag, FI.frag.data(), 2 * FI.frag.size());
  put(P.f_vec, FI.vec.data(), 4 * FI.vec.size());
  put(P.f_nbr, FI.nbr.data(), 2 * FI.nbr.size());
  put(P.f_slot, FI.slot_tab.data(), 4 * FI.slot_tab.size());
  put(P.f_tile, FI.tile_tab.data(), 4 * FI.tile_tab.size());
  put(P.f_chk, FI.chk.data(), 8 * FI.chk.size());
  put(P.f_tok, FI.slot_token.data(), 4 * FI.slot_token.size());
  put(P.f_e, FI.eperm.data(), 4 * FI.eperm.size());
  put(P.f_p, FI.pperm.data(), 4 * FI.pperm.size());
  put(P.f_w1, FI.w1perm.data(), 4 * FI.w1perm.size());
  put(P.g1_meta, G1m.data(), 4 * G1m.size());
  put(P.g1_tab, G1.data(), 2 * G1.size());
  put(P.g2_meta, G2m.data(), 4 * G2m.size());
  put(P.g2_tab, G2.data(), 2 * G2.size());
  put(P.g1s_tab, G1s.data(), 2 * G1s.size());
  put(P.g2s_tab, G2s.data(), 2 * G2s.size());
  for (int l = 0; l < n_layers; ++l) {
    const auto &q = P.layer[l];
    const int8_t *Wq = w->w_q + l * D * D, *Wk = w->w_k + l * D * D, *Wv = w->w_v + l * D * D;
    const int8_t *Wo = w->w_o + l * D * D, *W1 = w->w_ff1 + l * D * F, *W2 = w->w_ff2 + l * F * D;
    pack_map(d, 3 * d, [&](int k, int j) {
      const int8_t *src = j < d ? Wq : (j < 2 * d ? Wk : Wv);
      return src[(size_t)k * D + (j % d)];
    }, (uint16_t *)(img.data() + q.qkv));
    pack_map(d, d, [&](int k, int j) { return Wo[(size_t)k * D + j]; }, (uint16_t *)(img.data() + q.o));
    pack_map(d, dff, [&](int k, int j) { return W1[(size_t)k * F + j]; }, (uint16_t *)(img.data() + q.ff1));
    pack_map(dff, d, [&](int k, int j) { return W2[(size_t)k * D + j]; }, (uint16_t *)(img.data() + q.ff2));
    if (q.qkv_tb) {
      // input slot k of step k / 32 reads the code of feature 32 (k / 32) + 4 (k % 8) + (k % 32) / 8,
      // the byte order in which the token block writes the next layer's codes
      pack_map(d, 3 * d, [&](int k, int j) {
        const int8_t *src = j < d ? Wq : (j < 2 * d ? Wk : Wv);
        const int f = 32 * (k >> 5) + 4 * (k & 7) + ((k & 31) >> 3);
        return src[(size_t)f * D + (j % d)];
      }, (uint16_t *)(img.data() + q.qkv_tb));
    }
    if (q.tb_o) {
      // Token block (transposed products: weights are the A operand, 16 tokens the columns).
      // A fragment (tile t, step s): lane l holds output row l & 15 and k-slots 8 (l >> 4) + e
      // in byte e.  Lane layout of d-wide activations: lane group g holds feature 4 v + g in
      // register v.  O and FF2 output row r of tile t is feature 16 t + 4 (r & 3) + (r >> 2)
      // (lane group g then holds v = 4 t + i); FF1 reads slot k of step s as feature
      // 32 s + 4 (k & 7) + (k >> 3) (the 8 codes lane group g packs for step s); FF1's outputs
      // keep their order and FF2 reads slot k of step s as hidden feature
      // 16 (2 s + ((k & 7) >> 2)) + 4 (k >> 3) + (k & 3).
      auto pack_a = [&](size_t dst, int T, int S, auto get) {
        int8_t *o8 = (int8_t *)(img.data() + dst);
        for (int t = 0; t < T; ++t)
          for (int st = 0; st < S; ++st)
            for (int l = 0; l < 64; ++l)
              for (int e = 0; e < 8; ++e) o8[(((size_t)t * S + st) * 64 + l) * 8 + e] = get(t, st, l & 15, 8 * (l >> 4) + e);
      };
      auto out_x = [](int t, int r) { return 16 * t + 4 * (r & 3) + (r >> 2); };
      auto in_x = [](int st, int k) { return 32 * st + 4 * (k & 7) + (k >> 3); };
      auto in_h = [](int st, int k) { return 16 * (2 * st + ((k & 7) >> 2)) + 4 * (k >> 3) + (k & 3); };
      pack_a(q.tb_o, d / 16, d / 32, [&](int t, int st, int r, int k) { return Wo[(size_t)(32 * st + k) * D + out_x(t, r)]; });
      pack_a(q.tb_1, dff / 16, d / 32, [&](int t, int st, int r, int k) { return W1[(size_t)in_x(st, k) * F + 16 * t + r]; });
      pack_a(q.tb_2, d / 16, dff / 32, [&](int t, int st, int r, int k) { return W2[(size_t)in_h(st, k) * D + out_x(t, r)]; });
      // b_o, ln1_g, ln1_b, b_ff2, ln2_g, ln2_b in lane order: [vector][g][v] = vector[4 v + g]
      float *vx = (float *)(img.data() + q.tb_vec);
      const float *srcs[6] = {w->b_o + l * D, w->ln1_g + l * D, w->ln1_b + l * D, w->b_ff2 + l * D,
                              w->ln2_g + l * D, w->ln2_b + l * D};
      for (int k = 0; k < 6; ++k)
        for (int g = 0; g < 4; ++g)
          for (int v = 0; v < d / 4; ++v) vx[(size_t)k * d + g * (d / 4) + v] = srcs[k][4 * v + g];
    }
    {
      std::vector<float> bqs(D);
      for (size_t c = 0; c < D; ++c) bqs[c] = w->b_q[l * D + c] * M.kq;   // scaled query bias
      put(q.b_qkv, bqs.data(), 4 * D);
    }
    put(q.b_qkv + 4 * D, w->b_k + l * D, 4 * D);
    put(q.b_qkv + 8 * D, w->b_v + l * D, 4 * D);
    put(q.b_o, w->b_o + l * D, 4 * D);
    put(q.b_ff1, w->b_ff1 + l * F, 4 * F);
    put(q.b_ff2, w->b_ff2 + l * D, 4 * D);
    put(q.ln1_g, w->ln1_g + l * D, 4 * D);
    put(q.ln1_b, w->ln1_b + l * D, 4 * D);
    put(q.ln2_g, w->ln2_g + l * D, 4 * D);
    put(q.ln2_b, w->ln2_b + l * D, 4 * D);
  }

  // device
  void *blk = nullptr;
  hipError_t e = hipMalloc(&blk, P.total);
  if (e != hipSuccess) return from_hip(e);
  e = hipMemcpy(blk, img.data(), P.total, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(blk);
    return AECCT_ERR_DEVICE;
  }
  aecct_model *am = new (std::nothrow) aecct_model;
  if (!am) {
    (void)hipFree(blk);
    return AECCT_ERR_OUT_OF_MEMORY;
  }
  unsigned char *b = (unsigned char *)blk;
  M.dev_block = blk;
  M.device_bytes = P.total;
  M.chk_ptr = (const int32_t *)(b + P.chk_ptr);
  M.chk_idx = (const int32_t *)(b + P.chk_idx);
  M.m1_ptr = (const int32_t *)(b + P.m1_ptr);
  M.m1_idx = (const int32_t *)(b + P.m1_idx);
  M.m2_ptr = (const int32_t *)(b + P.m2_ptr);
  M.m2_idx = (const int32_t *)(b + P.m2_idx);
  M.g1_meta = (const int32_t *)(b + P.g1_meta);
  M.g1_tab = (const uint16_t *)(b + P.g1_tab);
  M.g2_meta = (const int32_t *)(b + P.g2_meta);
  M.g2_tab = (const uint16_t *)(b + P.g2_tab);
  M.g1_groups = (int32_t)(G1.size() / 4);
  M.g2_groups = (int32_t)(G2.size() / 4);
  M.g1s_tab = G1s.empty() ? nullptr : (const uint16_t *)(b + P.g1s_tab);
  M.g2s_tab = G2s.empty() ? nullptr : (const uint16_t *)(b + P.g2s_tab);
  M.embed = (const float *)(b + P.embed);
  M.pos = w->pos ? (const float *)(b + P.pos) : nullptr;
  M.head_w1 = (const float *)(b + P.w1);
  M.head_w1_lo = (const float *)(b + P.w1lo);
  M.embed_lo = (const float *)(b + P.embed_lo);
  M.pos_lo = w->pos ? (const float *)(b + P.pos_lo) : nullptr;
  M.head_wo = (const float *)(b + P.wo);
  M.head_bo = (const float *)(b + P.bo);
  for (int l = 0; l < n_layers; ++l) {
    const auto &q = P.layer[l];
    auto &Lw = M.layer[l];
    Lw.qkv = (const uint16_t *)(b + q.qkv);
    Lw.o = (const uint16_t *)(b + q.o);
    Lw.ff1 = (const uint16_t *)(b + q.ff1);
    Lw.ff2 = (const uint16_t *)(b + q.ff2);
    Lw.b_qkv = (const float *)(b + q.b_qkv);
    Lw.b_o = (const float *)(b + q.b_o);
    Lw.b_ff1 = (const float *)(b + q.b_ff1);
    Lw.b_ff2 = (const float *)(b + q.b_ff2);
    Lw.ln1_g = (const float *)(b + q.ln1_g);
    Lw.ln1_b = (const float *)(b + q.ln1_b);
    Lw.ln2_g = (const float *)(b + q.ln2_g);
    Lw.ln2_b = (const float *)(b + q.ln2_b);
    Lw.tb_o = q.tb_o ? (const uint64_t *)(b + q.tb_o) : nullptr;
    Lw.tb_1 = q.tb_1 ? (const uint64_t *)(b + q.tb_1) : nullptr;
    Lw.tb_2 = q.tb_2 ? (const uint64_t *)(b + q.tb_2) : nullptr;
    Lw.tb_vec = q.tb_vec ? (const float *)(b + q.tb_vec) : nullptr;
    Lw.qkv_tb = q.qkv_tb ? (const uint16_t *)(b + q.qkv_tb) : nullptr;
  }
  if (!FI.frag.empty()) {
    aecct::FusedTables &T = M.fused;
    T.ready = true;
    T.frag = (const uint16_t *)(b + P.f_frag);
    T.vec = (const float *)(b + P.f_vec);
    T.nbr = (const uint32_t *)(b + P.f_nbr);
    T.nbr_words = (int)(FI.nbr.size() / 2);
    T.slot_tab = (const uint32_t *)(b + P.f_slot);
    T.tile_tab = (const uint32_t *)(b + P.f_tile);
    T.chk = (const uint64_t *)(b + P.f_chk);
    T.slot_token = (const int32_t *)(b + P.f_tok);
    T.eperm = (const float *)(b + P.f_e);
    T.pperm = FI.pperm.empty() ? nullptr : (const float *)(b + P.f_p);
    T.w1perm = (const float *)(b + P.f_w1);
  }
  // the layered path's projection + attention form
  const int lattn = resolve_layered_attention(M, lattn_req);
  if (lattn < 0) {
    (void)hipFree(blk);
    delete am;
    return AECCT_ERR_UNSUPPORTED;
  }
  M.lattn = lattn;
  am->M = M;
  *out = am;
  return AECCT_OK;
}

void aecct_destroy(aecct_model *model) {
  if (!model) return;
  if (model->M.dev_block) (void)hipFree(model->M.dev_block);
  delete model;
}

aecct_status aecct_get_info(const aecct_model *model, aecct_model_info *info) {
  if (!model || !info) return AECCT_ERR_INVALID_ARG;
  const Model &M = model->M;
  info->n = M.n; info->m = M.m; info->L = M.L; info->d = M.d; info->n_layers = M.n_layers;
  info->heads = M.heads; info->first_ring_heads = M.hf; info->d_ff = M.dff; info->path = M.path;
  info->nnz_first_ring = M.nnz1; info->nnz_second_ring = M.nnz2; info->device_bytes = M.device_bytes;
  info->attention = M.attention;
  info->layered_attention = M.lattn;
  info->act_scale_mode = M.act_word ? AECCT_ACT_SCALE_WORD : AECCT_ACT_SCALE_TOKEN;
  info->device = M.device;
  info->compute_units = M.cu_count;
  info->lds_bytes = (int64_t)M.lds_max;
  return AECCT_OK;
}

aecct_status aecct_workspace_size(const aecct_model *model, int64_t batch, size_t *bytes) {
  if (!model || !bytes || batch < 0) return AECCT_ERR_INVALID_ARG;
  if (model->M.path == AECCT_PATH_FUSED || batch == 0) {
    *bytes = 0;
    return AECCT_OK;
  }
  *bytes = ws_plan(model->M, chunk_words(model->M, batch)).total;
  return AECCT_OK;
}

// The current device is the model's (every entry point that touches its memory checks this).
static aecct_status check_device(const Model &M) {
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return AECCT_ERR_DEVICE;
  return cur == M.device ? AECCT_OK : AECCT_ERR_INVALID_ARG;
}

// A decode of `batch` words in chunks of at most `cw` words, each chunk's layered activations in
// `ws` laid out by ws_plan(M, cw) (unused on the fused path).
static aecct_status decode_chunks(const Model &M, const float *y, int64_t batch, uint8_t *bits, float *logits,
                                  unsigned char *ws, int64_t cw, hipStream_t s) {
  if (M.path == AECCT_PATH_FUSED)
    return aecct::launch_fused(M, y, batch, bits, logits, s) == hipSuccess ? AECCT_OK : AECCT_ERR_DEVICE;
  const WsPlan W = ws_plan(M, cw);
  float *x = (float *)(ws + W.x), *qkv = (float *)(ws + W.qkv), *x1 = (float *)(ws + W.x1);
  int8_t *xq = (int8_t *)(ws + W.xq), *oq = (int8_t *)(ws + W.oq), *x1q = (int8_t *)(ws + W.x1q);
  int8_t *gq = (int8_t *)(ws + W.gq);
  float *ax = (float *)(ws + W.ax), *ao = (float *)(ws + W.ao), *a1 = (float *)(ws + W.a1), *ag = (float *)(ws + W.ag);
  float *o32 = M.act_word ? (float *)(ws + W.o32) : nullptr, *h32 = M.act_word ? (float *)(ws + W.h32) : nullptr;
  // With the token block, X and Xq are kept in its lane order from the embedding to the head.
  // The fused projection + attention (keys and values in LDS as fp32, or as int16 accumulators
  // for long words) leaves O in fp32 (in the QKV space); the token block then applies Eq. 2
  // itself. The lane-pair form on words of at most 384 tokens and the unfused attention quantise
  // O as they write it (a quarter of the bytes).  With one
  // alpha per word every quantisation point is redone over the whole word from the fp32 values
  // (natural layout, unfused form, no token block).
  const bool pw = M.act_word != 0;
  const bool tb = !pw && aecct::token_block_supported(M);
  const bool qa = M.lattn == AECCT_LAYERED_ATTN_LDS_F32, qw = M.lattn == AECCT_LAYERED_ATTN_LDS_I16;
  const bool qs = M.lattn == AECCT_LAYERED_ATTN_LDS_SPLIT;
  // the lane-pair form that writes O as Eq. 2 codes, which the token block then takes as they are
  const bool qa_codes = qa && tb && aecct::qkv_attention_pair_quantises(M);
  for (int64_t w0 = 0; w0 < batch; w0 += cw) {
    const int64_t nw = batch - w0 < cw ? batch - w0 : cw;
    const int64_t rows = nw * M.L;
    // with the token block the embedding leaves t_i per token (in ag, unused on that path) and
    // the first token block rebuilds X from it rather than reading X back
    float *tt = tb && rows <= INT32_MAX ? ag : nullptr;
    hipError_t e = aecct::launch_embed(M, y + w0 * M.n, nw, tt ? nullptr : x, xq, ax, tb, s, tt);
    if (pw && e == hipSuccess) e = aecct::launch_word_quant(M, x, nw, M.d, false, xq, ax, s);
    for (int l = 0; l < M.n_layers && e == hipSuccess; ++l) {
      if (qa) {
        e = aecct::launch_qkv_attention(M, l, xq, ax, nw, qkv, tb && !qa_codes ? nullptr : oq, ao, tb, s);
      } else if (qw) {
        e = aecct::launch_qkv_attention_i16(M, l, xq, ax, nw, qkv, tb, s);
      } else if (qs) {
        e = aecct::launch_qkv_attention_split(M, l, xq, ax, nw, qkv, tb, s);
      } else {
        e = aecct::launch_qkv(M, l, xq, ax, rows, qkv, tb, s);
        if (e == hipSuccess) e = aecct::launch_attention(M, qkv, nw, o32, oq, ao, s);
        if (pw && e == hipSuccess) e = aecct::launch_word_quant(M, o32, nw, M.d, false, oq, ao, s);
      }
      if (e != hipSuccess) break;
      if (tb) {
        // the last layer leaves the head's z per token in a1 (free once the layers are done)
        float *zl = l == M.n_layers - 1 ? a1 : nullptr;
        const float *t0 = l == 0 ? tt : nullptr;
        e = (qa && !qa_codes) || qw || qs
                ? aecct::launch_token_block(M, l, qkv, nullptr, nullptr, x, rows, xq, ax, s, zl, t0)
                : aecct::launch_token_block(M, l, nullptr, oq, ao, x, rows, xq, ax, s, zl, t0);
      } else {
        e = aecct::launch_oproj_ln(M, l, oq, ao, x, rows, x1, x1q, a1, s);
        if (pw && e == hipSuccess) e = aecct::launch_word_quant(M, x1, nw, M.d, false, x1q, a1, s);
        if (pw) {
          if (e == hipSuccess) e = aecct::launch_ffn1_f32(M, l, x1q, a1, rows, h32, s);
          if (e == hipSuccess) e = aecct::launch_word_quant(M, h32, nw, M.dff, true, gq, ag, s);
        } else if (e == hipSuccess) {
          e = aecct::launch_ffn1(M, l, x1q, a1, rows, gq, ag, s);
        }
        if (e == hipSuccess) e = aecct::launch_ffn2_ln(M, l, gq, ag, x1, rows, x, xq, ax, s);
        if (pw && e == hipSuccess) e = aecct::launch_word_quant(M, x, nw, M.d, false, xq, ax, s);
      }
    }
    if (e == hipSuccess)
      e = aecct::launch_head_tiled(M, x, y + w0 * M.n, nw, bits + w0 * M.n, logits ? logits + w0 * M.n : nullptr, tb,
                                   a1, s, tb);   // with the token block, z is already in a1
    if (e != hipSuccess) return AECCT_ERR_DEVICE;
  }
  return AECCT_OK;
}

aecct_status aecct_decode(const aecct_model *model, const float *y, int64_t batch, uint8_t *bits, float *logits,
                          void *workspace, size_t workspace_bytes, void *stream) {
  if (!model || batch < 0) return AECCT_ERR_INVALID_ARG;
  if (batch == 0) return AECCT_OK;
  if (!y || !bits) return AECCT_ERR_INVALID_ARG;
  const Model &M = model->M;
  const aecct_status dv = check_device(M);
  if (dv != AECCT_OK) return dv;
  size_t need = 0;
  aecct_workspace_size(model, batch, &need);
  if (workspace_bytes < need) return AECCT_ERR_WORKSPACE_TOO_SMALL;
  if (need && !workspace) return AECCT_ERR_INVALID_ARG;
  return decode_chunks(M, y, batch, bits, logits, (unsigned char *)workspace, chunk_words(M, batch),
                       (hipStream_t)stream);
}

aecct_status aecct_decode_static(const aecct_model *model, const float *y, int64_t batch, uint8_t *bits,
                                 float *logits, void *stream) {
  if (!model || batch < 0) return AECCT_ERR_INVALID_ARG;
  if (batch == 0) return AECCT_OK;
  if (!y || !bits) return AECCT_ERR_INVALID_ARG;
  const Model &M = model->M;
  const aecct_status dv = check_device(M);
  if (dv != AECCT_OK) return dv;
  int64_t cw = 1;
  if (M.path != AECCT_PATH_FUSED) {
    if (!M.static_scratch) return AECCT_ERR_DEVICE;
    if (ws_plan(M, 1).total > kStaticScratchBytes) return AECCT_ERR_WORKSPACE_TOO_SMALL;
    cw = chunk_words_within(M, batch, kStaticScratchBytes);
  }
  return decode_chunks(M, y, batch, bits, logits, M.static_scratch, cw, (hipStream_t)stream);
}

// ---- stage entry points --------------------------------------------------------------------

#define AECCT_STAGE_CHECK(cond)                          \
  do {                                                   \
    if (!(cond)) return AECCT_ERR_INVALID_ARG;           \
    const aecct_status dv_ = check_device(model->M);     \
    if (dv_ != AECCT_OK) return dv_;                     \
  } while (0)
// steps that quantise: a row's codes depend on the whole word when alpha is per word
#define AECCT_STAGE_PER_TOKEN() \
  do {                          \
    if (model->M.act_word) return AECCT_ERR_UNSUPPORTED; \
  } while (0)

static inline aecct_status launched(hipError_t e) { return e == hipSuccess ? AECCT_OK : AECCT_ERR_DEVICE; }

aecct_status aecct_stage_embed(const aecct_model *model, const float *y, int64_t words, float *x, int8_t *xq,
                               float *ax, void *stream) {
  AECCT_STAGE_CHECK(model && words >= 0 && (words == 0 || (y && x && xq && ax)));
  AECCT_STAGE_PER_TOKEN();
  return launched(aecct::launch_embed(model->M, y, words, x, xq, ax, false, (hipStream_t)stream));
}

aecct_status aecct_stage_qkv(const aecct_model *model, int32_t layer, const int8_t *xq, const float *ax,
                             int64_t words, float *qkv, void *stream) {
  AECCT_STAGE_CHECK(model && words >= 0 && layer >= 0 && layer < model->M.n_layers && (words == 0 || (xq && ax && qkv)));
  return launched(aecct::launch_qkv(model->M, layer, xq, ax, words * model->M.L, qkv, false, (hipStream_t)stream));
}

aecct_status aecct_stage_attention(const aecct_model *model, const float *qkv, int64_t words, float *o, int8_t *oq,
                                   float *ao, void *stream) {
  AECCT_STAGE_CHECK(model && words >= 0 && (words == 0 || (qkv && oq && ao)));
  AECCT_STAGE_PER_TOKEN();
  return launched(aecct::launch_attention(model->M, qkv, words, o, oq, ao, (hipStream_t)stream));
}

aecct_status aecct_stage_oproj_ln(const aecct_model *model, int32_t layer, const int8_t *oq, const float *ao,
                                  const float *x, int64_t words, float *x1, int8_t *x1q, float *a1, void *stream) {
  AECCT_STAGE_CHECK(model && words >= 0 && layer >= 0 && layer < model->M.n_layers &&
                    (words == 0 || (oq && ao && x && x1 && x1q && a1)));
  AECCT_STAGE_PER_TOKEN();
  return launched(aecct::launch_oproj_ln(model->M, layer, oq, ao, x, words * model->M.L, x1, x1q, a1,
                                         (hipStream_t)stream));
}

aecct_status aecct_stage_ffn1(const aecct_model *model, int32_t layer, const int8_t *x1q, const float *a1,
                              int64_t words, int8_t *gq, float *ag, void *stream) {
  AECCT_STAGE_CHECK(model && words >= 0 && layer >= 0 && layer < model->M.n_layers && (words == 0 || (x1q && a1 && gq && ag)));
  AECCT_STAGE_PER_TOKEN();
  return launched(aecct::launch_ffn1(model->M, layer, x1q, a1, words * model->M.L, gq, ag, (hipStream_t)stream));
}

aecct_status aecct_stage_ffn2_ln(const aecct_model *model, int32_t layer, const int8_t *gq, const float *ag,
                                 const float *x1, int64_t words, float *x, int8_t *xq, float *ax, void *stream) {
  AECCT_STAGE_CHECK(model && words >= 0 && layer >= 0 && layer < model->M.n_layers &&
                    (words == 0 || (gq && ag && x1 && x && xq && ax)));
  AECCT_STAGE_PER_TOKEN();
  return launched(aecct::launch_ffn2_ln(model->M, layer, gq, ag, x1, words * model->M.L, x, xq, ax,
                                        (hipStream_t)stream));
}

aecct_status aecct_stage_head(const aecct_model *model, const float *x, const float *y, int64_t words, uint8_t *bits,
                              float *logits, void *stream) {
  AECCT_STAGE_CHECK(model && words >= 0 && (words == 0 || (x && y && bits)));
  return launched(aecct::launch_head(model->M, x, y, words, bits, logits, false, (hipStream_t)stream));
}

aecct_status aecct_ternary_gemm(const aecct_model *model, int32_t layer, int32_t kind, const int8_t *a, int64_t rows,
                                int32_t *acc, void *stream) {
  AECCT_STAGE_CHECK(model && rows >= 0 && layer >= 0 && layer < model->M.n_layers && kind >= 0 && kind < 6 &&
                    (rows == 0 || (a && acc)));
  return launched(aecct::launch_ternary_gemm(model->M, layer, kind, a, rows, acc, (hipStream_t)stream));
}

}  // extern "C"
