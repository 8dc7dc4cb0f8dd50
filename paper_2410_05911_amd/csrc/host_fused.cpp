// Host packing of the fused path's tables (declarations and layout in host_fused.h and
// kernel_fused.hip).
#include <algorithm>
#include <cstdint>
#include <functional>
#include <vector>

#include "host_fused.h"

namespace aecct {

// Token tiles of the fused path.  In tile t the neighbour loop of head group grp runs
// T(t, grp) = the longest list of that group among the tile's tokens, so a decode costs
// sum over tiles of T(t, 0) + T(t, 1) steps.  Given per-token loop lengths w0, w1, this picks
// NT tiles of at most 16 tokens minimising that sum: a depth-first search over the tiles'
// (T0, T1) caps, taken as pairs of attained lengths in non-increasing order, pruned by the best
// cost so far, by tokens no chosen or later cap can cover, and by capacity; a full set of caps
// is accepted when a token-to-tile assignment within 16 per tile exists (augmenting paths).
// The search stops after a fixed number of nodes and keeps the best partition found; it
// starts from tiles filled in order of longest lists.  Returns the token of each slot (-1 for
// padding).
std::vector<int32_t> fused_tile_partition(int L, int NT, const std::vector<int> &w0, const std::vector<int> &w1) {
  struct Cap { int a, b; };
  auto cost_of = [&](const std::vector<int32_t> &slots) {
    long c = 0;
    for (int t = 0; t < NT; ++t) {
      int a = 0, b = 0;
      for (int k = 0; k < 16; ++k) {
        const int tok = slots[16 * t + k];
        if (tok >= 0) { a = std::max(a, w0[tok]); b = std::max(b, w1[tok]); }
      }
      c += a + b;
    }
    return c;
  };
  auto fill = [&](std::vector<int> order) {
    std::vector<int32_t> slots(16 * NT, -1);
    for (int i = 0; i < L; ++i) slots[i] = order[i];
    return slots;
  };
  std::vector<int> order(L);
  for (int t = 0; t < L; ++t) order[t] = t;
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) {
    if (w1[x] != w1[y]) return w1[x] > w1[y];
    return w0[x] > w0[y];
  });
  std::vector<int32_t> best = fill(order);
  long best_cost = cost_of(best);
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return w0[x] + w1[x] > w0[y] + w1[y]; });
  {
    std::vector<int32_t> s2 = fill(order);
    const long c2 = cost_of(s2);
    if (c2 < best_cost) { best = s2; best_cost = c2; }
  }
  std::vector<int> va(w0.begin(), w0.end()), vb(w1.begin(), w1.end());
  std::sort(va.begin(), va.end());
  va.erase(std::unique(va.begin(), va.end()), va.end());
  std::sort(vb.begin(), vb.end());
  vb.erase(std::unique(vb.begin(), vb.end()), vb.end());
  std::vector<Cap> caps;
  for (int b : vb)
    for (int a : va) caps.push_back({a, b});
  std::sort(caps.begin(), caps.end(), [](const Cap &x, const Cap &y) { return x.b != y.b ? x.b > y.b : x.a > y.a; });
  const int nc = (int)caps.size();
  // assignment of every token to one of the chosen caps, at most 16 per tile
  std::vector<int> assign(L), load(NT);
  auto feasible = [&](const std::vector<Cap> &cs) {
    std::vector<std::vector<int>> opts(L);
    for (int t = 0; t < L; ++t)
      for (int k = 0; k < NT; ++k)
        if (w0[t] <= cs[k].a && w1[t] <= cs[k].b) opts[t].push_back(k);
    std::fill(assign.begin(), assign.end(), -1);
    std::fill(load.begin(), load.end(), 0);
    std::vector<char> seen(NT);
    std::function<bool(int)> aug = [&](int t) -> bool {
      for (int k : opts[t]) {
        if (seen[k]) continue;
        seen[k] = 1;
        if (load[k] < 16) { ++load[k]; assign[t] = k; return true; }
        for (int u = 0; u < L; ++u)
          if (assign[u] == k && aug(u)) { assign[t] = k; return true; }
      }
      return false;
    };
    std::vector<int> ord(L);
    for (int t = 0; t < L; ++t) ord[t] = t;
    std::sort(ord.begin(), ord.end(), [&](int x, int y) { return opts[x].size() < opts[y].size(); });
    for (int t : ord) {
      std::fill(seen.begin(), seen.end(), 0);
      if (!aug(t)) return false;
    }
    return true;
  };
  std::vector<Cap> chosen;
  std::vector<int> cover(L, 0);                // chosen caps covering each token
  long nodes = 0;
  const long kMaxNodes = 20000;
  std::function<void(int, long)> dfs = [&](int j, long sum) {
    if (++nodes > kMaxNodes) return;
    const int k = (int)chosen.size();
    // tokens no chosen cap covers: later caps (b no larger than caps[j].b) must take them
    int unc = 0, unc_b = -1, unc_lb = 0;
    for (int t = 0; t < L; ++t)
      if (!cover[t]) { ++unc; unc_b = std::max(unc_b, w1[t]); unc_lb = std::max(unc_lb, w0[t] + w1[t]); }
    if (k == NT) {
      if (unc == 0 && sum < best_cost && feasible(chosen)) {
        std::vector<int32_t> slots(16 * NT, -1);
        std::vector<int> fillk(NT, 0);
        for (int t = 0; t < L; ++t) slots[16 * assign[t] + fillk[assign[t]]++] = t;
        const long c = cost_of(slots);
        if (c < best_cost) { best = slots; best_cost = c; }
      }
      return;
    }
    if (unc > 16 * (NT - k) || sum + unc_lb >= best_cost) return;
    for (int i = j; i < nc; ++i) {
      if (caps[i].b < unc_b) break;            // caps are ordered by b: none later covers them
      if (sum + caps[i].a + caps[i].b >= best_cost) continue;
      chosen.push_back(caps[i]);
      for (int t = 0; t < L; ++t) cover[t] += w0[t] <= caps[i].a && w1[t] <= caps[i].b;
      dfs(i, sum + caps[i].a + caps[i].b);
      for (int t = 0; t < L; ++t) cover[t] -= w0[t] <= caps[i].a && w1[t] <= caps[i].b;
      chosen.pop_back();
      if (nodes > kMaxNodes) return;
    }
  };
  dfs(0, 0);
  return best;
}


void build_fused(const Model &M, const uint8_t *H, const aecct_weights *w, const std::vector<int32_t> &m1_ptr,
                 const std::vector<int32_t> &m1_idx, const std::vector<int32_t> &m2_ptr,
                 const std::vector<int32_t> &m2_idx, FusedImage &F) {
  const int L = M.L, n = M.n, m = M.m, NT = (L + 15) / 16, S = 16 * NT, N = M.n_layers;
  const size_t D = fz::D, FF = fz::DFF;
  auto len = [&](int mask, int tok) {
    return mask == 0 ? m1_ptr[tok + 1] - m1_ptr[tok] : m2_ptr[tok + 1] - m2_ptr[tok];
  };
  auto mask_of = [&](int head) { return head < M.hf ? 0 : 1; };
  auto work = [&](int tok, int grp) {
    int mx = 0;
    for (int g = 0; g < 4; ++g) mx = std::max(mx, len(mask_of(4 * grp + g), tok));
    return mx;
  };
  // token slots: tiles chosen to minimise the padded neighbour-loop steps
  {
    std::vector<int> w0(L), w1(L);
    for (int t = 0; t < L; ++t) { w0[t] = work(t, 0); w1[t] = work(t, 1); }
    F.slot_token = fused_tile_partition(L, NT, w0, w1);
  }
  // Per tile and head group the neighbour loop runs T = the longest list among the tile's
  // lanes (padding slots have none).
  F.tile_tab.assign(2 * NT, 0);
  for (int t = 0; t < NT; ++t)
    for (int grp = 0; grp < 2; ++grp) {
      int T = 1;
      for (int c = 0; c < 16; ++c) {
        const int tok = F.slot_token[16 * t + c];
        if (tok < 0) continue;
        for (int g = 0; g < 4; ++g) T = std::max(T, len(mask_of(4 * grp + g), tok));
      }
      F.tile_tab[2 * t + grp] = (uint32_t)T;
    }
  // Stored length of the (tile, mask) lists of a mask some head reads: every list of the mask
  // in the tile, and T of every head group that reads the mask.  A mask no head reads gets an
  // empty region (its lists are never stored or read).
  bool used[2] = {false, false};
  for (int h = 0; h < 8; ++h) used[mask_of(h)] = true;
  std::vector<int> padT(2 * NT, 0);
  for (int t = 0; t < NT; ++t) {
    for (int c = 0; c < 16; ++c) {
      const int tok = F.slot_token[16 * t + c];
      if (tok < 0) continue;
      for (int mask = 0; mask < 2; ++mask)
        if (used[mask]) padT[2 * t + mask] = std::max(padT[2 * t + mask], len(mask, tok));
    }
    for (int grp = 0; grp < 2; ++grp)
      for (int g = 0; g < 4; ++g) {
        const int mask = mask_of(4 * grp + g);
        padT[2 * t + mask] = std::max(padT[2 * t + mask], (int)F.tile_tab[2 * t + grp]);
      }
  }
  // Columns within a tile: a seeded local search over swaps of two columns of one tile that
  // lowers the LDS bank collisions of the key/value gathers (the 16 lanes of one head read the
  // rows of their e-th neighbours; rows of slots with equal column mod 16 (or mod 8 within a
  // half of the lanes) share banks).  Tile membership, hence every loop length, is unchanged.
  {
    auto nb = [&](int mask, int tok, int e) {
      const std::vector<int32_t> &ptr = mask == 0 ? m1_ptr : m2_ptr;
      const std::vector<int32_t> &idx = mask == 0 ? m1_idx : m2_idx;
      const int cnt = ptr[tok + 1] - ptr[tok];
      return e < cnt ? idx[ptr[tok] + e] : L;      // entries past the list read the pad row
    };
    std::vector<int> col(L + 1, 0);                // the pad row (index L) sits in column 0
    auto refresh = [&]() {
      for (int sl = 0; sl < S; ++sl)
        if (F.slot_token[sl] >= 0) col[F.slot_token[sl]] = sl % 16;
    };
    auto cost = [&]() {
      long total = 0;
      for (int t = 0; t < NT; ++t)
        for (int grp = 0; grp < 2; ++grp) {
          const int T = (int)F.tile_tab[2 * t + grp];
          int weight[2] = {0, 0};                  // lane groups reading each mask
          for (int g = 0; g < 4; ++g) ++weight[mask_of(4 * grp + g)];
          for (int mask = 0; mask < 2; ++mask) {
            if (!weight[mask]) continue;
            for (int e = 0; e < T; ++e) {
              int seen_tok[16], cnt16[16] = {0}, cnt8a[8] = {0}, cnt8b[8] = {0}, ns = 0;
              for (int c = 0; c < 16; ++c) {
                const int tok = F.slot_token[16 * t + c];
                if (tok < 0) continue;
                const int j = nb(mask, tok, e);
                bool dup = false;
                for (int q = 0; q < ns; ++q) dup |= seen_tok[q] == j;
                if (dup) continue;
                seen_tok[ns++] = j;
                ++cnt16[col[j]];
                if (c < 8) ++cnt8a[col[j] % 8]; else ++cnt8b[col[j] % 8];
              }
              int m16 = 0, m8 = 0;
              for (int b = 0; b < 16; ++b) m16 = std::max(m16, cnt16[b]);
              for (int b = 0; b < 8; ++b) m8 = std::max(m8, std::max(cnt8a[b], cnt8b[b]));
              total += (long)weight[mask] * (m16 + m8);
            }
          }
        }
      return total;
    };
    refresh();
    long best = cost();
    uint64_t rng = 0x9E3779B97F4A7C15ull;
    auto next = [&]() { rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17; return rng; };
    const int iters = 2000;
    for (int it = 0; it < iters; ++it) {
      const int t = (int)(next() % NT);
      const int a = 16 * t + (int)(next() % 16), b = 16 * t + (int)(next() % 16);
      if (a == b || (F.slot_token[a] < 0 && F.slot_token[b] < 0)) continue;
      std::swap(F.slot_token[a], F.slot_token[b]);
      refresh();
      const long cst = cost();
      if (cst <= best) {
        best = cst;
      } else {
        std::swap(F.slot_token[a], F.slot_token[b]);
        refresh();
      }
    }
  }
  std::vector<int> slot_of(L);
  for (int sl = 0; sl < S; ++sl)
    if (F.slot_token[sl] >= 0) slot_of[F.slot_token[sl]] = sl;
  // neighbour lists: byte offsets of the neighbours' 16-byte key rows in ascending token order,
  // padded with the offset of the pad row (row 16 NT of a head), in groups of four entries
  // per column: entry e of column c at tbase + 64 (e / 4) + 4 c + e % 4.  A (tile, mask)
  // region holds floor(padT / 4) + 1 groups, one more than the full groups of any loop over
  // it, so the kernel may always read the group after the last full one.
  F.slot_tab.assign(2 * S, 0);
  {
    std::vector<size_t> tbase(2 * NT);
    size_t total = 0;
    for (int tm = 0; tm < 2 * NT; ++tm) {
      tbase[tm] = total;
      total += (size_t)(padT[tm] / 4 + 1) * 64;
    }
    F.nbr.assign(total, (uint16_t)(S * 16));
    for (int sl = 0; sl < S; ++sl)
      for (int mask = 0; mask < 2; ++mask) {
        const int t = sl / 16, c = sl % 16, tok = F.slot_token[sl];
        const size_t base = tbase[2 * t + mask] + 4 * (size_t)c;
        uint32_t cnt = 0;
        if (tok >= 0 && used[mask]) {
          const std::vector<int32_t> &ptr = mask == 0 ? m1_ptr : m2_ptr;
          const std::vector<int32_t> &idx = mask == 0 ? m1_idx : m2_idx;
          cnt = (uint32_t)(ptr[tok + 1] - ptr[tok]);
          for (uint32_t e = 0; e < cnt; ++e)
            F.nbr[base + 64 * (e / 4) + e % 4] = (uint16_t)(slot_of[idx[ptr[tok] + e]] * 16);
        }
        F.slot_tab[2 * sl + mask] = (uint32_t)base | (cnt << 16);
      }
  }
  while (F.nbr.size() % 8) F.nbr.push_back(0);
  F.chk.assign(m, 0);
  for (int j = 0; j < m; ++j)
    for (int i = 0; i < n; ++i)
      if (H[(size_t)j * n + i]) F.chk[j] |= (uint64_t)1 << i;
  F.eperm.assign((size_t)S * 32, 0.0f);
  if (w->pos) F.pperm.assign((size_t)S * 32, 0.0f);
  for (int sl = 0; sl < S; ++sl)
    for (int g = 0; g < 4; ++g)
      for (int v = 0; v < 8; ++v) {
        if (F.slot_token[sl] < 0) continue;   // padding slots keep zero rows
        const size_t src = (size_t)F.slot_token[sl] * D + 4 * v + g, dst = ((size_t)sl * 4 + g) * 8 + v;
        F.eperm[dst] = w->embed[src];
        if (w->pos) F.pperm[dst] = w->pos[src];
      }
  F.w1perm.resize(32);
  for (int g = 0; g < 4; ++g)
    for (int v = 0; v < 8; ++v) F.w1perm[8 * g + v] = w->head_w1[4 * v + g];

  // input slot e of lane group g -> feature, per producer layout
  auto in_x = [](int g, int e) { return 4 * e + g; };                                   // LN outputs, embedding
  auto in_o = [](int g, int e) { return e < 4 ? 4 * g + e : 16 + 4 * g + (e - 4); };   // attention output
  auto in_g = [](int s, int g, int e) { return 16 * (2 * s + (e >> 2)) + 4 * g + (e & 3); };  // ReLU hidden
  // output row r of tile o -> feature
  auto out_ln = [](int o, int r) { return 16 * o + 4 * (r & 3) + (r >> 2); };
  F.frag.assign((size_t)N * fz::FRAGS * 64, 0);
  F.vec.assign((size_t)N * fz::VEC, 0.0f);
  for (int l = 0; l < N; ++l) {
    const int8_t *Wq = w->w_q + l * D * D, *Wk = w->w_k + l * D * D, *Wv = w->w_v + l * D * D;
    const int8_t *Wo = w->w_o + l * D * D, *W1 = w->w_ff1 + l * D * FF, *W2 = w->w_ff2 + l * FF * D;
    uint16_t *fr = F.frag.data() + (size_t)l * fz::FRAGS * 64;
    auto put_frag = [&](int idx, auto value) {   // value(lane row r, lane group g, slot e) -> ternary
      for (int lane = 0; lane < 64; ++lane) {
        uint16_t v = 0;
        for (int e = 0; e < 8; ++e) v |= (uint16_t)(code2(value(lane & 15, lane >> 4, e)) << (2 * e));
        fr[(size_t)idx * 64 + lane] = v;
      }
    };
    for (int o = 0; o < 6; ++o)
      put_frag(o, [&](int r, int g, int e) {
        const int col = 16 * o + r, mat = col / 32, j = col % 32;
        const int8_t *W = mat == 0 ? Wq : (mat == 1 ? Wk : Wv);
        return W[(size_t)in_x(g, e) * D + j];
      });
    for (int o = 0; o < 2; ++o)
      put_frag(fz::F_O + o, [&](int r, int g, int e) { return Wo[(size_t)in_o(g, e) * D + out_ln(o, r)]; });
    for (int o = 0; o < 8; ++o)
      put_frag(fz::F_FF1 + o, [&](int r, int g, int e) { return W1[(size_t)in_x(g, e) * FF + 16 * o + r]; });
    for (int o = 0; o < 2; ++o)
      for (int st = 0; st < 4; ++st)
        put_frag(fz::F_FF2 + 4 * o + st,
                 [&](int r, int g, int e) { return W2[(size_t)in_g(st, g, e) * D + out_ln(o, r)]; });
    float *V = F.vec.data() + (size_t)l * fz::VEC;
    for (size_t j = 0; j < D; ++j) {
      V[fz::V_BQKV + j] = w->b_q[l * D + j] * M.kq;
      V[fz::V_BQKV + 32 + j] = w->b_k[l * D + j];
      V[fz::V_BQKV + 64 + j] = w->b_v[l * D + j];
    }
    for (size_t j = 0; j < FF; ++j) V[fz::V_BFF1 + j] = w->b_ff1[l * FF + j];
    for (int o = 0; o < 2; ++o)
      for (int g = 0; g < 4; ++g)
        for (int i = 0; i < 4; ++i) {
          const int f = 16 * o + 4 * i + g, at = 16 * o + 4 * g + i;
          V[fz::V_BO + at] = w->b_o[l * D + f];
          V[fz::V_BFF2 + at] = w->b_ff2[l * D + f];
        }
    for (int g = 0; g < 4; ++g)
      for (int v = 0; v < 8; ++v) {
        const int f = 4 * v + g, at = 8 * g + v;
        V[fz::V_LN1G + at] = w->ln1_g[l * D + f];
        V[fz::V_LN1B + at] = w->ln1_b[l * D + f];
        V[fz::V_LN2G + at] = w->ln2_g[l * D + f];
        V[fz::V_LN2B + at] = w->ln2_b[l * D + f];
      }
    V[fz::V_SQ + 0] = M.layer[l].sq_qs;
    for (int k = 1; k < 6; ++k) V[fz::V_SQ + k] = M.layer[l].sq[k];
  }
}

}  // namespace aecct
