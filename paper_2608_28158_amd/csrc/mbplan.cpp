// Prefix-aware microbatch and data-parallel planning (HARTS, Sec. 3.2).
//
// Trajectories are ranked lexicographically; with the adjacent longest
// common prefixes L and a sparse-table range minimum over them, the compact
// trie work of any set of ranks is its summed lengths minus the LCPs of
// rank neighbours (eq. compact-trie-cost), O(1) for a contiguous interval
// (prefix sums) and O(members) otherwise.  Candidates:
//   - exact contiguous DP per K (eq. contiguous-dp) up to exact_max
//     trajectories, otherwise merge/split evolution of the natural
//     partition at sampled K (merges save, splits cost, the boundary LCP:
//     eq. cut-prefix-loss);
//   - trie-aware greedy (eq. greedy-insertion-delta), 4 orders x 2
//     policies, small-microbatch elimination, K aligned to D by singleton
//     splits; the fewest-microbatch, least-work one is kept;
//   - refinement: boundary refinement of contiguous anchors and sparse
//     repair (moves, then swaps, within 8 ranks).
// Each candidate gets replicas and slots (heaviest first, to the replica
// with the least work so far) and the plan minimising
// J = (total work, sum of slot maxima, heaviest replica) is returned
// (eq. prefix-plan-objective).  Ties everywhere fall to the earlier
// candidate, smaller index or smaller rank, as spelled out per step.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <new>
#include <set>
#include <string>
#include <tuple>
#include <vector>

#include "harts.h"
#include "plan.hpp"

using harts::set_error;

namespace {

constexpr int32_t kN0 = 512;   // exact search threshold
constexpr int32_t kQmax = 32;  // sampled K budget
constexpr int32_t kH = 8;      // refinement window (ranks)
constexpr int32_t kBref = 3;   // refined anchors

using Parts = std::vector<std::pair<int32_t, int32_t>>;  // contiguous rank intervals
using Groups = std::vector<std::vector<int32_t>>;        // sorted ranks per microbatch

struct Lex {
  int32_t N = 0;
  std::vector<int32_t> order, rank;
  std::vector<int64_t> len;     // by rank
  std::vector<int64_t> L;       // L[r] = LCP(rank r - 1, rank r), L[0] = 0
  std::vector<int64_t> plen, pL;  // prefix sums
  std::vector<std::vector<int64_t>> sp;  // sparse table of L
  std::vector<int32_t> lg;

  void build(int32_t n, const int64_t* off, const int32_t* tok) {
    N = n;
    order.resize(N);
    for (int32_t i = 0; i < N; ++i) order[i] = i;
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
      return std::lexicographical_compare(tok + off[a], tok + off[a + 1], tok + off[b], tok + off[b + 1]);
    });
    rank.assign(N, 0);
    for (int32_t r = 0; r < N; ++r) rank[order[r]] = r;
    len.assign(N, 0);
    L.assign(N, 0);
    for (int32_t r = 0; r < N; ++r) {
      const int32_t i = order[r];
      len[r] = off[i + 1] - off[i];
      if (r > 0) {
        const int32_t j = order[r - 1];
        const int64_t n2 = std::min(len[r], off[j + 1] - off[j]);
        int64_t k = 0;
        while (k < n2 && tok[off[i] + k] == tok[off[j] + k]) ++k;
        L[r] = k;
      }
    }
    plen.assign(N + 1, 0);
    pL.assign(N + 1, 0);
    for (int32_t r = 0; r < N; ++r) {
      plen[r + 1] = plen[r] + len[r];
      pL[r + 1] = pL[r] + L[r];
    }
    lg.assign(N + 1, 0);
    for (int32_t i = 2; i <= N; ++i) lg[i] = lg[i / 2] + 1;
    sp.assign(lg[std::max(N, 1)] + 1, std::vector<int64_t>());
    sp[0] = L;
    for (size_t k = 1; k < sp.size(); ++k) {
      const int32_t span = 1 << k;
      sp[k].assign(std::max(0, N - span + 1), 0);
      for (int32_t i = 0; i + span <= N; ++i)
        sp[k][i] = std::min(sp[k - 1][i], sp[k - 1][i + span / 2]);
    }
  }
  // min L[a .. b], a <= b
  int64_t rmq(int32_t a, int32_t b) const {
    const int32_t k = lg[b - a + 1];
    return std::min(sp[k][a], sp[k][b - (1 << k) + 1]);
  }
  int64_t lcp_ranks(int32_t r1, int32_t r2) const {
    const int32_t a = std::min(r1, r2), b = std::max(r1, r2);
    return rmq(a + 1, b);
  }
  int64_t W(int32_t a, int32_t b) const {  // ranks a..b inclusive
    return (plen[b + 1] - plen[a]) - (pL[b + 1] - pL[a + 1]);
  }
  int64_t work(const std::vector<int32_t>& rs) const {  // sorted ranks
    int64_t w = 0;
    for (size_t i = 0; i < rs.size(); ++i) {
      w += len[rs[i]];
      if (i) w -= lcp_ranks(rs[i - 1], rs[i]);
    }
    return w;
  }
  // eq. greedy-insertion-delta: work added by inserting rank r into ms
  int64_t delta(const std::vector<int32_t>& ms, int32_t r) const {
    auto it = std::lower_bound(ms.begin(), ms.end(), r);
    const bool hq = it != ms.end(), hp = it != ms.begin();
    int64_t d = len[r];
    if (hp) d -= lcp_ranks(*(it - 1), r);
    if (hq) d -= lcp_ranks(r, *it);
    if (hp && hq) d += lcp_ranks(*(it - 1), *it);
    return d;
  }
};

Groups to_groups(const Parts& parts) {
  Groups g;
  for (const auto& p : parts) {
    std::vector<int32_t> m;
    for (int32_t r = p.first; r <= p.second; ++r) m.push_back(r);
    g.push_back(std::move(m));
  }
  return g;
}

void insert_sorted(std::vector<int32_t>& v, int32_t r) { v.insert(std::lower_bound(v.begin(), v.end(), r), r); }
void erase_one(std::vector<int32_t>& v, int32_t r) { v.erase(std::lower_bound(v.begin(), v.end(), r)); }

Parts natural_partition(const Lex& lx, int64_t T) {
  Parts out;
  std::vector<std::pair<int32_t, int32_t>> stack{{0, lx.N - 1}};
  while (!stack.empty()) {
    const auto [a, b] = stack.back();
    stack.pop_back();
    if (lx.W(a, b) <= T || a == b) {
      out.push_back({a, b});
      continue;
    }
    std::tuple<int64_t, int64_t, int64_t, int32_t> best{INT64_MAX, 0, 0, 0};
    for (int32_t t = a + 1; t <= b; ++t) {
      const int64_t wl = lx.W(a, t - 1), wr = lx.W(t, b);
      const auto key = std::make_tuple(lx.L[t], std::max(wl, wr), wl > wr ? wl - wr : wr - wl, t);
      if (key < best) best = key;
    }
    const int32_t t = std::get<3>(best);
    stack.push_back({t, b});  // left first
    stack.push_back({a, t - 1});
  }
  return out;
}

std::vector<std::pair<int32_t, Parts>> exact_dp(const Lex& lx, int64_t T, const std::vector<int32_t>& Ks) {
  const int32_t N = lx.N, kmax = Ks.back();
  struct St {
    int64_t tot = -1, mx = 0;
    int32_t arg = -1;
  };
  std::vector<std::vector<St>> F(kmax + 1, std::vector<St>(N + 1));
  F[0][0].tot = 0;
  for (int32_t k = 1; k <= kmax; ++k) {
    int32_t s_min = 0;  // first s with W(s, e - 1) <= T; moves right with e
    for (int32_t e = 1; e <= N; ++e) {
      while (s_min < e && lx.W(s_min, e - 1) > T) ++s_min;
      St best;
      for (int32_t s = s_min; s < e; ++s) {
        const St& pr = F[k - 1][s];
        if (pr.tot < 0) continue;
        const int64_t w = lx.W(s, e - 1);
        const int64_t tot = pr.tot + w, mx = std::max(pr.mx, w);
        if (best.tot < 0 || tot < best.tot || (tot == best.tot && mx < best.mx)) {
          best.tot = tot;
          best.mx = mx;
          best.arg = s;
        }
      }
      F[k][e] = best;
    }
  }
  std::vector<std::pair<int32_t, Parts>> out;
  for (const int32_t K : Ks) {
    if (F[K][N].tot < 0) continue;
    Parts parts;
    int32_t e = N;
    for (int32_t k = K; k > 0; --k) {
      const int32_t s = F[k][e].arg;
      parts.push_back({s, e - 1});
      e = s;
    }
    std::reverse(parts.begin(), parts.end());
    out.push_back({K, parts});
  }
  return out;
}

std::vector<int32_t> sampled_ks(const std::vector<int32_t>& Ks) {
  if (static_cast<int32_t>(Ks.size()) <= kQmax) return Ks;
  std::set<int32_t> pick(Ks.begin(), Ks.begin() + kQmax / 2);
  const std::vector<int32_t> rest(Ks.begin() + kQmax / 2, Ks.end());
  const int32_t m = kQmax - kQmax / 2;
  for (int32_t i = 0; i < m; ++i) {
    const double x = static_cast<double>(i) * static_cast<double>(rest.size() - 1) / static_cast<double>(m - 1);
    pick.insert(rest[static_cast<size_t>(std::nearbyint(x))]);  // ties to even
  }
  return std::vector<int32_t>(pick.begin(), pick.end());
}

bool evolve(const Lex& lx, int64_t T, Parts& parts, int32_t K) {
  while (static_cast<int32_t>(parts.size()) > K) {
    int32_t bi = -1;
    std::pair<int64_t, int32_t> bk;
    for (size_t i = 0; i + 1 < parts.size(); ++i) {
      if (lx.W(parts[i].first, parts[i + 1].second) > T) continue;
      const auto key = std::make_pair(-lx.L[parts[i + 1].first], parts[i + 1].first);
      if (bi < 0 || key < bk) { bk = key; bi = static_cast<int32_t>(i); }
    }
    if (bi < 0) return false;
    parts[bi].second = parts[bi + 1].second;
    parts.erase(parts.begin() + bi + 1);
  }
  while (static_cast<int32_t>(parts.size()) < K) {
    int32_t bi = -1, bt = -1;
    std::tuple<int64_t, int64_t, int32_t> bk;
    for (size_t i = 0; i < parts.size(); ++i) {
      const auto [a, b] = parts[i];
      for (int32_t t = a + 1; t <= b; ++t) {
        const auto key = std::make_tuple(lx.L[t], std::max(lx.W(a, t - 1), lx.W(t, b)), t);
        if (bi < 0 || key < bk) { bk = key; bi = static_cast<int32_t>(i); bt = t; }
      }
    }
    if (bi < 0) return false;
    const auto [a, b] = parts[bi];
    parts[bi] = {a, bt - 1};
    parts.insert(parts.begin() + bi + 1, {bt, b});
  }
  return true;
}

bool greedy(const Lex& lx, int64_t T, int32_t D, const std::vector<int32_t>& order, bool best_fit, Groups& g) {
  g.clear();
  std::vector<int64_t> w;
  for (const int32_t r : order) {
    int32_t bi = -1;
    std::pair<int64_t, int32_t> bk;
    for (size_t i = 0; i < g.size(); ++i) {
      const int64_t dc = lx.delta(g[i], r);
      if (w[i] + dc > T) continue;
      const auto key = best_fit ? std::make_pair(-(w[i] + dc), static_cast<int32_t>(i))
                                : std::make_pair(-(lx.len[r] - dc), static_cast<int32_t>(i));
      if (bi < 0 || key < bk) { bk = key; bi = static_cast<int32_t>(i); }
    }
    if (bi < 0) {
      g.push_back({r});
      w.push_back(lx.len[r]);
    } else {
      w[bi] += lx.delta(g[bi], r);
      insert_sorted(g[bi], r);
    }
  }
  // small-microbatch elimination
  bool changed = true;
  while (changed && g.size() > 1) {
    changed = false;
    std::vector<int32_t> idx(g.size());
    for (size_t i = 0; i < g.size(); ++i) idx[i] = static_cast<int32_t>(i);
    std::vector<int64_t> gw(g.size());
    for (size_t i = 0; i < g.size(); ++i) gw[i] = lx.work(g[i]);
    std::stable_sort(idx.begin(), idx.end(), [&](int32_t a, int32_t b) { return gw[a] < gw[b]; });
    for (const int32_t i : idx) {
      Groups trial = g;
      bool ok = true;
      for (const int32_t r : g[i]) {
        int32_t bj = -1;
        int64_t bdc = 0;
        for (size_t j = 0; j < trial.size(); ++j) {
          if (static_cast<int32_t>(j) == i) continue;
          const int64_t dc = lx.delta(trial[j], r);
          if (lx.work(trial[j]) + dc > T) continue;
          if (bj < 0 || dc < bdc) { bdc = dc; bj = static_cast<int32_t>(j); }
        }
        if (bj < 0) { ok = false; break; }
        insert_sorted(trial[bj], r);
      }
      if (ok) {
        trial.erase(trial.begin() + i);
        g = std::move(trial);
        changed = true;
        break;
      }
    }
  }
  // K aligned to D by singleton splits
  while (g.size() % D) {
    int32_t bi = -1, br = -1;
    int64_t bc = 0;
    for (size_t i = 0; i < g.size(); ++i) {
      if (g[i].size() < 2) continue;
      const int64_t wm = lx.work(g[i]);
      for (const int32_t r : g[i]) {
        std::vector<int32_t> rest = g[i];
        erase_one(rest, r);
        const int64_t cost = lx.work(rest) + lx.len[r] - wm;
        if (bi < 0 || cost < bc) { bc = cost; bi = static_cast<int32_t>(i); br = r; }
      }
    }
    if (bi < 0) return false;
    erase_one(g[bi], br);
    g.push_back({br});
  }
  return true;
}

std::vector<std::vector<int32_t>> greedy_orders(const Lex& lx) {
  const int32_t N = lx.N;
  std::vector<int32_t> asc(N);
  for (int32_t r = 0; r < N; ++r) asc[r] = r;
  std::vector<int32_t> desc(asc.rbegin(), asc.rend());
  std::vector<int32_t> by_len = asc, by_u = asc;
  std::stable_sort(by_len.begin(), by_len.end(), [&](int32_t a, int32_t b) { return lx.len[a] > lx.len[b]; });
  std::vector<int64_t> u(N);
  for (int32_t r = 0; r < N; ++r) {
    int64_t s = 0;
    if (r > 0) s = std::max(s, lx.L[r]);
    if (r + 1 < N) s = std::max(s, lx.L[r + 1]);
    u[r] = lx.len[r] - s;
  }
  std::stable_sort(by_u.begin(), by_u.end(), [&](int32_t a, int32_t b) { return u[a] > u[b]; });
  return {asc, desc, by_len, by_u};
}

Groups sparse_repair(const Lex& lx, int64_t T, Groups g) {
  const int32_t N = lx.N;
  std::vector<int32_t> where(N);
  for (size_t i = 0; i < g.size(); ++i)
    for (const int32_t r : g[i]) where[r] = static_cast<int32_t>(i);
  for (int it = 0; it < 4; ++it) {
    bool found = false;
    bool is_move = true;
    std::tuple<int64_t, int32_t, int32_t> bk;
    for (int32_t r = 0; r < N; ++r) {
      const int32_t a = where[r];
      if (g[a].size() < 2) continue;
      std::set<int32_t> near;
      for (int32_t x = std::max(0, r - kH); x < std::min(N, r + kH + 1); ++x)
        if (x != r && where[x] != a) near.insert(where[x]);
      const int64_t wa0 = lx.work(g[a]);
      std::vector<int32_t> na = g[a];
      erase_one(na, r);
      const int64_t wa = lx.work(na);
      for (const int32_t b : near) {
        std::vector<int32_t> nb = g[b];
        insert_sorted(nb, r);
        const int64_t wb = lx.work(nb);
        if (wb > T) continue;
        const int64_t gain = wa0 + lx.work(g[b]) - wa - wb;
        const auto key = std::make_tuple(-gain, r, b);
        if (gain > 0 && (!found || key < bk)) { bk = key; found = true; }
      }
    }
    if (!found) {
      is_move = false;
      for (int32_t r = 0; r < N; ++r)
        for (int32_t s = r + 1; s < std::min(N, r + kH + 1); ++s) {
          const int32_t a = where[r], b = where[s];
          if (a == b) continue;
          std::vector<int32_t> na = g[a], nb = g[b];
          erase_one(na, r);
          insert_sorted(na, s);
          erase_one(nb, s);
          insert_sorted(nb, r);
          const int64_t wa = lx.work(na), wb = lx.work(nb);
          if (wa > T || wb > T) continue;
          const int64_t gain = lx.work(g[a]) + lx.work(g[b]) - wa - wb;
          const auto key = std::make_tuple(-gain, r, s);
          if (gain > 0 && (!found || key < bk)) { bk = key; found = true; }
        }
    }
    if (!found) break;
    const int32_t r = std::get<1>(bk), x = std::get<2>(bk);
    if (is_move) {
      const int32_t a = where[r], b = x;
      erase_one(g[a], r);
      insert_sorted(g[b], r);
      where[r] = b;
    } else {
      const int32_t s = x, a = where[r], b = where[s];
      erase_one(g[a], r);
      insert_sorted(g[a], s);
      erase_one(g[b], s);
      insert_sorted(g[b], r);
      where[r] = b;
      where[s] = a;
    }
  }
  return g;
}

Parts boundary_refine(const Lex& lx, int64_t T, Parts parts) {
  for (int sweep = 0; sweep < 2; ++sweep) {
    bool moved = false;
    for (size_t i = 0; i + 1 < parts.size(); ++i) {
      const int32_t a = parts[i].first, b = parts[i + 1].second, cut = parts[i].second + 1;
      bool have = false;
      std::tuple<int64_t, int64_t, int32_t> best;
      for (int32_t t = std::max(a + 1, cut - kH); t <= std::min(b, cut + kH); ++t) {
        const int64_t wl = lx.W(a, t - 1), wr = lx.W(t, b);
        if (wl > T || wr > T) continue;
        const auto key = std::make_tuple(wl + wr, std::max(wl, wr), t);
        if (!have || key < best) { best = key; have = true; }
      }
      if (have && std::get<2>(best) != cut) {
        const int32_t t = std::get<2>(best);
        parts[i] = {a, t - 1};
        parts[i + 1] = {t, b};
        moved = true;
      }
    }
    if (!moved) break;
  }
  return parts;
}

struct Assigned {
  int64_t J[3];
  std::vector<int32_t> replica, slot;
  std::vector<int64_t> work;
};

Assigned assign(const Lex& lx, const Groups& g, int32_t D) {
  const int32_t K = static_cast<int32_t>(g.size());
  Assigned A;
  A.work.resize(K);
  for (int32_t i = 0; i < K; ++i) A.work[i] = lx.work(g[i]);
  std::vector<int32_t> order(K);
  for (int32_t i = 0; i < K; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return A.work[a] > A.work[b]; });
  std::vector<int64_t> cum(D, 0);
  A.replica.assign(K, 0);
  A.slot.assign(K, 0);
  int64_t slot_max = 0, total = 0;
  for (int32_t j = 0; j < K / D; ++j) {
    std::vector<int32_t> reps(D);
    for (int32_t d = 0; d < D; ++d) reps[d] = d;
    std::stable_sort(reps.begin(), reps.end(), [&](int32_t a, int32_t b) { return cum[a] < cum[b]; });
    int64_t mx = 0;
    for (int32_t k = 0; k < D; ++k) {
      const int32_t gi = order[j * D + k], d = reps[k];
      A.replica[gi] = d;
      A.slot[gi] = j;
      cum[d] += A.work[gi];
      mx = std::max(mx, A.work[gi]);
    }
    slot_max += mx;
  }
  for (int32_t i = 0; i < K; ++i) total += A.work[i];
  A.J[0] = total;
  A.J[1] = slot_max;
  A.J[2] = *std::max_element(cum.begin(), cum.end());
  return A;
}

}  // namespace

extern "C" int harts_mb_plan(int32_t n_traj, const int64_t* tok_off, const int32_t* tokens, int32_t D,
                             int64_t T, int32_t exact_max, int32_t* group, int32_t* mb_replica,
                             int32_t* mb_slot, int64_t* mb_work, harts_mb_result* result) {
  if (!tok_off || !tokens || !group || !mb_replica || !mb_slot || !mb_work || !result) {
    set_error("harts_mb_plan: NULL argument");
    return HARTS_EINVAL;
  }
  if (D < 1 || T < 1 || n_traj < D || exact_max < 0) {
    set_error("harts_mb_plan: need D >= 1, T >= 1, n_traj >= D and exact_max >= 0");
    return HARTS_EINVAL;
  }
  for (int32_t i = 0; i < n_traj; ++i) {
    const int64_t len = tok_off[i + 1] - tok_off[i];
    if (tok_off[i] < 0 || len < 1 || len > T) {
      set_error("harts_mb_plan: trajectory " + std::to_string(i) + " is empty or above the capacity");
      return HARTS_EINVAL;
    }
  }
  try {
    const int32_t n0 = exact_max ? exact_max : kN0;
    Lex lx;
    lx.build(n_traj, tok_off, tokens);
    const int32_t N = n_traj;
    const Parts P0 = natural_partition(lx, T);
    const int64_t G = lx.W(0, N - 1);
    const int64_t K0 = static_cast<int64_t>(P0.size());
    const int64_t kmin = D * std::max<int64_t>(1, (G + T * D - 1) / (T * D));
    const int64_t kmax = std::max(kmin, std::min<int64_t>(D * ((K0 + D - 1) / D), static_cast<int64_t>(D) * (N / D)));
    std::vector<int32_t> Ks;
    for (int64_t K = kmin; K <= kmax; K += D) Ks.push_back(static_cast<int32_t>(K));
    std::vector<Groups> cands;
    std::vector<Parts> evolved;
    if (N <= n0) {
      for (const auto& kp : exact_dp(lx, T, Ks)) cands.push_back(to_groups(kp.second));
    } else {
      for (const int32_t K : sampled_ks(Ks)) {
        Parts parts = P0;
        if (evolve(lx, T, parts, K)) {
          evolved.push_back(parts);
          cands.push_back(to_groups(parts));
        }
      }
    }
    bool have_g = false;
    Groups gbest;
    std::pair<int64_t, int64_t> gkey;
    for (const auto& order : greedy_orders(lx))
      for (const bool bf : {true, false}) {
        Groups g;
        if (!greedy(lx, T, D, order, bf, g)) continue;
        int64_t tot = 0;
        for (const auto& m : g) tot += lx.work(m);
        const auto key = std::make_pair(static_cast<int64_t>(g.size()), tot);
        if (!have_g || key < gkey) { gkey = key; gbest = g; have_g = true; }
      }
    if (!evolved.empty()) {
      std::vector<int32_t> picks;
      std::vector<int64_t> works;
      for (const auto& p : evolved) {
        int64_t w = 0;
        for (const auto& ab : p) w += lx.W(ab.first, ab.second);
        works.push_back(w);
      }
      const int64_t kg = have_g ? gkey.first : -1;
      auto picked = [&](int32_t i) { return std::find(picks.begin(), picks.end(), i) != picks.end(); };
      if (have_g)
        for (size_t i = 0; i < evolved.size(); ++i)
          if (static_cast<int64_t>(evolved[i].size()) == kg) { picks.push_back(static_cast<int32_t>(i)); break; }
      {
        int32_t bi = -1;
        for (size_t i = 0; i < evolved.size(); ++i)
          if (!picked(static_cast<int32_t>(i)) && (bi < 0 || works[i] < works[bi])) bi = static_cast<int32_t>(i);
        if (bi >= 0) picks.push_back(bi);
      }
      if (have_g) {
        int32_t bi = -1;
        int64_t bd = 0;
        for (size_t i = 0; i < evolved.size(); ++i) {
          if (picked(static_cast<int32_t>(i))) continue;
          const int64_t dd = std::llabs(static_cast<int64_t>(evolved[i].size()) - kg);
          if (bi < 0 || dd < bd) { bd = dd; bi = static_cast<int32_t>(i); }
        }
        if (bi >= 0) picks.push_back(bi);
      }
      for (size_t k = 0; k < picks.size() && static_cast<int32_t>(k) < kBref; ++k)
        cands.push_back(sparse_repair(lx, T, to_groups(boundary_refine(lx, T, evolved[picks[k]]))));
    }
    if (have_g) cands.push_back(sparse_repair(lx, T, gbest));
    int32_t best = -1;
    Assigned bestA;
    for (size_t c = 0; c < cands.size(); ++c) {
      const Groups& g = cands[c];
      if (g.empty() || g.size() % D) continue;
      bool fits = true;
      for (const auto& m : g) fits = fits && !m.empty() && lx.work(m) <= T;
      if (!fits) continue;
      Assigned A = assign(lx, g, D);
      if (best < 0 || std::lexicographical_compare(A.J, A.J + 3, bestA.J, bestA.J + 3)) {
        best = static_cast<int32_t>(c);
        bestA = std::move(A);
      }
    }
    if (best < 0) {
      set_error("harts_mb_plan: no feasible plan");
      return HARTS_EINVAL;
    }
    const Groups& g = cands[best];
    for (size_t gi = 0; gi < g.size(); ++gi) {
      for (const int32_t r : g[gi]) group[lx.order[r]] = static_cast<int32_t>(gi);
      mb_replica[gi] = bestA.replica[gi];
      mb_slot[gi] = bestA.slot[gi];
      mb_work[gi] = bestA.work[gi];
    }
    result->K = static_cast<int32_t>(g.size());
    result->work_total = bestA.J[0];
    result->slot_critical = bestA.J[1];
    result->replica_max = bestA.J[2];
    result->natural_K = static_cast<int32_t>(K0);
    result->trie_work = G;
  } catch (const std::bad_alloc&) {
    set_error("harts_mb_plan: out of host memory");
    return HARTS_ENOMEM;
  }
  set_error("");
  return HARTS_OK;
}
