// Views of a plan's compact rows (host).
//
// Compact-to-semantic map (HARTS, Sec. 3.5): every nonterminal
// semantic position of the original batch, in its original order, with the
// compact row that holds its logits and the token that follows it in its
// trajectory; and, per compact row, the positions it serves (the gradient
// of a shared logit row sums over them, eq. mapped-logp-grad).
//
// Linear in the number of semantic positions S.
//
// Causal-convolution context (Sec. 4.2): the predecessors of every row on
// its own trajectory, and the transposed table of consumers.
#include <algorithm>
#include <cstdint>
#include <new>
#include <string>
#include <vector>

#include "harts.h"
#include "plan.hpp"

using harts::set_error;

extern "C" int harts_semantic_map(const harts_plan_t* p, const int32_t* tokens, int64_t n_pos,
                                  int32_t* m, int32_t* y, int64_t* row_off, int32_t* row_pos) {
  if (!p || !tokens || !m || !y || !row_off || !row_pos) {
    set_error("harts_semantic_map: NULL argument");
    return HARTS_EINVAL;
  }
  const int64_t want = p->S - p->n_leaves;
  if (n_pos != want) {
    set_error("harts_semantic_map: n_pos must be S - n_leaves = " + std::to_string(want));
    return HARTS_EINVAL;
  }
  if (p->C > INT32_MAX || n_pos > INT32_MAX) {
    set_error("harts_semantic_map: more than 2^31 - 1 rows or positions");
    return HARTS_EUNSUPPORTED;
  }
  try {
    // positions in batch order: trajectories by ascending leaf id, each from
    // its root; position t of a trajectory is served by the physical row of
    // its token and predicts the token of position t + 1
    std::vector<int32_t> path;
    int64_t s = 0;
    for (const int32_t leaf : p->leaf_seg) {
      path.clear();
      for (int32_t v = leaf; v >= 0; v = p->parent[v]) path.push_back(v);
      std::reverse(path.begin(), path.end());
      int64_t prev = -1;  // physical row of the previous position
      for (const int32_t v : path) {
        const int64_t r0 = p->seg_row[v];
        const int64_t len = p->seg_end[v] - p->seg_start[v];
        for (int64_t i = 0; i < len; ++i) {
          const int64_t row = r0 + i;
          if (prev >= 0) {
            m[s] = static_cast<int32_t>(prev);
            y[s] = tokens[row];
            ++s;
          }
          prev = row;
        }
      }
    }
    if (s != n_pos) {
      set_error("harts_semantic_map: internal position count mismatch");
      return HARTS_EINVAL;
    }
    // per compact row, its positions ordered by (next token, position):
    // a counting sort by row, then a sort within each row (rows serve as
    // many positions as trajectories pass through them)
    const int64_t C = p->C;
    std::fill(row_off, row_off + C + 1, 0);
    for (int64_t j = 0; j < n_pos; ++j) ++row_off[m[j] + 1];
    for (int64_t c = 0; c < C; ++c) row_off[c + 1] += row_off[c];
    std::vector<int64_t> fill(row_off, row_off + C);
    for (int64_t j = 0; j < n_pos; ++j) row_pos[fill[m[j]]++] = static_cast<int32_t>(j);
    for (int64_t c = 0; c < C; ++c) {
      int32_t* b = row_pos + row_off[c];
      int32_t* e = row_pos + row_off[c + 1];
      if (e - b > 1)
        std::sort(b, e, [&](int32_t a, int32_t d) { return y[a] != y[d] ? y[a] < y[d] : a < d; });
    }
  } catch (const std::bad_alloc&) {
    set_error("harts_semantic_map: out of host memory");
    return HARTS_ENOMEM;
  }
  set_error("");
  return HARTS_OK;
}

extern "C" int harts_conv_context(const harts_plan_t* p, int32_t w, int32_t* pred, int64_t* succ_off,
                                  int32_t* succ) {
  if (!p || !pred || !succ_off || !succ) {
    set_error("harts_conv_context: NULL argument");
    return HARTS_EINVAL;
  }
  if (w < 2 || w > 8) {
    set_error("harts_conv_context: width must be in [2, 8]");
    return HARTS_EUNSUPPORTED;
  }
  if (p->C >= (int64_t{1} << 28)) {
    set_error("harts_conv_context: need fewer than 2^28 rows");
    return HARTS_EUNSUPPORTED;
  }
  try {
    const int32_t n = p->n_seg;
    const int64_t C = p->C;
    const int k = w - 1;
    // anc[v][j - 1] = physical row of trajectory position s_v - j, j = 1..k
    // (-1 before the trajectory start); parents first
    std::vector<std::vector<int32_t>> kids(n);
    std::vector<int32_t> roots;
    for (int32_t v = 0; v < n; ++v) (p->parent[v] >= 0 ? kids[p->parent[v]] : roots).push_back(v);
    std::vector<int32_t> anc(static_cast<size_t>(n) * k, -1), stack(roots.rbegin(), roots.rend());
    while (!stack.empty()) {
      const int32_t v = stack.back();
      stack.pop_back();
      const int32_t u = p->parent[v];
      if (u >= 0) {
        const int64_t lu = p->seg_end[u] - p->seg_start[u];
        for (int j = 1; j <= k; ++j)
          anc[static_cast<size_t>(v) * k + j - 1] =
              j <= lu ? static_cast<int32_t>(p->seg_row[u] + lu - j) : anc[static_cast<size_t>(u) * k + j - lu - 1];
      }
      for (auto it = kids[v].rbegin(); it != kids[v].rend(); ++it) stack.push_back(*it);
    }
    for (int32_t v = 0; v < n; ++v) {
      const int64_t len = p->seg_end[v] - p->seg_start[v];
      for (int64_t t = 0; t < len; ++t) {
        const int64_t row = p->seg_row[v] + t;
        for (int i = 1; i <= k; ++i)
          pred[row * k + i - 1] = i <= t ? static_cast<int32_t>(row - i) : anc[static_cast<size_t>(v) * k + i - t - 1];
      }
    }
    // consumers of each row, ordered by (tap, consumer row): counting sort
    std::fill(succ_off, succ_off + C + 1, 0);
    for (int64_t s = 0; s < C; ++s)
      for (int i = 1; i <= k; ++i)
        if (pred[s * k + i - 1] >= 0) ++succ_off[pred[s * k + i - 1] + 1];
    for (int64_t r = 0; r < C; ++r) succ_off[r + 1] += succ_off[r];
    std::vector<int64_t> fill(succ_off, succ_off + C);
    for (int i = 1; i <= k; ++i)
      for (int64_t s = 0; s < C; ++s) {
        const int32_t r = pred[s * k + i - 1];
        if (r >= 0) succ[fill[r]++] = static_cast<int32_t>(s * 8 + i);
      }
  } catch (const std::bad_alloc&) {
    set_error("harts_conv_context: out of host memory");
    return HARTS_ENOMEM;
  }
  set_error("");
  return HARTS_OK;
}

