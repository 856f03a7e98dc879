// Compact-to-semantic map of a plan (HARTS, Sec. 3.5): every nonterminal
// semantic position of the original batch, in its original order, with the
// compact row that holds its logits and the token that follows it in its
// trajectory; and, per compact row, the positions it serves (the gradient
// of a shared logit row sums over them, eq. mapped-logp-grad).
//
// Linear in the number of semantic positions S.
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
