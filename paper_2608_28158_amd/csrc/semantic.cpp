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


// Asymmetric Q/KV views for full attention (Sec. 4.2, eqs. asymmetric-qkv
// and bottom-right): one view per input sequence of the plan.  Its queries
// are the sequence's own rows; its key/value row lists the physical rows of
// the trajectory positions before its first own token (its h ancestors),
// then its own rows.
namespace {

// Physical rows of the trajectory positions [0, upto) of segment v's path.
void ancestor_rows(const harts_plan_t* p, int32_t v, std::vector<int32_t>& path, std::vector<int32_t>& out) {
  path.clear();
  for (int32_t u = p->parent[v]; u >= 0; u = p->parent[u]) path.push_back(u);
  out.clear();
  for (auto it = path.rbegin(); it != path.rend(); ++it) {
    const int32_t u = *it;
    const int64_t len = p->seg_end[u] - p->seg_start[u];
    for (int64_t k = 0; k < len; ++k) out.push_back(static_cast<int32_t>(p->seg_row[u] + k));
  }
}

constexpr int64_t kAttnTile = 128;   // rows a workgroup owns

void sort_tiles(int32_t* tiles, const std::vector<int64_t>& work) {
  const size_t n = work.size();
  std::vector<size_t> ord(n);
  for (size_t j = 0; j < n; ++j) ord[j] = j;
  std::stable_sort(ord.begin(), ord.end(), [&](size_t a, size_t b) { return work[a] > work[b]; });
  std::vector<int32_t> tmp(tiles, tiles + 2 * n);
  for (size_t j = 0; j < n; ++j) {
    tiles[2 * j] = tmp[2 * ord[j]];
    tiles[2 * j + 1] = tmp[2 * ord[j] + 1];
  }
}

}  // namespace

extern "C" int harts_attn_layout(const harts_plan_t* p, harts_attn_sizes* out) {
  if (!p || !out) {
    set_error("harts_attn_layout: NULL argument");
    return HARTS_EINVAL;
  }
  int64_t n_kv = 0, nq = 0, nk = 0;
  for (int32_t i = 0; i < p->n_seq; ++i) {
    const int32_t first = p->chain_seg[p->seq_chain_off[i]];
    const int64_t h = p->seg_start[first], l = p->seq_n_own[i];
    n_kv += h + l;
    nq += (l + kAttnTile - 1) / kAttnTile;
    nk += (h + l + kAttnTile - 1) / kAttnTile;
  }
  if (n_kv >= INT32_MAX || p->C >= INT32_MAX) {
    set_error("harts_attn_layout: more than 2^31 - 1 view rows");
    return HARTS_EUNSUPPORTED;
  }
  out->n_views = p->n_seq;
  out->n_kv = n_kv;
  out->n_qtiles = nq;
  out->n_kvtiles = nk;
  return HARTS_OK;
}

extern "C" int harts_attn_views(const harts_plan_t* p, int32_t* views, int32_t* kv_rows, int32_t* qtiles,
                                int32_t* kvtiles, int64_t* row_off, int32_t* row_ent) {
  harts_attn_sizes lay;
  if (int rc = harts_attn_layout(p, &lay)) return rc;
  if (!views || !kv_rows || !qtiles || !kvtiles || !row_off || !row_ent) {
    set_error("harts_attn_views: NULL argument");
    return HARTS_EINVAL;
  }
  try {
    std::vector<int32_t> path, anc;
    std::vector<int64_t> qwork, kwork;   // keys a query tile steps over; queries a key tile does
    int64_t off = 0, nq = 0, nk = 0;
    for (int32_t i = 0; i < p->n_seq; ++i) {
      const int32_t first = p->chain_seg[p->seq_chain_off[i]];
      ancestor_rows(p, first, path, anc);
      const int64_t h = static_cast<int64_t>(anc.size()), l = p->seq_n_own[i];
      views[4 * i + 0] = static_cast<int32_t>(p->seq_row[i]);
      views[4 * i + 1] = static_cast<int32_t>(l);
      views[4 * i + 2] = static_cast<int32_t>(off);
      views[4 * i + 3] = static_cast<int32_t>(h);
      for (int64_t k = 0; k < h; ++k) kv_rows[off + k] = anc[k];
      for (int64_t k = 0; k < l; ++k) kv_rows[off + h + k] = static_cast<int32_t>(p->seq_row[i] + k);
      for (int64_t t0 = 0; t0 < l; t0 += kAttnTile, ++nq) {
        qtiles[2 * nq] = i;
        qtiles[2 * nq + 1] = static_cast<int32_t>(t0);
        qwork.push_back(h + t0);
      }
      for (int64_t k0 = 0; k0 < h + l; k0 += kAttnTile, ++nk) {
        kvtiles[2 * nk] = i;
        kvtiles[2 * nk + 1] = static_cast<int32_t>(k0);
        kwork.push_back(l - std::max<int64_t>(0, k0 - h));
      }
      off += h + l;
    }
    // heaviest tiles first (fewer stragglers at the end of a launch); ties
    // keep the view order
    sort_tiles(qtiles, qwork);
    sort_tiles(kvtiles, kwork);
    // view entries of every compact row, ascending
    const int64_t C = p->C;
    std::fill(row_off, row_off + C + 1, 0);
    for (int64_t e = 0; e < off; ++e) ++row_off[kv_rows[e] + 1];
    for (int64_t r = 0; r < C; ++r) row_off[r + 1] += row_off[r];
    std::vector<int64_t> fill(row_off, row_off + C);
    for (int64_t e = 0; e < off; ++e) row_ent[fill[kv_rows[e]]++] = static_cast<int32_t>(e);
  } catch (const std::bad_alloc&) {
    set_error("harts_attn_views: out of host memory");
    return HARTS_ENOMEM;
  }
  set_error("");
  return HARTS_OK;
}
