// Host planner: minimum-call planning and plan recovery (HARTS, Sec. 3.3,
// Algorithm "minimum-call"), plus the physical row layout, replay row maps,
// requested-state slots and the device descriptor image consumed by the
// packed linear-attention calls.
//
// Everything is iterative (segment chains can be arbitrarily deep) and
// linear in the number of segments plus the replay length.
#include <algorithm>
#include <climits>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "plan.hpp"

namespace harts {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }

namespace {

constexpr int64_t kAlignWords = 64;  // 256-byte sections in the blob

int64_t align_up(int64_t x) { return (x + kAlignWords - 1) / kAlignWords * kAlignWords; }

inline int64_t anchor_of(int64_t p, int64_t B) { return (p / B) * B; }  // eq. resume-anchor

}  // namespace

// Block target of a round: enough blocks that the (block, head) work units
// fill the GPU about 3.5 times over (896 workgroups: 56 blocks at 16 heads).
// Larger blocks move fewer block states through HBM and start fewer
// workgroups (each reads a start state before its first chunk); smaller
// ones expose more workgroups.  56 blocks measured best on the 64k-token
// agentic workload at 16 heads: 48-chunk blocks in its long-sequence round,
// 1.777 ms per step against 1.797 ms with 16-chunk blocks (80 blocks).
int32_t default_min_blocks(int32_t H) {
  constexpr int32_t kTargetUnits = 56 * 16;
  return std::max<int32_t>(1, (kTargetUnits + H - 1) / H);
}

namespace {

struct Builder {
  int32_t n;
  int64_t B;
  const int32_t* parent;
  const int64_t* len;
  std::vector<int32_t> kid_off, kids, roots;  // children by ascending id
  std::vector<int32_t> pre;                   // preorder, trees in root order
  std::vector<int32_t> tpre, tin, direct;
  harts_plan_s* P;

  bool children_and_positions() {
    std::vector<int32_t> cnt(n + 1, 0);
    for (int32_t v = 0; v < n; ++v) {
      const int32_t p = parent[v];
      if (p < -1 || p >= n || p == v) {
        set_error("harts_plan: parent of segment " + std::to_string(v) + " is invalid");
        return false;
      }
      if (len[v] <= 0) {
        set_error("harts_plan: segment " + std::to_string(v) + " has length <= 0");
        return false;
      }
      if (p >= 0) ++cnt[p + 1];
      else roots.push_back(v);
    }
    if (roots.empty()) {
      set_error("harts_plan: the parent array has no root (cycle)");
      return false;
    }
    kid_off.assign(n + 1, 0);
    for (int32_t v = 0; v < n; ++v) kid_off[v + 1] = kid_off[v] + cnt[v + 1];
    kids.assign(kid_off[n], 0);
    std::vector<int32_t> fill(kid_off.begin(), kid_off.end() - 1);
    for (int32_t v = 0; v < n; ++v)  // ascending v keeps children sorted by id
      if (parent[v] >= 0) kids[fill[parent[v]]++] = v;

    P->seg_start.assign(n, 0);
    P->seg_end.assign(n, 0);
    P->seg_tree.assign(n, -1);
    pre.reserve(n);
    std::vector<int32_t> stack;
    for (size_t t = 0; t < roots.size(); ++t) {
      stack.push_back(roots[t]);
      while (!stack.empty()) {
        const int32_t v = stack.back();
        stack.pop_back();
        const int64_t s = parent[v] >= 0 ? P->seg_end[parent[v]] : 0;
        if (s > (INT64_MAX / 4) - len[v]) {
          set_error("harts_plan: trajectory positions overflow");
          return false;
        }
        P->seg_start[v] = s;
        P->seg_end[v] = s + len[v];
        P->seg_tree[v] = static_cast<int32_t>(t);
        pre.push_back(v);
        for (int32_t j = kid_off[v + 1] - 1; j >= kid_off[v]; --j) stack.push_back(kids[j]);
      }
    }
    if (static_cast<int32_t>(pre.size()) != n) {
      set_error("harts_plan: the parent array has a cycle");
      return false;
    }
    return true;
  }

  // Dynamic program of eqs. leaf-calls, tin and tpre, children before parents.
  // The largest and second-largest child T_pre give every max_{u != o} in O(1).
  void dynamic_program() {
    tpre.assign(n, 0);
    tin.assign(n, 0);
    for (int32_t i = n - 1; i >= 0; --i) {
      const int32_t v = pre[i];
      const int32_t b = kid_off[v], e = kid_off[v + 1];
      if (b == e) {
        tpre[v] = tin[v] = 1;
        continue;
      }
      int32_t m1 = 0, m2 = 0, n_m1 = 0;
      for (int32_t j = b; j < e; ++j) {
        const int32_t x = tpre[kids[j]];
        if (x > m1) { m2 = m1; m1 = x; n_m1 = 1; }
        else if (x == m1) { ++n_m1; }
        else if (x > m2) { m2 = x; }
      }
      if (n_m1 > 1) m2 = m1;
      int32_t best = INT32_MAX;
      for (int32_t j = b; j < e; ++j) {
        const int32_t o = kids[j];
        const int32_t h = (e - b == 1) ? 0 : (tpre[o] == m1 ? m2 : m1);
        best = std::min(best, std::max(tin[o], 1 + h));
      }
      tin[v] = best;
      const bool early = P->seg_end[v] < anchor_of(P->seg_start[v], B) + B;  // eq. early-start
      tpre[v] = early ? m1 : best;
    }
  }

  struct SeqTmp {
    int32_t tree, round, first, creation;
    int64_t anchor;
    int32_t init_kind;   // 0 tree, 1 slot
    int32_t init_a;      // tree index, or producer creation index
    int64_t init_pos;    // boundary position for a slot
  };
  std::vector<SeqTmp> seqs;
  std::vector<std::pair<int32_t, int64_t>> requests;  // (producer creation, position)

  // Recover, as an explicit stack that visits exactly what the recursive
  // procedure visits, in the same order.
  bool recover() {
    direct.assign(n, -1);
    struct Frame {
      int32_t v, seq, K, r;
      bool ready, entered, same;
      int32_t o, next;  // chosen direct child; next child slot to launch
    };
    std::vector<Frame> st;
    P->tree_calls.assign(roots.size(), 0);
    for (size_t t = 0; t < roots.size(); ++t) {
      const int32_t root = roots[t];
      const int32_t K = tpre[root];
      P->tree_calls[t] = K;
      seqs.push_back({static_cast<int32_t>(t), 1, root, static_cast<int32_t>(seqs.size()), 0, 0,
                      static_cast<int32_t>(t), 0});
      st.push_back({root, static_cast<int32_t>(seqs.size() - 1), K, 1, true, false, false, -1, 0});
      while (!st.empty()) {
        Frame& f = st.back();
        const int32_t v = f.v;
        const int32_t b = kid_off[v], e = kid_off[v + 1];
        if (!f.entered) {
          f.entered = true;
          if (b == e) { st.pop_back(); continue; }  // leaf: sequence ends here
          const int64_t av = anchor_of(P->seg_start[v], B);
          f.same = f.ready && (P->seg_end[v] < av + B);
          const int32_t delta = f.same ? 0 : 1;
          const int32_t K_side = f.K - delta;
          int32_t over = 0;
          for (int32_t j = b; j < e; ++j) over += tpre[kids[j]] > K_side ? 1 : 0;
          int32_t o = -1;
          for (int32_t j = b; j < e && o < 0; ++j) {
            const int32_t c = kids[j];
            const int32_t need = f.same ? tpre[c] : tin[c];
            if (need <= f.K && over - (tpre[c] > K_side ? 1 : 0) == 0) o = c;
          }
          if (o < 0) {
            set_error("harts_plan: internal error, no feasible direct continuation");
            return false;
          }
          f.o = o;
          f.next = b;
          direct[v] = o;
          const Frame child{o, f.seq, f.K, f.r, f.same, false, false, -1, 0};
          st.push_back(child);
          continue;
        }
        // side children, in child order, after the direct continuation
        int32_t j = f.next;
        while (j < e && kids[j] == f.o) ++j;
        if (j >= e) { st.pop_back(); continue; }
        f.next = j + 1;
        const int32_t u = kids[j];
        const int64_t bv = anchor_of(P->seg_end[v], B);
        const SeqTmp& parent_seq = seqs[f.seq];
        SeqTmp s{parent_seq.tree, 0, u, static_cast<int32_t>(seqs.size()), bv, 0, 0, 0};
        if (f.same) {
          s.round = f.r;
          s.init_kind = parent_seq.init_kind;
          s.init_a = parent_seq.init_a;
          s.init_pos = parent_seq.init_pos;
        } else {
          s.round = f.r + 1;
          s.init_kind = 1;
          s.init_a = f.seq;
          s.init_pos = bv;
          requests.emplace_back(f.seq, bv);
        }
        const int32_t delta = f.same ? 0 : 1;
        const Frame child{u, s.creation, f.K - delta, f.r + delta, true, false, false, -1, 0};
        seqs.push_back(s);
        st.push_back(child);
      }
    }
    return true;
  }

  bool finish() {
    harts_plan_s& p = *P;
    const int32_t n_seq = static_cast<int32_t>(seqs.size());
    int32_t K = 0;
    for (const auto& s : seqs) K = std::max(K, s.round);
    p.K = K;
    p.n_seq = n_seq;
    p.n_trees = static_cast<int32_t>(roots.size());
    // stable counting sort of creation order by round
    std::vector<int32_t> cnt(K + 2, 0);
    for (const auto& s : seqs) ++cnt[s.round];
    p.round_seq_off.assign(K + 1, 0);
    for (int32_t r = 1; r <= K; ++r) p.round_seq_off[r] = p.round_seq_off[r - 1] + cnt[r];
    std::vector<int32_t> id_of(n_seq), pos(p.round_seq_off.begin(), p.round_seq_off.end() - 1);
    std::vector<int32_t> order(n_seq);
    for (int32_t c = 0; c < n_seq; ++c) {
      const int32_t id = pos[seqs[c].round - 1]++;
      id_of[c] = id;
      order[id] = c;
    }
    // slots: dedupe (producer id, position), sorted
    std::vector<std::pair<int32_t, int64_t>> keys;
    keys.reserve(requests.size());
    for (const auto& rq : requests) keys.emplace_back(id_of[rq.first], rq.second);
    std::sort(keys.begin(), keys.end());
    keys.erase(std::unique(keys.begin(), keys.end()), keys.end());
    p.n_slots = static_cast<int32_t>(keys.size());
    p.n_bank = p.n_trees + p.n_slots;
    p.slot_seq.resize(keys.size());
    p.slot_pos.resize(keys.size());
    for (size_t j = 0; j < keys.size(); ++j) {
      p.slot_seq[j] = keys[j].first;
      p.slot_pos[j] = keys[j].second;
    }
    auto slot_index = [&](int32_t producer_id, int64_t position) -> int32_t {
      auto it = std::lower_bound(keys.begin(), keys.end(), std::make_pair(producer_id, position));
      return static_cast<int32_t>(it - keys.begin());
    };
    // leaves
    std::vector<int32_t> leaf_index(n, -1);
    for (int32_t v = 0; v < n; ++v)
      if (kid_off[v] == kid_off[v + 1]) {
        leaf_index[v] = static_cast<int32_t>(p.leaf_seg.size());
        p.leaf_seg.push_back(v);
      }
    p.n_leaves = static_cast<int32_t>(p.leaf_seg.size());
    // per-sequence fields, chains and physical rows
    p.seq_round.resize(n_seq);
    p.seq_tree.resize(n_seq);
    p.seq_first_seg.resize(n_seq);
    p.seq_final_leaf.resize(n_seq);
    p.seq_init_bank.resize(n_seq);
    p.seq_anchor.resize(n_seq);
    p.seq_n_replay.resize(n_seq);
    p.seq_replay_off.assign(n_seq + 1, 0);
    p.seq_row.resize(n_seq);
    p.seq_n_own.resize(n_seq);
    p.seq_chain_off.assign(n_seq + 1, 0);
    p.chain_seg.reserve(n);
    p.seg_row.assign(n, 0);
    p.seg_seq.assign(n, -1);
    int64_t row = 0;
    for (int32_t id = 0; id < n_seq; ++id) {
      const SeqTmp& s = seqs[order[id]];
      p.seq_round[id] = s.round;
      p.seq_tree[id] = s.tree;
      p.seq_first_seg[id] = s.first;
      p.seq_anchor[id] = s.anchor;
      p.seq_init_bank[id] = s.init_kind == 0 ? s.init_a
                                              : p.n_trees + slot_index(id_of[s.init_a], s.init_pos);
      p.seq_chain_off[id] = static_cast<int32_t>(p.chain_seg.size());
      p.seq_row[id] = row;
      int32_t v = s.first, last = s.first;
      while (v >= 0) {
        p.chain_seg.push_back(v);
        p.seg_row[v] = row;
        p.seg_seq[v] = id;
        row += len[v];
        last = v;
        v = direct[v];
      }
      p.seq_n_own[id] = row - p.seq_row[id];
      p.seq_final_leaf[id] = leaf_index[last];
      p.seq_n_replay[id] = P->seg_start[s.first] - s.anchor;
    }
    p.seq_chain_off[n_seq] = static_cast<int32_t>(p.chain_seg.size());
    p.C = row;
    // requests grouped by producer (keys are sorted by producer then position)
    p.seq_req_off.assign(n_seq + 1, 0);
    for (const auto& kk : keys) ++p.seq_req_off[kk.first + 1];
    for (int32_t i = 0; i < n_seq; ++i) p.seq_req_off[i + 1] += p.seq_req_off[i];
    p.req_chunk.resize(keys.size());
    p.req_bank.resize(keys.size());
    for (size_t j = 0; j < keys.size(); ++j) {
      const int32_t prod = keys[j].first;
      p.req_chunk[j] = static_cast<int32_t>((keys[j].second - p.seq_anchor[prod]) / B);
      p.req_bank[j] = p.n_trees + static_cast<int32_t>(j);
    }
    // replay rows: positions [anchor, s_first) on the path above the first segment
    int64_t R = 0;
    for (int32_t id = 0; id < n_seq; ++id) {
      p.seq_replay_off[id] = R;
      R += p.seq_n_replay[id];
    }
    p.seq_replay_off[n_seq] = R;
    p.R = R;
    p.replay_row.assign(R, 0);
    for (int32_t id = 0; id < n_seq; ++id) {
      const int32_t first = p.seq_first_seg[id];
      int32_t w = parent[first];
      for (int64_t pos = P->seg_start[first] - 1, j = p.seq_replay_off[id + 1] - 1;
           pos >= p.seq_anchor[id]; --pos, --j) {
        while (pos < P->seg_start[w]) w = parent[w];
        p.replay_row[j] = p.seg_row[w] + pos - P->seg_start[w];
      }
    }
    // multiplicity q_v and semantic positions S
    p.seg_mult.assign(n, 0);
    for (int32_t i = n - 1; i >= 0; --i) {
      const int32_t v = pre[i];
      if (kid_off[v] == kid_off[v + 1]) p.seg_mult[v] = 1;
      if (parent[v] >= 0) p.seg_mult[parent[v]] += p.seg_mult[v];
    }
    p.S = 0;
    for (int32_t l : p.leaf_seg) p.S += P->seg_end[l];
    if (p.C + p.R > INT32_MAX - 2 * B) {
      set_error("harts_plan: packed rows exceed int32 indexing");
      return false;
    }
    p.seg_tpre = tpre;
    p.seg_tin = tin;
    return true;
  }

  // Blocks of a round for a given block size: cuts every L chunks and at
  // every requested boundary.
  int32_t count_blocks(const RoundLayout& L, int32_t bc) const {
    const harts_plan_s& p = *P;
    int64_t total = 0;
    for (int32_t i = L.seq_begin; i < L.seq_begin + L.n_seq; ++i) {
      const int64_t tok = p.seq_n_replay[i] + p.seq_n_own[i];
      const int32_t nc = static_cast<int32_t>((tok + B - 1) / B);
      int32_t c0 = 0, rq = p.seq_req_off[i];
      const int32_t rq_end = p.seq_req_off[i + 1];
      while (c0 < nc) {
        int32_t c1 = std::min(nc, c0 + bc);
        while (rq < rq_end && p.req_chunk[rq] <= c0) ++rq;
        if (rq < rq_end && p.req_chunk[rq] <= c1) c1 = p.req_chunk[rq];
        ++total;
        c0 = c1;
      }
    }
    return static_cast<int32_t>(total);
  }

  void build_blob() {
    harts_plan_s& p = *P;
    p.blob.clear();
    p.rounds.clear();
    const int32_t K = p.K;
    const int32_t min_blocks = p.min_blocks;
    int64_t off = 0;
    p.rounds.assign(K, RoundLayout{});
    p.n_chunks = 0;
    for (int32_t r = 0; r < K; ++r) {
      RoundLayout& L = p.rounds[r];
      L.seq_begin = p.round_seq_off[r];
      L.n_seq = p.round_seq_off[r + 1] - p.round_seq_off[r];
      L.own_row_begin = L.n_seq ? p.seq_row[L.seq_begin] : 0;
      for (int32_t i = L.seq_begin; i < L.seq_begin + L.n_seq; ++i) {
        const int64_t tok = p.seq_n_replay[i] + p.seq_n_own[i];
        const int64_t nc = (tok + B - 1) / B;
        L.n_chunks += nc;
        L.n_rows += tok;
        L.n_own += p.seq_n_own[i];
        L.n_replay += p.seq_n_replay[i];
        L.max_seq_chunks = std::max<int32_t>(L.max_seq_chunks, static_cast<int32_t>(nc));
      }
      p.n_chunks += L.n_chunks;
      // block size: the largest of 64, 48, 32, 24, 16, 12, 8 chunks that
      // still cuts the round into >= min_blocks blocks, so that (block, head)
      // work units fill the GPU and no single block dominates the critical
      // path
      static const int32_t cands[] = {64, 48, 32, 24, 16, 12, 8};
      L.block_chunks = 8;
      for (const int32_t cand : cands) {
        if (count_blocks(L, cand) >= min_blocks) { L.block_chunks = cand; break; }
      }
      L.n_blk = count_blocks(L, L.block_chunks);
      L.seq_tab = off;
      off = align_up(off + int64_t(L.n_seq) * SEQ_WORDS);
      L.init_idx = off;
      off = align_up(off + L.n_seq);
      L.chunk_tab = off;
      off = align_up(off + 2 * L.n_chunks);
      L.blk_tab = off;
      off = align_up(off + int64_t(L.n_blk) * BLK_WORDS);
      L.blk_launch = off;
      off = align_up(off + int64_t(L.n_blk) * LCH_WORDS);
    }
    p.off_replay_row = off;
    off = align_up(off + p.R);
    p.off_req_chunk = off;
    off = align_up(off + int64_t(p.req_chunk.size()));
    p.off_req_bank = off;
    off = align_up(off + int64_t(p.req_bank.size()));
    // replayed compact rows and their replay indices, sorted (for the reduction)
    std::vector<std::pair<int64_t, int64_t>> rr(p.R);
    for (int64_t j = 0; j < p.R; ++j) rr[j] = {p.replay_row[j], j};
    std::sort(rr.begin(), rr.end());
    std::vector<int32_t> red_rows, red_off;
    for (int64_t j = 0; j < p.R; ++j)
      if (j == 0 || rr[j].first != rr[j - 1].first) {
        red_rows.push_back(static_cast<int32_t>(rr[j].first));
        red_off.push_back(static_cast<int32_t>(j));
      }
    red_off.push_back(static_cast<int32_t>(p.R));
    p.n_red = static_cast<int64_t>(red_rows.size());
    p.off_red_rows = off;
    off = align_up(off + p.n_red);
    p.off_red_off = off;
    off = align_up(off + p.n_red + 1);
    p.off_red_idx = off;
    off = align_up(off + p.R);

    p.blob.assign(std::max<int64_t>(off, kAlignWords), 0);
    int32_t* b = p.blob.data();
    for (int32_t r = 0; r < K; ++r) {
      RoundLayout& L = p.rounds[r];
      int64_t chunk_off = 0;
      int64_t blk_next = 0;
      int32_t max_seq_blocks = 0;
      for (int32_t li = 0; li < L.n_seq; ++li) {
        const int32_t i = L.seq_begin + li;
        const int64_t tok = p.seq_n_replay[i] + p.seq_n_own[i];
        const int64_t nc = (tok + B - 1) / B;
        int32_t* e = b + L.seq_tab + int64_t(li) * SEQ_WORDS;
        e[SEQ_CHUNK_OFF] = static_cast<int32_t>(chunk_off);
        e[SEQ_N_TOK] = static_cast<int32_t>(tok);
        e[SEQ_N_REPLAY] = static_cast<int32_t>(p.seq_n_replay[i]);
        e[SEQ_REPLAY_OFF] = static_cast<int32_t>(p.seq_replay_off[i]);
        e[SEQ_OWN_ROW] = static_cast<int32_t>(p.seq_row[i]);
        e[SEQ_INIT_BANK] = p.seq_init_bank[i];
        e[SEQ_FINAL_LEAF] = p.seq_final_leaf[i];
        e[SEQ_REQ_OFF] = p.seq_req_off[i];
        e[SEQ_N_REQ] = p.seq_req_off[i + 1] - p.seq_req_off[i];
        e[SEQ_N_CHUNKS] = static_cast<int32_t>(nc);
        b[L.init_idx + li] = p.seq_init_bank[i];
        // blocks of this sequence
        e[SEQ_BLK_OFF] = static_cast<int32_t>(blk_next);
        int32_t nb = 0;
        int32_t c0 = 0;
        int32_t rq = p.seq_req_off[i];
        const int32_t rq_end = p.seq_req_off[i + 1];
        while (c0 < nc) {
          int32_t c1 = std::min<int32_t>(static_cast<int32_t>(nc), c0 + L.block_chunks);
          while (rq < rq_end && p.req_chunk[rq] <= c0) ++rq;
          int32_t end_bank = -1;
          if (rq < rq_end && p.req_chunk[rq] <= c1) {
            c1 = p.req_chunk[rq];
            end_bank = p.req_bank[rq];
          }
          int32_t* bk = b + L.blk_tab + blk_next * BLK_WORDS;
          bk[BLK_SEQ] = li;
          bk[BLK_C0] = c0;
          bk[BLK_NC] = c1 - c0;
          bk[BLK_IDX] = nb;
          bk[BLK_END_BANK] = end_bank;
          ++blk_next;
          ++nb;
          c0 = c1;
        }
        e[SEQ_N_BLK] = nb;
        max_seq_blocks = std::max(max_seq_blocks, nb);
        for (int64_t c = 0; c < nc; ++c) {
          b[L.chunk_tab + 2 * (chunk_off + c)] = li;
          b[L.chunk_tab + 2 * (chunk_off + c) + 1] = static_cast<int32_t>(c);
        }
        chunk_off += nc;
      }
      L.max_seq_blocks = max_seq_blocks;
      // launch order of the block kernels: longest block first (stable), so
      // that the last workgroups to start are the shortest ones
      std::vector<int32_t> order(L.n_blk);
      for (int32_t j = 0; j < L.n_blk; ++j) order[j] = j;
      const int32_t* bt = b + L.blk_tab;
      std::stable_sort(order.begin(), order.end(), [bt](int32_t x, int32_t y) {
        return bt[x * BLK_WORDS + BLK_NC] > bt[y * BLK_WORDS + BLK_NC];
      });
      for (int32_t j = 0; j < L.n_blk; ++j) {
        const int32_t* bk = bt + order[j] * BLK_WORDS;
        const int32_t* e = b + L.seq_tab + int64_t(bk[BLK_SEQ]) * SEQ_WORDS;
        int32_t* ln = b + L.blk_launch + int64_t(j) * LCH_WORDS;
        ln[LCH_BLK] = order[j];
        ln[LCH_SEQ] = bk[BLK_SEQ];
        ln[LCH_C0] = bk[BLK_C0];
        ln[LCH_NC] = bk[BLK_NC];
        ln[LCH_IDX] = bk[BLK_IDX];
        ln[LCH_N_BLK] = e[SEQ_N_BLK];
        ln[LCH_FINAL_LEAF] = e[SEQ_FINAL_LEAF];
        ln[LCH_INIT_BANK] = e[SEQ_INIT_BANK];
        ln[LCH_N_TOK] = e[SEQ_N_TOK];
        ln[LCH_N_REPLAY] = e[SEQ_N_REPLAY];
        ln[LCH_REPLAY_OFF] = e[SEQ_REPLAY_OFF];
        ln[LCH_OWN_ROW] = e[SEQ_OWN_ROW];
        ln[LCH_CHUNK_OFF] = e[SEQ_CHUNK_OFF];
      }
    }
    for (int64_t j = 0; j < p.R; ++j) b[p.off_replay_row + j] = static_cast<int32_t>(p.replay_row[j]);
    for (size_t j = 0; j < p.req_chunk.size(); ++j) {
      b[p.off_req_chunk + j] = p.req_chunk[j];
      b[p.off_req_bank + j] = p.req_bank[j];
    }
    for (int64_t j = 0; j < p.n_red; ++j) {
      b[p.off_red_rows + j] = red_rows[j];
      b[p.off_red_off + j] = red_off[j];
    }
    b[p.off_red_off + p.n_red] = red_off[p.n_red];
    for (int64_t j = 0; j < p.R; ++j) b[p.off_red_idx + j] = static_cast<int32_t>(rr[j].second);
  }
};

}  // namespace
}  // namespace harts

using harts::set_error;

extern "C" int harts_plan_set_blocks(harts_plan_t* p, int32_t H, int32_t min_blocks) {
  if (!p || H < 1 || min_blocks < 0 || min_blocks > (1 << 20)) {
    set_error("harts_plan_set_blocks: need a plan, H >= 1 and 0 <= min_blocks <= 2^20");
    return HARTS_EINVAL;
  }
  const int32_t target = min_blocks ? min_blocks : harts::default_min_blocks(H);
  if (target == p->min_blocks) return HARTS_OK;
  const int32_t old = p->min_blocks;
  try {
    harts::Builder bld;
    bld.n = p->n_seg;
    bld.B = p->chunk;
    bld.P = p;
    p->min_blocks = target;
    bld.build_blob();
  } catch (const std::bad_alloc&) {
    p->min_blocks = old;
    set_error("harts_plan_set_blocks: out of host memory (the plan's device tables are gone)");
    p->blob.clear();
    p->rounds.clear();
    return HARTS_ENOMEM;
  }
  set_error("");
  return HARTS_OK;
}

extern "C" const char* harts_last_error(void) { return harts::g_last_error.c_str(); }

extern "C" int harts_plan(int32_t n_seg, const int32_t* parent, const int64_t* seg_len,
                          int32_t chunk, harts_plan_t** out) {
  if (!out) { set_error("harts_plan: out is NULL"); return HARTS_EINVAL; }
  *out = nullptr;
  if (n_seg < 1 || !parent || !seg_len) {
    set_error("harts_plan: need n_seg >= 1 and non-NULL parent / seg_len");
    return HARTS_EINVAL;
  }
  if (chunk < 1) { set_error("harts_plan: chunk must be >= 1"); return HARTS_EINVAL; }
  harts_plan_s* p = new (std::nothrow) harts_plan_s();
  if (!p) { set_error("harts_plan: out of host memory"); return HARTS_ENOMEM; }
  try {
    harts::Builder bld;
    bld.n = n_seg;
    bld.B = chunk;
    bld.parent = parent;
    bld.len = seg_len;
    bld.P = p;
    p->n_seg = n_seg;
    p->chunk = chunk;
    p->min_blocks = harts::default_min_blocks(16);
    if (!bld.children_and_positions()) { delete p; return HARTS_EINVAL; }
    bld.dynamic_program();
    if (!bld.recover() || !bld.finish()) { delete p; return HARTS_EINVAL; }
    bld.build_blob();
    p->parent.assign(parent, parent + n_seg);
  } catch (const std::bad_alloc&) {
    delete p;
    set_error("harts_plan: out of host memory");
    return HARTS_ENOMEM;
  }
  set_error("");
  *out = p;
  return HARTS_OK;
}

extern "C" void harts_plan_free(harts_plan_t* plan) { delete plan; }

extern "C" int harts_plan_get_info(const harts_plan_t* p, harts_plan_info* info) {
  if (!p || !info) { set_error("harts_plan_get_info: NULL argument"); return HARTS_EINVAL; }
  info->n_seg = p->n_seg;
  info->n_trees = p->n_trees;
  info->n_leaves = p->n_leaves;
  info->n_rounds = p->K;
  info->n_seq = p->n_seq;
  info->n_slots = p->n_slots;
  info->n_bank = p->n_bank;
  info->chunk = p->chunk;
  info->C = p->C;
  info->S = p->S;
  info->R = p->R;
  info->n_req = static_cast<int64_t>(p->req_chunk.size());
  info->n_chunks = p->n_chunks;
  info->blob_bytes = static_cast<int64_t>(p->blob.size() * sizeof(int32_t));
  return HARTS_OK;
}

template <typename T>
static void copy_out(T* dst, const std::vector<T>& src) {
  if (dst && !src.empty()) std::memcpy(dst, src.data(), src.size() * sizeof(T));
}

extern "C" int harts_plan_export(const harts_plan_t* p, const harts_plan_arrays* d) {
  if (!p || !d) { set_error("harts_plan_export: NULL argument"); return HARTS_EINVAL; }
  copy_out(d->seg_start, p->seg_start);
  copy_out(d->seg_end, p->seg_end);
  copy_out(d->seg_row, p->seg_row);
  copy_out(d->seg_seq, p->seg_seq);
  copy_out(d->seg_mult, p->seg_mult);
  copy_out(d->seg_tpre, p->seg_tpre);
  copy_out(d->seg_tin, p->seg_tin);
  copy_out(d->seg_tree, p->seg_tree);
  copy_out(d->leaf_seg, p->leaf_seg);
  copy_out(d->tree_calls, p->tree_calls);
  copy_out(d->round_seq_off, p->round_seq_off);
  copy_out(d->seq_round, p->seq_round);
  copy_out(d->seq_tree, p->seq_tree);
  copy_out(d->seq_first_seg, p->seq_first_seg);
  copy_out(d->seq_final_leaf, p->seq_final_leaf);
  copy_out(d->seq_init_bank, p->seq_init_bank);
  copy_out(d->seq_anchor, p->seq_anchor);
  copy_out(d->seq_n_replay, p->seq_n_replay);
  copy_out(d->seq_replay_off, p->seq_replay_off);
  copy_out(d->seq_row, p->seq_row);
  copy_out(d->seq_n_own, p->seq_n_own);
  copy_out(d->seq_chain_off, p->seq_chain_off);
  copy_out(d->chain_seg, p->chain_seg);
  copy_out(d->seq_req_off, p->seq_req_off);
  copy_out(d->req_chunk, p->req_chunk);
  copy_out(d->req_bank, p->req_bank);
  copy_out(d->slot_seq, p->slot_seq);
  copy_out(d->slot_pos, p->slot_pos);
  copy_out(d->replay_row, p->replay_row);
  return HARTS_OK;
}

extern "C" int harts_plan_round_info(const harts_plan_t* p, int32_t round, harts_round_info* info) {
  if (!p || !info) { set_error("harts_plan_round_info: NULL argument"); return HARTS_EINVAL; }
  if (round < 0 || round >= p->K) { set_error("harts_plan_round_info: round out of range"); return HARTS_EINVAL; }
  const harts::RoundLayout& L = p->rounds[round];
  info->n_seq = L.n_seq;
  info->seq_begin = L.seq_begin;
  info->n_blk = L.n_blk;
  info->block_chunks = L.block_chunks;
  info->n_chunks = L.n_chunks;
  info->n_rows = L.n_rows;
  info->n_own = L.n_own;
  info->n_replay = L.n_replay;
  info->own_row_begin = L.own_row_begin;
  info->init_idx_off = L.init_idx * static_cast<int64_t>(sizeof(int32_t));
  info->seq_tab_off = L.seq_tab * static_cast<int64_t>(sizeof(int32_t));
  info->blk_tab_off = L.blk_tab * static_cast<int64_t>(sizeof(int32_t));
  info->launch_off = L.blk_launch * static_cast<int64_t>(sizeof(int32_t));
  return HARTS_OK;
}

extern "C" int harts_plan_blob(const harts_plan_t* p, void* host_dst, size_t bytes) {
  if (!p || !host_dst) { set_error("harts_plan_blob: NULL argument"); return HARTS_EINVAL; }
  const size_t need = p->blob.size() * sizeof(int32_t);
  if (bytes < need) { set_error("harts_plan_blob: destination too small"); return HARTS_ENOMEM; }
  std::memcpy(host_dst, p->blob.data(), need);
  return HARTS_OK;
}
