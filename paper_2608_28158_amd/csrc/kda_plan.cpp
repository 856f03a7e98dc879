// Host tables of the KDA path (HARTS, Sec. 2.2 and Sec. 3.4): the plan's
// sequences laid out as packed 64-row chunks, in sequence order (so a
// round's sequences and chunks are contiguous).  A sequence's packed rows
// are its replay rows (trajectory positions [anchor, fork), eq.
// mandatory-replay) followed by its own rows, zero-padded to whole chunks;
// it starts from a bank entry (a tree's initial state or a requested
// boundary state of an earlier round) and writes the states at the start of
// its requested chunks into the bank (eq. chunkla-interface).
#include <algorithm>
#include <cstdint>
#include <new>
#include <string>
#include <vector>

#include "harts.h"
#include "plan.hpp"

using harts::set_error;

namespace {

constexpr int32_t kKdaChunk = 64;

}  // namespace

extern "C" int harts_kda_layout(const harts_plan_t* p, harts_kda_sizes* out) {
  if (!p || !out) {
    set_error("harts_kda_layout: NULL argument");
    return HARTS_EINVAL;
  }
  if (p->chunk != kKdaChunk) {
    set_error("harts_kda_layout: the KDA kernels need a plan with chunk 64");
    return HARTS_EUNSUPPORTED;
  }
  int64_t nc = 0;
  int32_t groups = 0;
  for (int32_t r = 0; r < p->K; ++r) {
    std::vector<int32_t> seen;
    for (int32_t i = p->round_seq_off[r]; i < p->round_seq_off[r + 1]; ++i) {
      nc += (p->seq_n_replay[i] + p->seq_n_own[i] + kKdaChunk - 1) / kKdaChunk;
      if (std::find(seen.begin(), seen.end(), p->seq_init_bank[i]) == seen.end()) {
        seen.push_back(p->seq_init_bank[i]);
        ++groups;
      }
    }
  }
  if (nc * kKdaChunk >= INT32_MAX) {
    set_error("harts_kda_layout: more than 2^31 - 1 packed rows");
    return HARTS_EUNSUPPORTED;
  }
  // compact rows with replay copies hold several packed rows: one slot each
  int64_t n_multi = 0, n_slots = 0;
  try {
    std::vector<int32_t> copies(static_cast<size_t>(p->C), 0);
    for (int64_t j = 0; j < p->R; ++j) ++copies[p->replay_row[j]];
    for (int64_t r = 0; r < p->C; ++r)
      if (copies[r] > 0) {
        ++n_multi;
        n_slots += 1 + copies[r];
      }
  } catch (const std::bad_alloc&) {
    set_error("harts_kda_layout: out of host memory");
    return HARTS_ENOMEM;
  }
  out->n_chunks = nc;
  out->n_slots = n_slots;
  out->n_seq = p->n_seq;
  out->n_rounds = p->K;
  out->n_groups = groups;
  out->n_req = static_cast<int32_t>(p->req_chunk.size());
  out->n_multi = static_cast<int32_t>(n_multi);
  return HARTS_OK;
}

extern "C" int harts_kda_tables(const harts_plan_t* p, int32_t* chunk_rows, int32_t* seq_tab, int32_t* req_tab,
                                int32_t* group_tab, int32_t* group_seq, int32_t* pos_slot, int32_t* multi_row,
                                int64_t* multi_off) {
  harts_kda_sizes sz;
  if (int rc = harts_kda_layout(p, &sz)) return rc;
  if (!chunk_rows || !seq_tab || (sz.n_req > 0 && !req_tab) || !group_tab || !group_seq || !pos_slot ||
      (sz.n_multi > 0 && !multi_row) || !multi_off) {
    set_error("harts_kda_tables: NULL argument");
    return HARTS_EINVAL;
  }
  try {
    int64_t c0 = 0;
    int32_t ng = 0, gm = 0;
    for (int32_t r = 0; r < p->K; ++r) {
      // sequences of the round grouped by initial bank entry (first appearance order)
      std::vector<int32_t> banks;
      for (int32_t i = p->round_seq_off[r]; i < p->round_seq_off[r + 1]; ++i)
        if (std::find(banks.begin(), banks.end(), p->seq_init_bank[i]) == banks.end())
          banks.push_back(p->seq_init_bank[i]);
      for (int32_t b : banks) {
        group_tab[4 * ng + 0] = r;
        group_tab[4 * ng + 1] = b;
        group_tab[4 * ng + 2] = gm;
        int32_t n = 0;
        for (int32_t i = p->round_seq_off[r]; i < p->round_seq_off[r + 1]; ++i)
          if (p->seq_init_bank[i] == b) {
            group_seq[gm++] = i;
            ++n;
          }
        group_tab[4 * ng + 3] = n;
        ++ng;
      }
      for (int32_t i = p->round_seq_off[r]; i < p->round_seq_off[r + 1]; ++i) {
        const int64_t nrep = p->seq_n_replay[i], nown = p->seq_n_own[i];
        const int64_t nc = (nrep + nown + kKdaChunk - 1) / kKdaChunk;
        int32_t* s = seq_tab + 8 * i;
        s[0] = r;
        s[1] = static_cast<int32_t>(c0);
        s[2] = static_cast<int32_t>(nc);
        s[3] = p->seq_init_bank[i];
        s[4] = p->seq_req_off[i];
        s[5] = p->seq_req_off[i + 1] - p->seq_req_off[i];
        s[6] = p->seq_final_leaf[i];
        int32_t* rows = chunk_rows + c0 * kKdaChunk;
        int64_t k = 0;
        // packed row entry: physical row * 2 + 1 for an own row, * 2 for a replay row; -1 padding
        for (int64_t j = 0; j < nrep; ++j, ++k)
          rows[k] = static_cast<int32_t>(p->replay_row[p->seq_replay_off[i] + j] * 2);
        for (int64_t j = 0; j < nown; ++j, ++k) rows[k] = static_cast<int32_t>((p->seq_row[i] + j) * 2 + 1);
        for (; k < nc * kKdaChunk; ++k) rows[k] = -1;
        c0 += nc;
      }
      // the order in which the state pass takes the round's sequences:
      // longest first (ties by id), so that the long chains start in the
      // first wave of workgroups and the short ones fill in behind them
      std::vector<int32_t> order;
      for (int32_t i = p->round_seq_off[r]; i < p->round_seq_off[r + 1]; ++i) order.push_back(i);
      std::stable_sort(order.begin(), order.end(),
                       [&](int32_t a, int32_t b) { return seq_tab[8 * a + 2] > seq_tab[8 * b + 2]; });
      for (size_t j = 0; j < order.size(); ++j) seq_tab[8 * (p->round_seq_off[r] + j) + 7] = order[j];
    }
    for (size_t j = 0; j < p->req_chunk.size(); ++j) {
      req_tab[2 * j] = p->req_chunk[j];
      req_tab[2 * j + 1] = p->req_bank[j];
    }
    // packed positions of every compact row; the rows with several of them
    // (ascending row order) get consecutive slots in ascending position order
    const int64_t C = p->C, npk = sz.n_chunks * kKdaChunk;
    std::vector<int32_t> count(static_cast<size_t>(C), 0), first(static_cast<size_t>(C), -1);
    for (int64_t e = 0; e < npk; ++e)
      if (chunk_rows[e] >= 0) ++count[chunk_rows[e] / 2];
    int32_t m = 0;
    multi_off[0] = 0;
    for (int64_t r = 0; r < C; ++r)
      if (count[r] > 1) {
        multi_row[m] = static_cast<int32_t>(r);
        first[r] = static_cast<int32_t>(multi_off[m]);
        multi_off[m + 1] = multi_off[m] + count[r];
        ++m;
      }
    for (int64_t e = 0; e < npk; ++e) {
      const int32_t r = chunk_rows[e] >= 0 ? chunk_rows[e] / 2 : -1;
      pos_slot[e] = r >= 0 && first[r] >= 0 ? first[r]++ : -1;
    }
  } catch (const std::bad_alloc&) {
    set_error("harts_kda_tables: out of host memory");
    return HARTS_ENOMEM;
  }
  set_error("");
  return HARTS_OK;
}
