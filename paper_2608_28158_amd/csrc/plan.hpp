// Internal definition of the plan object and of the device descriptor image.
// Shared by the host planner (plan.cpp) and the device-call layer (la.hip).
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "harts.h"

namespace harts {

// Fields of one sequence entry in a round's sequence table (int32 words).
enum SeqField : int {
  SEQ_CHUNK_OFF = 0,  // first chunk of the sequence within the round
  SEQ_N_TOK = 1,      // replay + own rows
  SEQ_N_REPLAY = 2,   // replay rows (< chunk)
  SEQ_REPLAY_OFF = 3, // global replay index of the first replay row
  SEQ_OWN_ROW = 4,    // physical row of the first own row
  SEQ_INIT_BANK = 5,  // bank entry of the initial state
  SEQ_FINAL_LEAF = 6, // leaf index receiving the final state
  SEQ_REQ_OFF = 7,    // first request (global index)
  SEQ_N_REQ = 8,      // requests of the sequence
  SEQ_N_CHUNKS = 9,   // chunks of the sequence
  SEQ_BLK_OFF = 10,   // first block of the sequence within the round
  SEQ_N_BLK = 11,     // blocks of the sequence
  SEQ_WORDS = 16
};

// Fields of one block entry (a run of consecutive chunks of one sequence;
// blocks end at every requested boundary and at most every `block_chunks`
// chunks).
enum BlkField : int {
  BLK_SEQ = 0,      // sequence (local index within the round)
  BLK_C0 = 1,       // first chunk (within the sequence)
  BLK_NC = 2,       // chunks in the block
  BLK_IDX = 3,      // block index within the sequence
  BLK_END_BANK = 4, // bank entry requested at the block's end, or -1
  BLK_WORDS = 8
};

// Fields of one entry of a round's launch table: the blocks in the order the
// block kernels take them (longest first), each entry holding every block
// and sequence field those kernels read, so that a workgroup finds its work
// with one load instead of a chain of dependent ones.
enum LaunchField : int {
  LCH_BLK = 0,         // block id (index into the block table)
  LCH_SEQ = 1,         // sequence (local index within the round)
  LCH_C0 = 2,          // first chunk of the block (within the sequence)
  LCH_NC = 3,          // chunks in the block
  LCH_IDX = 4,         // block index within the sequence
  LCH_N_BLK = 5,       // blocks of the sequence
  LCH_FINAL_LEAF = 6,  // leaf index receiving the sequence's final state
  LCH_INIT_BANK = 7,   // bank entry of the sequence's initial state, or -1
  LCH_N_TOK = 8,       // replay + own rows of the sequence
  LCH_N_REPLAY = 9,    // replay rows of the sequence
  LCH_REPLAY_OFF = 10, // global replay index of its first replay row
  LCH_OWN_ROW = 11,    // physical row of its first own row
  LCH_CHUNK_OFF = 12,  // its first chunk within the round
  LCH_WORDS = 16
};

struct RoundLayout {
  int32_t n_seq = 0, seq_begin = 0, max_seq_chunks = 0;
  int32_t n_blk = 0, block_chunks = 0, max_seq_blocks = 0;
  int64_t blk_tab = 0;    // int32 offset of the [n_blk][BLK_WORDS] block table
  int64_t blk_launch = 0; // int32 offset of the [n_blk][LCH_WORDS] launch table
  int64_t n_chunks = 0, n_rows = 0, n_own = 0, n_replay = 0, own_row_begin = 0;
  int64_t seq_tab = 0;    // int32 offset of the sequence table
  int64_t init_idx = 0;   // int32 offset of the [n_seq] init bank indices
  int64_t chunk_tab = 0;  // int32 offset of the [n_chunks][2] chunk table
};

}  // namespace harts

struct harts_plan_s {
  int32_t n_seg = 0, n_trees = 0, n_leaves = 0, K = 0, n_seq = 0, n_slots = 0;
  int32_t n_bank = 0, chunk = 0;
  int32_t min_blocks = 0;  // block target of the device tables (harts_plan_set_blocks)
  int64_t C = 0, S = 0, R = 0, n_chunks = 0;

  std::vector<int32_t> parent;  // the forest as given (-1 marks a root)
  std::vector<int64_t> seg_start, seg_end, seg_row, seg_mult;
  std::vector<int32_t> seg_seq, seg_tpre, seg_tin, seg_tree, leaf_seg;
  std::vector<int32_t> tree_calls, round_seq_off;
  std::vector<int32_t> seq_round, seq_tree, seq_first_seg, seq_final_leaf;
  std::vector<int32_t> seq_init_bank, seq_chain_off, chain_seg, seq_req_off;
  std::vector<int64_t> seq_anchor, seq_n_replay, seq_replay_off, seq_row;
  std::vector<int64_t> seq_n_own;
  std::vector<int32_t> req_chunk, req_bank, slot_seq;
  std::vector<int64_t> slot_pos, replay_row;

  // device descriptor image (int32 words) and its layout
  std::vector<int32_t> blob;
  std::vector<harts::RoundLayout> rounds;
  int64_t off_replay_row = 0, off_req_chunk = 0, off_req_bank = 0;
  int64_t off_red_rows = 0, off_red_off = 0, off_red_idx = 0, n_red = 0;
};

namespace harts {
void set_error(const std::string& msg);
}
