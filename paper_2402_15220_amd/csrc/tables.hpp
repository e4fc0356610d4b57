// Kernel context generated from the tree (ChunkAttention Section 3.3 and
// Figure 2): canonical tables plus the work lists the kernels consume.
#pragma once

#include <cstdint>
#include <unordered_map>
#include <vector>

#include "tree.hpp"
#include "worklist.hpp"

namespace ca {

// Canonical tables (the paper's (C, i, j) context with half-open ranges, plus
// Algorithm 2's per-sequence lists). Node index = breadth-first level order
// with children by ascending first token; rows follow a depth-first
// pre-order in which sequences ending at a node come first (ascending id).
struct Tables {
  std::vector<int64_t> row_seq;
  std::vector<int32_t> node_slot, node_len, node_row_begin, node_row_end, node_parent,
      node_start_pos;
  std::vector<int32_t> shr_node, shr_part_base;
  std::vector<int32_t> priv_ptr, priv_node, shr_ptr, shr_part;
  std::vector<int32_t> node_id;  // BFS index -> tree node id (internal)
  std::vector<int32_t> path_ptr, path_node;  // per row, all path nodes root -> leaf (internal)
};

void build_tables(const ChunkTree& tree, Tables* out);

// Kernel work lists derived from the tables.
//  * Shared nodes are grouped into runs: maximal parent->child chains of
//    shared nodes covering the same rows. Each run is cut into segments of at
//    most seg_chunks chunks; the chunk-first kernel handles one (segment,
//    head, row block) per workgroup and writes one partial per covered row.
//  * Each row's private chunks form one sequence-first item, or several of
//    at most split_chunks chunks (split_chunks <= 0 disables splitting).
//    An unsplit row is finished by its item (o written directly), which in
//    the sequential schedule also folds the row's chunk-first partials. With
//    partial_items (schedules where the chunk-first items run at the same
//    time), a row with shared chunks has its item write a partial and the
//    row's last contributor finishes it; split rows always write partials.
//    mg_rows lists the rows finished from partials.
//  * seg_chunks <= 0 picks the size automatically (about one chunk-first
//    block per compute unit, at most 16 chunks); explicit sizes are clamped
//    to 64.
//  * part lists per row: the row's segment partials root -> leaf, then its
//    sequence-first partials in chunk order.
struct WorkLists {
  std::vector<CfSeg> segs;
  std::vector<int32_t> seg_slots;
  std::vector<SfItem> items;
  std::vector<int32_t> priv_slot;  // per row private slots (indexed by items)
  std::vector<int32_t> part_ptr;   // [B+1]
  std::vector<int32_t> parts;
  std::vector<int32_t> mg_rows;    // rows whose result the merge kernel writes
  int64_t n_parts = 0;
  int32_t max_seg_rows = 0;
  int32_t seg_chunks = 0;  // segment size used
  // for in-place updates: row of each live sequence, and the index in
  // `items` of each row's single item (-1: none or several pieces)
  std::unordered_map<int64_t, int32_t> row_of_seq;
  std::vector<int32_t> item_of_row;
  // serial_reduce only: segments [seg_group_ptr[g], seg_group_ptr[g+1]) are
  // the g-th contributors of their rows and run in the g-th launch
  std::vector<int32_t> seg_group_ptr;
};

// serial_reduce: the partial-free variant (Section 3.3, further
// optimizations): each row has one accumulator (partial index = row) that the
// chunk-first segments fold into in path order, one launch per position in
// that order (seg_group_ptr), so no row has two writers at once; segments
// take up to 64 chunks (seg_chunks <= 0) and pad0 = 1 marks the ones that
// fold (not the first on their rows' paths).
// token_head_bytes: K+V bytes of one token of one head (2·d·element size),
// used by the automatic segment size to estimate the sequence-first stream.
// The derived fields of every item record (partial range, inline slots).
void fill_item_records(WorkLists* w);

void build_work(const ChunkTree& tree, const Tables& t, int32_t seg_chunks, int32_t split_chunks,
                bool partial_items, int32_t num_heads, int32_t num_cus, WorkLists* out,
                bool serial_reduce = false, int32_t token_head_bytes = 512);

// Bring work lists built for an earlier tree up to date when the only
// structural changes since were new private chunks at the end of sequences'
// paths (tree.grown()): row order, shared runs, segments and partials are
// unchanged, and each new chunk's slot is appended to its row's private list
// (the rows after it shift by one). Returns false, changing nothing, when a
// row cannot be patched this way (no single item for the row).
bool patch_work(const ChunkTree& tree, WorkLists* w);

// Compare two work lists up to the order of sequence-first items: every row
// has the same private slots and item kind, segments and partial lists are
// equal. Empty string when they agree, else what differs.
const char* same_work(const WorkLists& a, const WorkLists& b);

}  // namespace ca
