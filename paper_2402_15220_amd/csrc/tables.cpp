// Kernel context flattening (ChunkAttention Section 3.3, Figure 2).
#include "tables.hpp"

#include <algorithm>
#include <utility>

namespace ca {

void fill_item_records(WorkLists* w) {
  WorkLists& W = *w;
  for (SfItem& it : W.items) {
    it.part_b = W.part_ptr[it.row];
    it.part_e = W.part_ptr[it.row + 1];
    it.n_inline = std::min(it.ce - it.cb, kSfInline);
    it.pad = 0;
    for (int i = 0; i < kSfInline; ++i) it.slot[i] = i < it.n_inline ? W.priv_slot[it.cb + i] : 0;
  }
}

void build_tables(const ChunkTree& tree, Tables* out) {
  Tables& T = *out;
  const auto& nodes = tree.nodes();

  // Rows and covered ranges: iterative depth-first pre-order. Children are
  // stored sorted by first token, terminals sorted by id.
  T.row_seq.clear();
  std::vector<int32_t> rb(nodes.size(), 0), re(nodes.size(), 0);
  {
    std::vector<std::pair<int32_t, bool>> stack;
    stack.emplace_back(ChunkTree::kRoot, false);
    while (!stack.empty()) {
      auto [id, done] = stack.back();
      stack.pop_back();
      if (done) {
        re[id] = static_cast<int32_t>(T.row_seq.size());
        continue;
      }
      rb[id] = static_cast<int32_t>(T.row_seq.size());
      for (int64_t sid : nodes[id].terminals) T.row_seq.push_back(sid);
      stack.emplace_back(id, true);
      const auto& ch = nodes[id].children;
      for (auto it = ch.rbegin(); it != ch.rend(); ++it) stack.emplace_back(it->second, false);
    }
  }

  // Node order: breadth-first levels.
  T.node_id.clear();
  for (const auto& ch : nodes[ChunkTree::kRoot].children) T.node_id.push_back(ch.second);
  for (size_t i = 0; i < T.node_id.size(); ++i)
    for (const auto& ch : nodes[T.node_id[i]].children) T.node_id.push_back(ch.second);
  const size_t nn = T.node_id.size();
  std::vector<int32_t> index(nodes.size(), -1);
  for (size_t i = 0; i < nn; ++i) index[T.node_id[i]] = static_cast<int32_t>(i);

  T.node_slot.resize(nn);
  T.node_len.resize(nn);
  T.node_row_begin.resize(nn);
  T.node_row_end.resize(nn);
  T.node_parent.resize(nn);
  T.node_start_pos.resize(nn);
  for (size_t i = 0; i < nn; ++i) {
    const Node& N = nodes[T.node_id[i]];
    T.node_slot[i] = N.slot;
    T.node_len[i] = static_cast<int32_t>(N.tokens.size());
    T.node_row_begin[i] = rb[T.node_id[i]];
    T.node_row_end[i] = re[T.node_id[i]];
    if (N.parent == ChunkTree::kRoot) {
      T.node_parent[i] = -1;
      T.node_start_pos[i] = 0;
    } else {
      const int32_t p = index[N.parent];  // parents precede children in BFS order
      T.node_parent[i] = p;
      T.node_start_pos[i] = T.node_start_pos[p] + T.node_len[p];
    }
  }

  T.shr_node.clear();
  T.shr_part_base.clear();
  std::vector<int32_t> part_base(nn, -1);
  int32_t acc = 0;
  for (size_t i = 0; i < nn; ++i) {
    const int32_t cnt = T.node_row_end[i] - T.node_row_begin[i];
    if (cnt >= 2) {
      T.shr_node.push_back(static_cast<int32_t>(i));
      T.shr_part_base.push_back(acc);
      part_base[i] = acc;
      acc += cnt;
    }
  }

  const int64_t B = static_cast<int64_t>(T.row_seq.size());
  T.priv_ptr.assign(1, 0);
  T.shr_ptr.assign(1, 0);
  T.priv_node.clear();
  T.shr_part.clear();
  T.path_ptr.assign(1, 0);
  T.path_node.clear();
  std::vector<int32_t> path;
  const auto& seqs = tree.seqs();
  for (int64_t r = 0; r < B; ++r) {
    path.clear();
    for (int32_t x = seqs.at(T.row_seq[r]).term; x != ChunkTree::kRoot; x = nodes[x].parent)
      path.push_back(index[x]);
    for (auto it = path.rbegin(); it != path.rend(); ++it) {
      const int32_t i = *it;
      T.path_node.push_back(i);
      if (part_base[i] >= 0)
        T.shr_part.push_back(part_base[i] + static_cast<int32_t>(r) - T.node_row_begin[i]);
      else
        T.priv_node.push_back(i);
    }
    T.priv_ptr.push_back(static_cast<int32_t>(T.priv_node.size()));
    T.shr_ptr.push_back(static_cast<int32_t>(T.shr_part.size()));
    T.path_ptr.push_back(static_cast<int32_t>(T.path_node.size()));
  }
}

void build_work(const ChunkTree& tree, const Tables& T, int32_t seg_chunks, int32_t split_chunks,
                bool partial_items, int32_t num_heads, int32_t num_cus, WorkLists* out,
                bool serial_reduce, int32_t token_head_bytes) {
  WorkLists& W = *out;
  if (serial_reduce) {
    // every segment is one more launch: by default a run is one segment
    // unless longer than 64 chunks
    if (seg_chunks <= 0) seg_chunks = 64;
    split_chunks = 0;
    partial_items = false;
  }
  const int64_t B = static_cast<int64_t>(T.row_seq.size());
  const size_t nn = T.node_slot.size();

  // Runs: a shared node continues its parent's run when the parent is shared
  // and covers the same rows (BFS order visits parents first).
  std::vector<int32_t> run_of(nn, -1);
  std::vector<std::vector<int32_t>> runs;  // node indices root -> leaf
  for (int32_t i : T.shr_node) {
    const int32_t p = T.node_parent[i];
    if (p >= 0 && run_of[p] >= 0 && T.node_row_begin[p] == T.node_row_begin[i] &&
        T.node_row_end[p] == T.node_row_end[i]) {
      run_of[i] = run_of[p];
    } else {
      run_of[i] = static_cast<int32_t>(runs.size());
      runs.emplace_back();
    }
    runs[run_of[i]].push_back(i);
  }

  // Automatic segment size: about one chunk-first block per compute unit,
  // counting a run of L chunks over r rows as L * ceil(r/16) * H chunk-blocks
  // (16 rows per block in the fused launch). A segment is a chain of
  // dependent chunk steps, so segments stay at 16 chunks or fewer unless the
  // sequence-first stream (the private K/V at ~6 TB/s) is long enough to hide
  // a longer chain at ~3 us per chunk under load; longer segments mean fewer
  // partials per row. When the sequence-first blocks take more than one
  // round of the chip's resident slots (four blocks per compute unit) and
  // stream at least 4 chunks each, a chain is also at most twice as long as
  // the longest row's private chunk list: longer chains outlast the
  // sequence-first blocks and finish the rows late (measured on a tree of
  // 64 rows with 4 private chunks each: 57.0 us with 8-chunk segments
  // against 60.6 us for 16). Otherwise the chains are the critical path
  // whatever their length and fewer partials win (32 rows decoding from a
  // 4096-token prompt with 1 to 200 private tokens: 16-chunk segments 23-32
  // us, 2-8-chunk segments 26-43 us; 96 rows over a 2048-token prompt with
  // one private chunk: 40 us against 55 us with 2-chunk segments).
  if (seg_chunks <= 0) {
    int64_t work = 0;
    for (const auto& chain : runs) {
      const int64_t r = T.node_row_end[chain[0]] - T.node_row_begin[chain[0]];
      work += static_cast<int64_t>(chain.size()) * ((r + 15) / 16) * num_heads;
    }
    int64_t priv_tokens = 0;
    for (int32_t k : T.priv_node) priv_tokens += T.node_len[k];
    int64_t max_priv = 0;
    for (int64_t r = 0; r < B; ++r)
      max_priv = std::max<int64_t>(max_priv, T.priv_ptr[r + 1] - T.priv_ptr[r]);
    const double ksf_us = static_cast<double>(priv_tokens) * num_heads * token_head_bytes / 6.0e6;
    int64_t cap = std::min<int64_t>(64, std::max<int64_t>(16, static_cast<int64_t>(ksf_us / 3.0)));
    const int64_t cus = num_cus > 0 ? num_cus : 256;
    if (max_priv >= 4 && B * num_heads > 4 * cus) cap = std::min<int64_t>(cap, 2 * max_priv);
    // rounded up to a power of two: runs of 2^k chunks (the usual prompt
    // lengths) then split evenly into fewer segments, and fewer partials
    // won in 8 of 9 measured trees whose quota was not a power of two (e.g.
    // 48 rows over a 2048-token prompt: 12-chunk segments 25.7 us, 16-chunk
    // 22.9 us; the exception, 32 rows with 1536 shared tokens: 46.1 against
    // 47.0 us)
    int64_t quota = std::max<int64_t>(1, (work + cus - 1) / cus), pow2 = 1;
    while (pow2 < quota) pow2 <<= 1;
    seg_chunks = static_cast<int32_t>(std::min<int64_t>(cap, pow2));
  }
  if (seg_chunks > 64) seg_chunks = 64;  // the chunk-first kernel keeps a segment's slots in lanes
  W.seg_chunks = seg_chunks;

  W.segs.clear();
  W.seg_slots.clear();
  W.max_seg_rows = 0;
  std::vector<std::pair<int32_t, int32_t>> run_segs(runs.size());  // [first seg, n segs)
  int32_t part = 0;
  for (size_t ru = 0; ru < runs.size(); ++ru) {
    const auto& chain = runs[ru];
    const int32_t rb = T.node_row_begin[chain[0]], re = T.node_row_end[chain[0]];
    run_segs[ru].first = static_cast<int32_t>(W.segs.size());
    for (size_t s = 0; s < chain.size(); s += seg_chunks) {
      CfSeg sg{};
      sg.slot_off = static_cast<int32_t>(W.seg_slots.size());
      const size_t e = std::min(chain.size(), s + static_cast<size_t>(seg_chunks));
      for (size_t k = s; k < e; ++k) W.seg_slots.push_back(T.node_slot[chain[k]]);
      sg.n_chunks = static_cast<int32_t>(e - s);
      sg.row_begin = rb;
      sg.row_end = re;
      sg.part_base = part;
      part += re - rb;
      W.max_seg_rows = std::max(W.max_seg_rows, re - rb);
      W.segs.push_back(sg);
    }
    run_segs[ru].second = static_cast<int32_t>(W.segs.size()) - run_segs[ru].first;
  }

  // Sequence-first items and per-row partial lists.
  W.items.clear();
  W.priv_slot.clear();
  W.part_ptr.assign(1, 0);
  W.parts.clear();
  W.mg_rows.clear();
  (void)tree;
  for (int64_t r = 0; r < B; ++r) {
    // segment partials, root -> leaf: each run met along the path once
    int32_t last_run = -1;
    for (int32_t k = T.path_ptr[r]; k < T.path_ptr[r + 1]; ++k) {
      const int32_t ru = run_of[T.path_node[k]];
      if (ru < 0 || ru == last_run) continue;
      last_run = ru;
      for (int32_t s = run_segs[ru].first; s < run_segs[ru].first + run_segs[ru].second; ++s)
        W.parts.push_back(W.segs[s].part_base + static_cast<int32_t>(r) - W.segs[s].row_begin);
    }
    const int32_t pb = static_cast<int32_t>(W.priv_slot.size());
    for (int32_t k = T.priv_ptr[r]; k < T.priv_ptr[r + 1]; ++k)
      W.priv_slot.push_back(T.node_slot[T.priv_node[k]]);
    const int32_t pe = static_cast<int32_t>(W.priv_slot.size());
    const int32_t np = pe - pb;
    const bool has_shared = static_cast<int32_t>(W.parts.size()) > W.part_ptr.back();
    if (!(partial_items && has_shared) && (split_chunks <= 0 || np <= split_chunks)) {
      // the row's own item produces its output directly
      W.items.push_back(SfItem{static_cast<int32_t>(r), pb, pe, -1, 0, 0, 0, 0, {}});
    } else {
      // chunk-first partials and/or several private pieces: every piece
      // writes a partial and the merge epilogue produces the output
      const int32_t piece = split_chunks > 0 ? split_chunks : std::max(np, 1);
      for (int32_t c0 = pb; c0 < pe; c0 += piece) {
        const int32_t c1 = std::min(pe, c0 + piece);
        W.items.push_back(SfItem{static_cast<int32_t>(r), c0, c1, part, 0, 0, 0, 0, {}});
        W.parts.push_back(part);
        ++part;
      }
      W.mg_rows.push_back(static_cast<int32_t>(r));
    }
    W.part_ptr.push_back(static_cast<int32_t>(W.parts.size()));
  }
  // longest items first: they are dispatched first and finish with the rest
  std::stable_sort(W.items.begin(), W.items.end(), [](const SfItem& a, const SfItem& b) {
    return a.ce - a.cb > b.ce - b.cb;
  });
  W.n_parts = part;
  W.seg_group_ptr.clear();
  if (serial_reduce) {
    // contributor position of each segment on its rows' paths: runs root ->
    // leaf, segments in order (the same for every row a segment covers)
    std::vector<int32_t> seg_k(W.segs.size(), -1);
    for (int64_t r = 0; r < B; ++r) {
      int32_t k = 0, last_run = -1;
      for (int32_t e = T.path_ptr[r]; e < T.path_ptr[r + 1]; ++e) {
        const int32_t ru = run_of[T.path_node[e]];
        if (ru < 0 || ru == last_run) continue;
        last_run = ru;
        for (int32_t sgi = run_segs[ru].first; sgi < run_segs[ru].first + run_segs[ru].second; ++sgi)
          seg_k[sgi] = k++;
      }
    }
    // accumulator per row: partial index = row; rows with shared chunks fold it
    W.parts.clear();
    W.part_ptr.assign(1, 0);
    for (int64_t r = 0; r < B; ++r) {
      if (T.shr_ptr[r + 1] > T.shr_ptr[r]) W.parts.push_back(static_cast<int32_t>(r));
      W.part_ptr.push_back(static_cast<int32_t>(W.parts.size()));
    }
    std::vector<int32_t> order(W.segs.size());
    for (size_t i = 0; i < order.size(); ++i) order[i] = static_cast<int32_t>(i);
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return seg_k[a] < seg_k[b]; });
    std::vector<CfSeg> sorted;
    for (int32_t i : order) {
      CfSeg sg = W.segs[i];
      sg.part_base = sg.row_begin;
      sg.pad0 = seg_k[i] > 0 ? 1 : 0;
      sorted.push_back(sg);
      while (static_cast<int32_t>(W.seg_group_ptr.size()) <= seg_k[i])
        W.seg_group_ptr.push_back(static_cast<int32_t>(sorted.size()) - 1);
    }
    W.seg_group_ptr.push_back(static_cast<int32_t>(sorted.size()));
    W.segs.swap(sorted);
    W.n_parts = B;
  }
  // fixed-stride slot lists: segment i's at i * kSegSlotStride
  {
    std::vector<int32_t> packed(W.segs.size() * kSegSlotStride);
    for (size_t i = 0; i < W.segs.size(); ++i) {
      CfSeg& sg = W.segs[i];
      for (int k = 0; k < kSegSlotStride; ++k)
        packed[i * kSegSlotStride + k] = W.seg_slots[sg.slot_off + std::min(k, sg.n_chunks - 1)];
      sg.slot_off = static_cast<int32_t>(i * kSegSlotStride);
    }
    W.seg_slots.swap(packed);
  }
  fill_item_records(&W);
  W.row_of_seq.clear();
  for (int64_t r = 0; r < B; ++r) W.row_of_seq[T.row_seq[r]] = static_cast<int32_t>(r);
  W.item_of_row.assign(B, -1);
  std::vector<int32_t> pieces(B, 0);
  for (size_t i = 0; i < W.items.size(); ++i) {
    const int32_t r = W.items[i].row;
    if (pieces[r]++ == 0) W.item_of_row[r] = static_cast<int32_t>(i);
    else W.item_of_row[r] = -1;
  }
}

bool patch_work(const ChunkTree& tree, WorkLists* w) {
  WorkLists& W = *w;
  const auto& grown = tree.grown();
  for (const auto& g : grown) {  // check first: all or nothing
    auto it = W.row_of_seq.find(g.first);
    if (it == W.row_of_seq.end() || W.item_of_row[it->second] < 0) return false;
  }
  for (const auto& g : grown) {
    const int32_t r = W.row_of_seq.at(g.first);
    const int32_t self = W.item_of_row[r];
    const int32_t at = W.items[self].ce;  // end of the row's private list
    W.priv_slot.insert(W.priv_slot.begin() + at, tree.node(g.second).slot);
    for (auto& it : W.items)
      if (it.cb >= at && &it != &W.items[self]) {
        ++it.cb;
        ++it.ce;
      }
    ++W.items[self].ce;
  }
  // keep longest-first; rows keep their items
  std::vector<int32_t> order(W.items.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = static_cast<int32_t>(i);
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    return W.items[a].ce - W.items[a].cb > W.items[b].ce - W.items[b].cb;
  });
  std::vector<SfItem> sorted(W.items.size());
  for (size_t i = 0; i < order.size(); ++i) sorted[i] = W.items[order[i]];
  W.items.swap(sorted);
  for (size_t i = 0; i < W.items.size(); ++i) W.item_of_row[W.items[i].row] = static_cast<int32_t>(i);
  fill_item_records(&W);
  return true;
}

const char* same_work(const WorkLists& a, const WorkLists& b) {
  if (a.seg_slots != b.seg_slots || a.segs.size() != b.segs.size()) return "segments";
  for (size_t i = 0; i < a.segs.size(); ++i)
    if (a.segs[i].slot_off != b.segs[i].slot_off || a.segs[i].n_chunks != b.segs[i].n_chunks ||
        a.segs[i].row_begin != b.segs[i].row_begin || a.segs[i].row_end != b.segs[i].row_end ||
        a.segs[i].part_base != b.segs[i].part_base)
      return "segments";
  if (a.part_ptr != b.part_ptr || a.parts != b.parts || a.mg_rows != b.mg_rows ||
      a.n_parts != b.n_parts)
    return "partial lists";
  if (a.items.size() != b.items.size()) return "item count";
  auto key = [](const WorkLists& w) {
    std::vector<std::vector<int32_t>> k(w.item_of_row.size());
    for (const auto& it : w.items) {
      auto& v = k[it.row];
      v.push_back(it.out_part);
      v.insert(v.end(), w.priv_slot.begin() + it.cb, w.priv_slot.begin() + it.ce);
    }
    return k;
  };
  if (key(a) != key(b)) return "sequence-first items";
  for (const WorkLists* w : {&a, &b})
    for (const auto& it : w->items) {
      if (it.part_b != w->part_ptr[it.row] || it.part_e != w->part_ptr[it.row + 1] ||
          it.n_inline != std::min(it.ce - it.cb, kSfInline))
        return "item records";
      for (int i = 0; i < it.n_inline; ++i)
        if (it.slot[i] != w->priv_slot[it.cb + i]) return "item records";
    }
  return "";
}

}  // namespace ca
