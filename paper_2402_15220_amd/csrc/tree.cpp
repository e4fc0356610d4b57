// Host prefix tree of chunks (ChunkAttention Section 3.1); see tree.hpp.
#include "tree.hpp"

#include <algorithm>
#include <unordered_set>

namespace ca {

ChunkTree::ChunkTree(int32_t chunk_size, int64_t num_slots) : c_(chunk_size), pool_(num_slots) {
  nodes_.emplace_back();  // virtual root: no tokens, no slot
  nodes_[kRoot].live = true;
}

int32_t ChunkTree::new_node() {
  int32_t id;
  if (!free_nodes_.empty()) {
    id = free_nodes_.back();
    free_nodes_.pop_back();
    nodes_[id] = Node();
  } else {
    id = static_cast<int32_t>(nodes_.size());
    nodes_.emplace_back();
  }
  nodes_[id].live = true;
  return id;
}

void ChunkTree::free_node(int32_t id) {
  nodes_[id] = Node();
  free_nodes_.push_back(id);
}

int32_t ChunkTree::find_child(int32_t node, int32_t tok) const {
  const auto& ch = nodes_[node].children;
  auto it = std::lower_bound(ch.begin(), ch.end(), std::make_pair(tok, INT32_MIN));
  if (it != ch.end() && it->first == tok) return it->second;
  return -1;
}

void ChunkTree::add_child(int32_t parent, int32_t child) {
  auto& ch = nodes_[parent].children;
  std::pair<int32_t, int32_t> e(nodes_[child].tokens[0], child);
  ch.insert(std::lower_bound(ch.begin(), ch.end(), e), e);
}

void ChunkTree::remove_child(int32_t parent, int32_t child) {
  auto& ch = nodes_[parent].children;
  for (auto it = ch.begin(); it != ch.end(); ++it)
    if (it->second == child) {
      ch.erase(it);
      return;
    }
}

ChunkTree::Descent ChunkTree::descend(int32_t cur, const int32_t* t, int64_t n,
                                      int64_t pos) const {
  while (pos < n) {
    int32_t ch = find_child(cur, t[pos]);
    if (ch < 0) return {cur, pos, -1, 0};
    const auto& tok = nodes_[ch].tokens;
    const int64_t L = static_cast<int64_t>(tok.size());
    const int64_t m = std::min<int64_t>(L, n - pos);
    int64_t p = 0;
    while (p < m && tok[p] == t[pos + p]) ++p;
    if (p == L) {
      cur = ch;
      pos += L;
      continue;
    }
    return {cur, pos + p, ch, static_cast<int32_t>(p)};
  }
  return {cur, pos, -1, 0};
}

int64_t ChunkTree::match(const int32_t* tokens, int64_t n) const {
  return descend(kRoot, tokens, n, 0).pos;
}

// X keeps tokens[:p] and its slot; X' takes the tail, a fresh slot with the
// tail rows copied, X's children, count and terminal sequences.
int32_t ChunkTree::split(int32_t x, int32_t p, std::vector<KvJob>* jobs) {
  const int32_t slot = pool_.alloc();
  const int32_t xp = new_node();  // may reallocate nodes_: index afterwards
  Node& X = nodes_[x];
  Node& XP = nodes_[xp];
  const int32_t L = static_cast<int32_t>(X.tokens.size());
  XP.tokens.assign(X.tokens.begin() + p, X.tokens.end());
  XP.slot = slot;
  XP.count = X.count;
  XP.parent = x;
  XP.children = std::move(X.children);
  XP.terminals = std::move(X.terminals);
  for (auto& ch : XP.children) nodes_[ch.second].parent = xp;
  for (int64_t sid : XP.terminals) seqs_[sid].term = xp;
  X.tokens.resize(p);
  X.children.assign(1, {XP.tokens[0], xp});
  X.terminals.clear();
  if (jobs) {
    jobs->push_back({1, X.slot, p, slot, 0, L - p});
    jobs->push_back({2, 0, 0, X.slot, p, 0});
  }
  mark_structural();
  return x;
}

int32_t ChunkTree::new_chain(int32_t cur, const int32_t* t, int64_t n, int64_t pos,
                             int32_t row_base, std::vector<KvJob>* jobs) {
  while (pos < n) {
    const int64_t e = std::min<int64_t>(pos + c_, n);
    const int32_t slot = pool_.alloc();
    const int32_t nd = new_node();
    Node& N = nodes_[nd];
    N.tokens.assign(t + pos, t + e);
    N.slot = slot;
    N.parent = cur;
    add_child(cur, nd);
    if (jobs)
      jobs->push_back({0, row_base + static_cast<int32_t>(pos), 0, slot, 0,
                       static_cast<int32_t>(e - pos)});
    cur = nd;
    pos = e;
    dirty_ = true;
  }
  return cur;
}

Err ChunkTree::insert(int64_t sid, const int32_t* tokens, int64_t n, std::vector<KvJob>* jobs,
                      int64_t* matched) {
  if (n < 1) return Err::invalid;
  if (seqs_.count(sid)) return Err::exists;
  const Descent d = descend(kRoot, tokens, n, 0);
  const int64_t need = (d.split_node >= 0 ? 1 : 0) + chunks_for(n - d.pos, c_);
  if (need > pool_.available()) return Err::nomem;
  if (matched) *matched = d.pos;
  int32_t cur = d.cur;
  if (d.split_node >= 0) cur = split(d.split_node, d.split_at, jobs);
  const int32_t term = new_chain(cur, tokens, n, d.pos, 0, jobs);
  for (int32_t x = term; x != kRoot; x = nodes_[x].parent) nodes_[x].count++;
  auto& terms = nodes_[term].terminals;
  terms.insert(std::lower_bound(terms.begin(), terms.end(), sid), sid);
  seqs_[sid] = {term, n};
  mark_structural();
  return Err::ok;
}

Err ChunkTree::extend_impl(int64_t sid, const int32_t* tokens, int64_t n, int32_t row_base,
                           std::vector<KvJob>* jobs, int64_t* matched) {
  auto it = seqs_.find(sid);
  if (it == seqs_.end()) return Err::not_found;
  const int32_t t = it->second.term;
  int32_t end;
  int64_t m = 0;
  if (nodes_[t].count == 1) {
    // private last chunk: fill it, then grow new chunks below it
    const int64_t have = static_cast<int64_t>(nodes_[t].tokens.size());
    const int64_t f = std::min<int64_t>(c_ - have, n);
    if (chunks_for(n - f, c_) > pool_.available()) return Err::nomem;
    if (f > 0) {
      nodes_[t].tokens.insert(nodes_[t].tokens.end(), tokens, tokens + f);
      if (jobs)
        jobs->push_back({0, row_base, 0, nodes_[t].slot, static_cast<int32_t>(have),
                         static_cast<int32_t>(f)});
    }
    end = new_chain(t, tokens, n, f, row_base, jobs);
    if (end != t) {
      const size_t first = grown_.size();
      for (int32_t x = end; x != t; x = nodes_[x].parent) grown_.emplace_back(sid, x);
      std::reverse(grown_.begin() + static_cast<std::ptrdiff_t>(first), grown_.end());
    }
  } else {
    const Descent d = descend(t, tokens, n, 0);
    const int64_t need = (d.split_node >= 0 ? 1 : 0) + chunks_for(n - d.pos, c_);
    if (need > pool_.available()) return Err::nomem;
    m = d.pos;
    int32_t cur = d.cur;
    if (d.split_node >= 0) cur = split(d.split_node, d.split_at, jobs);
    end = new_chain(cur, tokens, n, d.pos, row_base, jobs);
    if (end != t) mark_structural();  // the sequence leaves a shared chunk
  }
  if (end != t) {
    auto& old = nodes_[t].terminals;
    old.erase(std::find(old.begin(), old.end(), sid));
    for (int32_t x = end; x != t; x = nodes_[x].parent) nodes_[x].count++;
    auto& terms = nodes_[end].terminals;
    terms.insert(std::lower_bound(terms.begin(), terms.end(), sid), sid);
    it = seqs_.find(sid);
    it->second.term = end;
    dirty_ = true;
  }
  it->second.length += n;
  if (matched) *matched = m;
  return Err::ok;
}

Err ChunkTree::extend(int64_t sid, const int32_t* tokens, int64_t n, int32_t row_base,
                      std::vector<KvJob>* jobs, int64_t* matched) {
  if (n < 1) return Err::invalid;
  return extend_impl(sid, tokens, n, row_base, jobs, matched);
}

Err ChunkTree::append_batch(int64_t n_seqs, const int64_t* sids, const int32_t* tokens,
                            std::vector<KvJob>* jobs) {
  if (n_seqs < 0) return Err::invalid;
  {
    std::unordered_set<int64_t> seen;
    for (int64_t i = 0; i < n_seqs; ++i) {
      if (!seen.insert(sids[i]).second) return Err::invalid;
      if (!seqs_.count(sids[i])) return Err::not_found;
    }
  }
  // Each single-token append needs at most one slot; when the pool might be
  // too small, rehearse the batch on a copy so the call is all or nothing.
  if (pool_.available() < n_seqs) {
    ChunkTree rehearsal(*this);
    for (int64_t i = 0; i < n_seqs; ++i) {
      Err e = rehearsal.extend_impl(sids[i], tokens + i, 1, 0, nullptr, nullptr);
      if (e != Err::ok) return e;
    }
  }
  for (int64_t i = 0; i < n_seqs; ++i) {
    Err e = extend_impl(sids[i], tokens + i, 1, static_cast<int32_t>(i), jobs, nullptr);
    if (e != Err::ok) return e;  // unreachable after the rehearsal
  }
  return Err::ok;
}

Err ChunkTree::remove(int64_t sid) {
  auto it = seqs_.find(sid);
  if (it == seqs_.end()) return Err::not_found;
  int32_t x = it->second.term;
  auto& terms = nodes_[x].terminals;
  terms.erase(std::find(terms.begin(), terms.end(), sid));
  seqs_.erase(it);
  while (x != kRoot) {
    const int32_t parent = nodes_[x].parent;
    if (--nodes_[x].count == 0) {
      remove_child(parent, x);
      pool_.release(nodes_[x].slot);
      free_node(x);
    }
    x = parent;
  }
  mark_structural();
  return Err::ok;
}

const char* ChunkTree::check() const {
  std::unordered_set<int32_t> slots;
  for (size_t id = 1; id < nodes_.size(); ++id) {
    const Node& N = nodes_[id];
    if (!N.live) continue;
    if (N.tokens.empty() || static_cast<int32_t>(N.tokens.size()) > c_) return "node length";
    if (!slots.insert(N.slot).second) return "slot used twice";
    int64_t through = static_cast<int64_t>(N.terminals.size());
    for (size_t i = 0; i < N.children.size(); ++i) {
      const Node& C = nodes_[N.children[i].second];
      if (C.parent != static_cast<int32_t>(id) || C.tokens[0] != N.children[i].first)
        return "child link";
      if (i && N.children[i - 1].first >= N.children[i].first) return "children order";
      through += C.count;
    }
    if (through != N.count) return "count";
    if (N.count >= 2 && N.parent != kRoot && nodes_[N.parent].count < 2) return "shared below private";
  }
  for (const auto& kv : seqs_) {
    int64_t len = 0;
    for (int32_t x = kv.second.term; x != kRoot; x = nodes_[x].parent)
      len += static_cast<int64_t>(nodes_[x].tokens.size());
    if (len != kv.second.length) return "sequence length";
  }
  if (static_cast<int64_t>(slots.size()) != pool_.in_use()) return "pool accounting";
  return "";
}

}  // namespace ca
