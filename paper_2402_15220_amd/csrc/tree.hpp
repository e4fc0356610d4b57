// Prefix-aware KV cache bookkeeping on the host (ChunkAttention, Section 3.1).
//
// The tree of chunks lives in host memory; every operation also emits the
// device copies it implies (KvJob), which the device layer enqueues. The rules
// that the paper leaves open are fixed as follows (and documented in the C
// header): fully matched chunks are descended, a mismatch or the end of a
// sequence inside a chunk splits it (the tail moves to a fresh slot), new
// tokens form chunks of at most c tokens, a chunk used by others is never
// filled, a private last chunk is filled before a new one is grown, removal
// frees zero-count chunks leaf first, and the slot pool is a LIFO free stack
// over ascending fresh ids. Children are kept sorted by first token.
#pragma once

#include <cstdint>
#include <unordered_map>
#include <utility>
#include <vector>

namespace ca {

enum class Err { ok = 0, invalid, nomem, not_found, exists };

// One device copy. kind 0: caller rows [src, src+n) -> slot rows
// [dst_pos, dst_pos+n); kind 1: slot rows of src_slot=src starting at src_pos
// -> dst slot (split tail); kind 2: no copy, set the slot's length to dst_pos.
// Kinds 0 and 1 also set the destination slot's length to dst_pos + n.
struct KvJob {
  int32_t kind;
  int32_t src;
  int32_t src_pos;
  int32_t dst_slot;
  int32_t dst_pos;
  int32_t n;
};

class SlotPool {
 public:
  explicit SlotPool(int64_t capacity) : cap_(capacity) {}
  int64_t available() const { return static_cast<int64_t>(free_.size()) + (cap_ - fresh_); }
  int64_t in_use() const { return fresh_ - static_cast<int64_t>(free_.size()); }
  int64_t capacity() const { return cap_; }
  int32_t alloc() {  // precondition: available() > 0
    if (!free_.empty()) {
      int32_t s = free_.back();
      free_.pop_back();
      return s;
    }
    return static_cast<int32_t>(fresh_++);
  }
  void release(int32_t s) { free_.push_back(s); }

 private:
  int64_t cap_;
  int64_t fresh_ = 0;
  std::vector<int32_t> free_;
};

struct Node {
  std::vector<int32_t> tokens;
  int32_t slot = -1;
  int32_t count = 0;   // sequences whose path contains this node
  int32_t parent = -1;
  std::vector<std::pair<int32_t, int32_t>> children;  // (first token, node id), ascending
  std::vector<int64_t> terminals;                      // ids ending here, ascending
  bool live = false;
};

struct SeqInfo {
  int32_t term;    // terminal node id
  int64_t length;  // tokens
};

class ChunkTree {
 public:
  ChunkTree(int32_t chunk_size, int64_t num_slots);

  int32_t chunk_size() const { return c_; }
  static constexpr int32_t kRoot = 0;

  int64_t match(const int32_t* tokens, int64_t n) const;
  Err insert(int64_t sid, const int32_t* tokens, int64_t n, std::vector<KvJob>* jobs,
             int64_t* matched);
  Err extend(int64_t sid, const int32_t* tokens, int64_t n, int32_t row_base,
             std::vector<KvJob>* jobs, int64_t* matched);
  Err append_batch(int64_t n_seqs, const int64_t* sids, const int32_t* tokens,
                   std::vector<KvJob>* jobs);
  Err remove(int64_t sid);

  // Structure changed since the flag was last cleared (a chunk appeared or
  // disappeared, a chunk was split, a sequence joined or left).
  bool dirty() const { return dirty_; }
  void clear_dirty() {
    dirty_ = false;
    private_growth_only_ = true;
    grown_.clear();
  }
  // Since the flag was last cleared, the only structural changes were new
  // chunks below sequences' private last chunks (decode growth); grown()
  // lists them as (sequence, node) in creation order.
  bool private_growth_only() const { return private_growth_only_; }
  const std::vector<std::pair<int64_t, int32_t>>& grown() const { return grown_; }

  const std::vector<Node>& nodes() const { return nodes_; }
  const Node& node(int32_t id) const { return nodes_[id]; }
  const std::unordered_map<int64_t, SeqInfo>& seqs() const { return seqs_; }
  const SlotPool& pool() const { return pool_; }
  int64_t num_seqs() const { return static_cast<int64_t>(seqs_.size()); }

  // Invariant check (every rule of the header); returns an empty string when
  // the tree is consistent, else a description of the first violation.
  const char* check() const;

 private:
  struct Descent {
    int32_t cur;
    int64_t pos;
    int32_t split_node;  // -1: no split
    int32_t split_at;
  };
  Descent descend(int32_t cur, const int32_t* t, int64_t n, int64_t pos) const;
  int32_t find_child(int32_t node, int32_t tok) const;
  void add_child(int32_t parent, int32_t child);
  void remove_child(int32_t parent, int32_t child);
  int32_t new_node();
  void free_node(int32_t id);
  int32_t split(int32_t x, int32_t p, std::vector<KvJob>* jobs);
  int32_t new_chain(int32_t cur, const int32_t* t, int64_t n, int64_t pos, int32_t row_base,
                    std::vector<KvJob>* jobs);
  static int64_t chunks_for(int64_t rem, int32_t c) { return (rem + c - 1) / c; }
  Err extend_impl(int64_t sid, const int32_t* tokens, int64_t n, int32_t row_base,
                  std::vector<KvJob>* jobs, int64_t* matched);

  int32_t c_;
  SlotPool pool_;
  std::vector<Node> nodes_;
  std::vector<int32_t> free_nodes_;
  std::unordered_map<int64_t, SeqInfo> seqs_;
  void mark_structural() {
    dirty_ = true;
    private_growth_only_ = false;
  }

  bool dirty_ = true;
  bool private_growth_only_ = false;
  std::vector<std::pair<int64_t, int32_t>> grown_;
};

}  // namespace ca
