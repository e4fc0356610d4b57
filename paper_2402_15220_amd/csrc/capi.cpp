// C ABI (include/chunkattn.h): host tree + lazy kernel-context upload +
// kernel launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>
#include <unordered_set>
#include <vector>

#include "../../include/chunkattn.h"
#include "kernels.hpp"
#include "tables.hpp"
#include "tree.hpp"

namespace {

thread_local std::string g_err;

ca_status fail(ca_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

ca_status from_err(ca::Err e, const char* what) {
  switch (e) {
    case ca::Err::ok:
      return CA_OK;
    case ca::Err::invalid:
      return fail(CA_ERR_INVALID, std::string(what) + ": invalid argument");
    case ca::Err::nomem:
      return fail(CA_ERR_NOMEM, std::string(what) + ": chunk pool exhausted");
    case ca::Err::not_found:
      return fail(CA_ERR_NOT_FOUND, std::string(what) + ": unknown sequence id");
    case ca::Err::exists:
      return fail(CA_ERR_EXISTS, std::string(what) + ": sequence id already live");
  }
  return fail(CA_ERR_INVALID, what);
}

ca_status hip_fail(hipError_t e, const char* what) {
  return fail(CA_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

// Called from the catch clause of an entry point: no C++ exception crosses
// the C ABI. Host allocations (tree, tables, work lists, messages) are the
// only source of exceptions in the library.
ca_status on_exception(const char* what) noexcept {
  auto note = [what](const char* tail) noexcept {
    try {
      g_err.assign(what).append(tail);
    } catch (...) {
      g_err.clear();  // no memory even for the message
    }
  };
  try {
    throw;
  } catch (const std::bad_alloc&) {
    note(": out of host memory");
  } catch (...) {
    note(": unexpected internal error");
  }
  return CA_ERR_HOST;
}

int env_int(const char* name, int dflt) {
  const char* s = std::getenv(name);
  return s && *s ? std::atoi(s) : dflt;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Double-buffered pinned host staging for small host-to-device copies on a
// stream: a buffer is written again only after the copy that last read it
// has completed.
struct PinnedStaging {
  char* h[2] = {nullptr, nullptr};
  size_t cap[2] = {0, 0};
  hipEvent_t ev[2] = {nullptr, nullptr};
  bool used[2] = {false, false};
  int next = 0;

  PinnedStaging() = default;
  PinnedStaging(const PinnedStaging&) = delete;
  PinnedStaging& operator=(const PinnedStaging&) = delete;
  ~PinnedStaging() {
    for (int i = 0; i < 2; ++i) {
      if (h[i]) (void)hipHostFree(h[i]);
      if (ev[i]) (void)hipEventDestroy(ev[i]);
    }
  }
  // A host buffer of at least `bytes` for the next copy.
  ca_status acquire(size_t bytes, char** out) {
    const int i = next;
    hipError_t e;
    if (!ev[i] && (e = hipEventCreateWithFlags(&ev[i], hipEventDisableTiming)) != hipSuccess)
      return hip_fail(e, "staging event");
    if (used[i] && (e = hipEventSynchronize(ev[i])) != hipSuccess) return hip_fail(e, "staging wait");
    if (bytes > cap[i]) {
      if (h[i]) (void)hipHostFree(h[i]);
      h[i] = nullptr;
      cap[i] = 0;
      const size_t c = align_up(std::max<size_t>(bytes * 2, 4096), 4096);
      if ((e = hipHostMalloc(reinterpret_cast<void**>(&h[i]), c, hipHostMallocDefault)) != hipSuccess)
        return hip_fail(e, "staging alloc");
      cap[i] = c;
    }
    *out = h[i];
    return CA_OK;
  }
  // Copy the acquired buffer's first `bytes` to `dst` on `stream`.
  ca_status copy(void* dst, size_t bytes, hipStream_t stream) {
    const int i = next;
    hipError_t e;
    if ((e = hipMemcpyAsync(dst, h[i], bytes, hipMemcpyHostToDevice, stream)) != hipSuccess)
      return hip_fail(e, "staging copy");
    if ((e = hipEventRecord(ev[i], stream)) != hipSuccess) return hip_fail(e, "staging record");
    used[i] = true;
    next ^= 1;
    return CA_OK;
  }
};

// Grow-only device buffer; the old one is freed after the stream drains
// (kernels already enqueued may still read it).
ca_status ensure_device(char** p, size_t* cap, size_t need, hipStream_t stream, const char* what) {
  if (need <= *cap) return CA_OK;
  hipError_t e;
  if (*p) {
    if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, what);
    (void)hipFree(*p);
    *p = nullptr;
    *cap = 0;
  }
  const size_t c = align_up(std::max<size_t>(need * 2, 4096), 4096);
  if ((e = hipMalloc(reinterpret_cast<void**>(p), c)) != hipSuccess) return hip_fail(e, what);
  *cap = c;
  return CA_OK;
}

}  // namespace

struct ca_cache {
  ca_config cfg{};
  bool table_only = false;
  ca::ChunkTree tree;
  ca::Tables tables;
  ca::WorkLists work;
  bool work_valid = false;
  int64_t patches = 0;        // in-place work-list updates so far
  bool check_patches = false; // compare every patch with a rebuild (CA_CHECK_PATCH=1)
  std::string patch_error;    // set when such a comparison failed
  int32_t seg_chunks = 0;  // 0: automatic
  int32_t num_cus = 256;
  int32_t split_chunks = 0;
  int32_t phase_mask = 7;
  int32_t schedule = 2;  // see ca_set_tuning
  ca::SideStream side;

  // device state
  int32_t* d_slot_len = nullptr;
  char* d_blob = nullptr;
  size_t d_blob_cap = 0;
  int32_t* d_cnt = nullptr;  // [B][H] arrival counters of the partial-writing schedules
  size_t d_cnt_cap = 0;
  int32_t prefill_split = 0;     // key-range parts of a prefill tile (0: automatic)
  float* d_pf_ws = nullptr;      // prefill partials of split tiles
  size_t d_pf_ws_cap = 0;
  int32_t* d_pf_cnt = nullptr;   // prefill arrival counters, one per tile
  size_t d_pf_cnt_cap = 0;
  PinnedStaging work_stage;     // kernel context uploads
  PinnedStaging prefill_stage;  // prefill paths
  PinnedStaging rowmap_stage;   // caller row orders
  int32_t* d_rowmap = nullptr;  // [B] tree row -> caller row, on the device
  size_t d_rowmap_cap = 0;
  std::vector<int32_t> rowmap;  // what d_rowmap holds (empty: nothing uploaded)
  char* d_path = nullptr;       // prefill path on the device (long paths)
  std::vector<int32_t> prefill_host_path;  // short paths, passed in the kernel arguments
  size_t d_path_cap = 0;
  ca::DevWork dw;
  bool dw_valid = false;
  int64_t uploads = 0;
  char* scratch = nullptr;  // this device's copy of the static scratch (ca_attention_noalloc)
  std::string scratch_error;  // why it is null

  // host export buffers
  ca::Tables exported;

  explicit ca_cache(const ca_config& c) : cfg(c), tree(c.chunk_size, c.num_slots) {}
  ~ca_cache() {
    if (d_slot_len) (void)hipFree(d_slot_len);
    if (d_blob) (void)hipFree(d_blob);
    if (d_cnt) (void)hipFree(d_cnt);
    if (side.fork) (void)hipEventDestroy(side.fork);
    if (side.join) (void)hipEventDestroy(side.join);
    if (side.stream) (void)hipStreamDestroy(side.stream);
    if (d_path) (void)hipFree(d_path);
    if (d_rowmap) (void)hipFree(d_rowmap);
    if (d_pf_ws) (void)hipFree(d_pf_ws);
    if (d_pf_cnt) (void)hipFree(d_pf_cnt);
  }

  size_t esize() const { return cfg.dtype == CA_FP16 ? 2 : 4; }
  int32_t token_head_bytes() const { return static_cast<int32_t>(2 * cfg.head_dim * esize()); }

  // Work lists for the current tree. Decode growth (new private chunks at
  // the end of paths) patches them in place (Section 3.3's context stays
  // valid except for those rows' chunk lists); anything else rebuilds the
  // tables and the work lists. `tables` keeps row_seq valid either way.
  void ensure_work() {
    if (work_valid && !tree.dirty()) return;
    bool patched = false;
    if (work_valid && tree.private_growth_only() && split_chunks <= 0 && !patch_error.size())
      patched = ca::patch_work(tree, &work);
    if (patched) {
      ++patches;
      if (check_patches) {
        ca::Tables t;
        ca::WorkLists full;
        ca::build_tables(tree, &t);
        // patched lists keep the segment size of their last rebuild
        ca::build_work(tree, t, work.seg_chunks, split_chunks, schedule != 0, cfg.num_heads,
                       num_cus, &full, schedule == 4, token_head_bytes());
        const char* d = ca::same_work(work, full);
        if (*d) patch_error = std::string("work-list patch differs from a rebuild: ") + d;
      }
    } else {
      ca::build_tables(tree, &tables);
      ca::build_work(tree, tables, seg_chunks, split_chunks, schedule != 0, cfg.num_heads, num_cus,
                     &work, schedule == 4, token_head_bytes());
    }
    work_valid = true;
    dw_valid = false;
    tree.clear_dirty();
  }

  size_t ws_bytes() const {
    const size_t np = static_cast<size_t>(work.n_parts);
    const size_t H = cfg.num_heads, D = cfg.head_dim;
    return align_up(np * H * D * 4, 256) + align_up(np * H * 2 * 4, 256);
  }

  // Flatten the work lists into one blob and copy it to the device on
  // `stream` through a double-buffered pinned staging area.
  ca_status upload(hipStream_t stream) {
    const auto& W = work;
    size_t off = 0;
    auto place = [&](size_t bytes) {
      const size_t o = off;
      off = align_up(off + bytes, 16);
      return o;
    };
    const size_t o_segs = place(W.segs.size() * sizeof(ca::CfSeg));
    const size_t o_seg_slots = place(W.seg_slots.size() * 4);
    const size_t o_items = place(W.items.size() * sizeof(ca::SfItem));
    const size_t o_priv = place(W.priv_slot.size() * 4);
    const size_t o_pptr = place(W.part_ptr.size() * 4);
    const size_t o_parts = place(W.parts.size() * 4);
    const size_t o_mg = place(W.mg_rows.size() * 4);
    const size_t total = std::max<size_t>(off, 16);

    ca_status st = ensure_device(&d_blob, &d_blob_cap, total, stream, "upload alloc");
    if (st != CA_OK) return st;
    char* h = nullptr;
    if ((st = work_stage.acquire(total, &h)) != CA_OK) return st;
    auto put = [&](size_t o, const void* src, size_t bytes) {
      if (bytes) std::memcpy(h + o, src, bytes);
    };
    put(o_segs, W.segs.data(), W.segs.size() * sizeof(ca::CfSeg));
    put(o_seg_slots, W.seg_slots.data(), W.seg_slots.size() * 4);
    put(o_items, W.items.data(), W.items.size() * sizeof(ca::SfItem));
    put(o_priv, W.priv_slot.data(), W.priv_slot.size() * 4);
    put(o_pptr, W.part_ptr.data(), W.part_ptr.size() * 4);
    put(o_parts, W.parts.data(), W.parts.size() * 4);
    put(o_mg, W.mg_rows.data(), W.mg_rows.size() * 4);
    if ((st = work_stage.copy(d_blob, total, stream)) != CA_OK) return st;

    dw.segs = reinterpret_cast<const ca::CfSeg*>(d_blob + o_segs);
    dw.seg_slots = reinterpret_cast<const int32_t*>(d_blob + o_seg_slots);
    dw.n_segs = static_cast<int32_t>(W.segs.size());
    dw.max_seg_rows = W.max_seg_rows;
    dw.items = reinterpret_cast<const ca::SfItem*>(d_blob + o_items);
    dw.n_items = static_cast<int32_t>(W.items.size());
    dw.priv_slot = reinterpret_cast<const int32_t*>(d_blob + o_priv);
    dw.part_ptr = reinterpret_cast<const int32_t*>(d_blob + o_pptr);
    dw.parts = reinterpret_cast<const int32_t*>(d_blob + o_parts);
    dw.mg_rows = reinterpret_cast<const int32_t*>(d_blob + o_mg);
    dw.n_mg = static_cast<int32_t>(W.mg_rows.size());
    dw.schedule = schedule;
    dw.seg_group_ptr = W.seg_group_ptr.data();
    dw.n_seg_groups = W.seg_group_ptr.empty() ? 0 : static_cast<int32_t>(W.seg_group_ptr.size()) - 1;
    dw_valid = true;
    ++uploads;
    return CA_OK;
  }

  // Tree row -> caller row for a caller order given as seq_ids[0..n) (every
  // live sequence once); uploaded only when it differs from the device copy.
  ca_status upload_row_map(const int64_t* seq_ids, int64_t n, hipStream_t stream) {
    const size_t B = tables.row_seq.size();
    std::vector<int32_t> map(B, -1);
    for (int64_t i = 0; i < n; ++i) {
      auto it = work.row_of_seq.find(seq_ids[i]);
      if (it == work.row_of_seq.end())
        return fail(CA_ERR_INVALID, "ca_attention_ordered: sequence " +
                                        std::to_string(seq_ids[i]) + " is not live");
      if (map[it->second] >= 0)
        return fail(CA_ERR_INVALID, "ca_attention_ordered: sequence " +
                                        std::to_string(seq_ids[i]) + " listed twice");
      map[it->second] = static_cast<int32_t>(i);
    }
    if (map == rowmap) return CA_OK;
    const size_t bytes = std::max<size_t>(B * sizeof(int32_t), 16);
    ca_status st = ensure_device(reinterpret_cast<char**>(&d_rowmap), &d_rowmap_cap, bytes, stream,
                                 "row map alloc");
    if (st != CA_OK) return st;
    char* h = nullptr;
    if ((st = rowmap_stage.acquire(bytes, &h)) != CA_OK) return st;
    std::memcpy(h, map.data(), B * sizeof(int32_t));
    if ((st = rowmap_stage.copy(d_rowmap, bytes, stream)) != CA_OK) return st;
    rowmap.swap(map);
    return CA_OK;
  }

  // The concurrent schedule's second stream (default priority) and its
  // fork/join events, created on first use.
  ca_status ensure_side() {
    hipError_t e;
    if (!side.stream &&
        (e = hipStreamCreateWithFlags(&side.stream, hipStreamNonBlocking)) != hipSuccess)
      return hip_fail(e, "side stream");
    if (!side.fork && (e = hipEventCreateWithFlags(&side.fork, hipEventDisableTiming)) != hipSuccess)
      return hip_fail(e, "fork event");
    if (!side.join && (e = hipEventCreateWithFlags(&side.join, hipEventDisableTiming)) != hipSuccess)
      return hip_fail(e, "join event");
    return CA_OK;
  }

  // At least n arrival counters in *p. They are zeroed once when allocated;
  // every launch leaves them at zero again.
  static ca_status ensure_counters(int32_t** p, size_t* cap_, size_t n, hipStream_t stream) {
    if (n <= *cap_) return CA_OK;
    hipError_t e;
    if (*p) {
      if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "counter sync");
      (void)hipFree(*p);
      *p = nullptr;
      *cap_ = 0;
    }
    const size_t cap = std::max<size_t>(n * 2, 1024);
    if ((e = hipMalloc(reinterpret_cast<void**>(p), cap * sizeof(int32_t))) != hipSuccess)
      return hip_fail(e, "counter alloc");
    if ((e = ca::launch_fill_i32(*p, static_cast<int64_t>(cap), 0, stream)) != hipSuccess)
      return hip_fail(e, "counter clear");
    *cap_ = cap;
    return CA_OK;
  }

  // Enqueue K/V copies. Jobs are batched per launch; a job that touches a
  // slot already touched by the pending batch starts a new launch, so copies
  // within one launch never depend on each other.
  ca_status run_jobs(const std::vector<ca::KvJob>& jobs, const void* k, const void* v,
                     hipStream_t stream) {
    if (table_only || jobs.empty()) return CA_OK;
    std::vector<ca::KvJob> batch;
    std::unordered_set<int32_t> touched;
    auto flush = [&]() -> ca_status {
      if (batch.empty()) return CA_OK;
      hipError_t e = ca::launch_kv_jobs(batch.data(), static_cast<int>(batch.size()),
                                        cfg.dtype == CA_FP16 ? 0 : 1, cfg.num_heads, cfg.head_dim,
                                        cfg.chunk_size, cfg.slot_stride, cfg.head_stride, k, v,
                                        cfg.k_pool, cfg.v_pool, d_slot_len, stream);
      batch.clear();
      touched.clear();
      if (e != hipSuccess) return hip_fail(e, "kv copy launch");
      return CA_OK;
    };
    for (const auto& j : jobs) {
      const bool hazard = touched.count(j.dst_slot) || (j.kind == 1 && touched.count(j.src));
      if (hazard || static_cast<int>(batch.size()) == ca::kKvJobsPerLaunch) {
        ca_status s = flush();
        if (s != CA_OK) return s;
      }
      batch.push_back(j);
      touched.insert(j.dst_slot);
      if (j.kind == 1) touched.insert(j.src);
    }
    return flush();
  }
};

extern "C" {

const char* ca_last_error(void) { return g_err.c_str(); }

ca_status ca_create(const ca_config* cfg, ca_cache** out) try {
  if (!cfg || !out) return fail(CA_ERR_INVALID, "ca_create: null argument");
  if (cfg->chunk_size < 1) return fail(CA_ERR_INVALID, "ca_create: chunk_size < 1");
  if (cfg->num_heads < 1) return fail(CA_ERR_INVALID, "ca_create: num_heads < 1");
  if (cfg->head_dim != 64 && cfg->head_dim != 128)
    return fail(CA_ERR_INVALID, "ca_create: head_dim must be 64 or 128");
  {
    // read as its integer representation: a value outside the enumeration is
    // rejected without being loaded as a ca_dtype
    int32_t dt;
    static_assert(sizeof(cfg->dtype) == sizeof(dt), "ca_dtype is a 32-bit enumeration");
    std::memcpy(&dt, &cfg->dtype, sizeof dt);
    if (dt != CA_FP16 && dt != CA_FP32) return fail(CA_ERR_INVALID, "ca_create: bad dtype");
  }
  if (cfg->num_slots < 1 || cfg->num_slots > INT32_MAX)
    return fail(CA_ERR_INVALID, "ca_create: num_slots out of range");
  if ((cfg->k_pool == nullptr) != (cfg->v_pool == nullptr))
    return fail(CA_ERR_INVALID, "ca_create: give both pools or neither");
  if ((reinterpret_cast<uintptr_t>(cfg->k_pool) | reinterpret_cast<uintptr_t>(cfg->v_pool)) & 15)
    return fail(CA_ERR_INVALID, "ca_create: pools must be 16-byte aligned");
  ca_config norm = *cfg;
  {
    const int64_t tile = static_cast<int64_t>(cfg->chunk_size) * cfg->head_dim;
    const int64_t es = cfg->dtype == CA_FP16 ? 2 : 4;
    if (norm.head_stride == 0) norm.head_stride = tile;
    if (norm.slot_stride == 0) norm.slot_stride = cfg->num_heads * norm.head_stride;
    if (norm.head_stride < tile || norm.slot_stride < (cfg->num_heads - 1) * norm.head_stride + tile)
      return fail(CA_ERR_INVALID, "ca_create: strides overlap tiles");
    if ((norm.head_stride * es) % 16 || (norm.slot_stride * es) % 16)
      return fail(CA_ERR_INVALID, "ca_create: strides must be multiples of 16 bytes");
  }
  ca_cache* c = new (std::nothrow) ca_cache(norm);
  if (!c) return fail(CA_ERR_HOST, "ca_create: out of host memory");
  c->table_only = cfg->k_pool == nullptr;
  c->seg_chunks = std::max(0, env_int("CA_CF_SEG", 0));
  c->split_chunks = env_int("CA_SPLIT", 0);
  c->schedule = std::min(4, std::max(0, env_int("CA_SCHEDULE", 2)));
  c->check_patches = env_int("CA_CHECK_PATCH", 0) != 0;
  c->prefill_split = std::min(64, std::max(0, env_int("CA_PREFILL_SPLIT", 0)));
  if (!c->table_only) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        cus > 0)
      c->num_cus = cus;
    hipError_t e = hipMalloc(reinterpret_cast<void**>(&c->d_slot_len),
                             static_cast<size_t>(cfg->num_slots) * sizeof(int32_t));
    if (e == hipSuccess) e = hipMemset(c->d_slot_len, 0, static_cast<size_t>(cfg->num_slots) * 4);
    if (e == hipSuccess) {
      // this device's scratch address (once per device, this device current);
      // only ca_attention_noalloc needs it, so a failure is reported there
      const hipError_t se = ca::scratch_address(&c->scratch);
      if (se != hipSuccess) {
        c->scratch = nullptr;
        c->scratch_error = hipGetErrorString(se);
        (void)hipGetLastError();  // not left for a later launch check to find
      }
    }
    if (e != hipSuccess) {
      delete c;
      return hip_fail(e, "ca_create");
    }
  }
  *out = c;
  return CA_OK;
} catch (...) {
  return on_exception("ca_create");
}

ca_status ca_destroy(ca_cache* cache) {
  delete cache;
  return CA_OK;
}

static ca_status check_tokens(const int32_t* tokens, int64_t n, const char* what) {
  if (!tokens || n < 1 || n > INT32_MAX) return fail(CA_ERR_INVALID, std::string(what) + ": bad tokens");
  for (int64_t i = 0; i < n; ++i)
    if (tokens[i] < 0) return fail(CA_ERR_INVALID, std::string(what) + ": negative token");
  return CA_OK;
}

static ca_status check_kv(const ca_cache* c, const void* k, const void* v, const char* what) {
  if (c->table_only) {
    if (k || v) return fail(CA_ERR_INVALID, std::string(what) + ": table-only cache takes no K/V");
    return CA_OK;
  }
  if (!k || !v) return fail(CA_ERR_INVALID, std::string(what) + ": null K/V");
  if ((reinterpret_cast<uintptr_t>(k) | reinterpret_cast<uintptr_t>(v)) & 15)
    return fail(CA_ERR_INVALID, std::string(what) + ": K/V must be 16-byte aligned");
  return CA_OK;
}

ca_status ca_match(const ca_cache* cache, const int32_t* tokens, int64_t n, int64_t* matched) try {
  if (!cache || !matched) return fail(CA_ERR_INVALID, "ca_match: null argument");
  ca_status s = check_tokens(tokens, n, "ca_match");
  if (s != CA_OK) return s;
  *matched = cache->tree.match(tokens, n);
  return CA_OK;
} catch (...) {
  return on_exception("ca_match");
}

ca_status ca_insert(ca_cache* cache, int64_t seq_id, const int32_t* tokens, int64_t n,
                    const void* k, const void* v, void* stream, int64_t* matched) try {
  if (!cache) return fail(CA_ERR_INVALID, "ca_insert: null cache");
  ca_status s = check_tokens(tokens, n, "ca_insert");
  if (s != CA_OK) return s;
  if ((s = check_kv(cache, k, v, "ca_insert")) != CA_OK) return s;
  std::vector<ca::KvJob> jobs;
  int64_t m = 0;
  ca::Err e = cache->tree.insert(seq_id, tokens, n, &jobs, &m);
  if (e != ca::Err::ok) return from_err(e, "ca_insert");
  if (matched) *matched = m;
  return cache->run_jobs(jobs, k, v, static_cast<hipStream_t>(stream));
} catch (...) {
  return on_exception("ca_insert");
}

ca_status ca_extend(ca_cache* cache, int64_t seq_id, const int32_t* tokens, int64_t n,
                    const void* k, const void* v, void* stream, int64_t* matched) try {
  if (!cache) return fail(CA_ERR_INVALID, "ca_extend: null cache");
  ca_status s = check_tokens(tokens, n, "ca_extend");
  if (s != CA_OK) return s;
  if ((s = check_kv(cache, k, v, "ca_extend")) != CA_OK) return s;
  std::vector<ca::KvJob> jobs;
  int64_t m = 0;
  ca::Err e = cache->tree.extend(seq_id, tokens, n, 0, &jobs, &m);
  if (e != ca::Err::ok) return from_err(e, "ca_extend");
  if (matched) *matched = m;
  return cache->run_jobs(jobs, k, v, static_cast<hipStream_t>(stream));
} catch (...) {
  return on_exception("ca_extend");
}

ca_status ca_append_batch(ca_cache* cache, int64_t n_seqs, const int64_t* seq_ids,
                          const int32_t* tokens, const void* k, const void* v, void* stream) try {
  if (!cache) return fail(CA_ERR_INVALID, "ca_append_batch: null cache");
  if (n_seqs < 0 || n_seqs > INT32_MAX) return fail(CA_ERR_INVALID, "ca_append_batch: bad n_seqs");
  if (n_seqs == 0) return CA_OK;
  if (!seq_ids) return fail(CA_ERR_INVALID, "ca_append_batch: null seq_ids");
  ca_status s = check_tokens(tokens, n_seqs, "ca_append_batch");
  if (s != CA_OK) return s;
  if ((s = check_kv(cache, k, v, "ca_append_batch")) != CA_OK) return s;
  std::vector<ca::KvJob> jobs;
  ca::Err e = cache->tree.append_batch(n_seqs, seq_ids, tokens, &jobs);
  if (e != ca::Err::ok) return from_err(e, "ca_append_batch");
  return cache->run_jobs(jobs, k, v, static_cast<hipStream_t>(stream));
} catch (...) {
  return on_exception("ca_append_batch");
}

ca_status ca_remove(ca_cache* cache, int64_t seq_id) try {
  if (!cache) return fail(CA_ERR_INVALID, "ca_remove: null cache");
  return from_err(cache->tree.remove(seq_id), "ca_remove");
} catch (...) {
  return on_exception("ca_remove");
}

ca_status ca_num_seqs(const ca_cache* cache, int64_t* B) {
  if (!cache || !B) return fail(CA_ERR_INVALID, "ca_num_seqs: null argument");
  *B = cache->tree.num_seqs();
  return CA_OK;
}

ca_status ca_seq_order(const ca_cache* cache, int64_t* seq_ids, int64_t cap) try {
  if (!cache || (!seq_ids && cache->tree.num_seqs() > 0))
    return fail(CA_ERR_INVALID, "ca_seq_order: null argument");
  if (cap < cache->tree.num_seqs()) return fail(CA_ERR_INVALID, "ca_seq_order: cap < B");
  ca_cache* c = const_cast<ca_cache*>(cache);
  c->ensure_work();
  std::copy(c->tables.row_seq.begin(), c->tables.row_seq.end(), seq_ids);
  return CA_OK;
} catch (...) {
  return on_exception("ca_seq_order");
}

ca_status ca_workspace_size(const ca_cache* cache, size_t* bytes) try {
  if (!cache || !bytes) return fail(CA_ERR_INVALID, "ca_workspace_size: null argument");
  ca_cache* c = const_cast<ca_cache*>(cache);
  c->ensure_work();
  *bytes = c->ws_bytes();
  return CA_OK;
} catch (...) {
  return on_exception("ca_workspace_size");
}

// Arguments common to the attention entry points; nothing is changed when
// they are refused.
static ca_status check_attention_io(const ca_cache* cache, const void* q, void* o, float scale) {
  if (!q || !o) return fail(CA_ERR_INVALID, "ca_attention: null q/o");
  if ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(o)) & 15)
    return fail(CA_ERR_INVALID, "ca_attention: q/o must be 16-byte aligned");
  if (!(scale >= 0.f) || std::isinf(scale)) return fail(CA_ERR_INVALID, "ca_attention: bad scale");
  (void)cache;
  return CA_OK;
}

// Enqueue the attention kernels for the uploaded kernel context. Partials
// go to ws (partial O, then 256-byte aligned (m, n) pairs), arrival counters
// to cnt (B * H of them, zero on entry; the kernels leave them zero).
static ca_status launch_attention_call(ca_cache* cache, const void* q, void* o, float scale,
                                       char* ws, int32_t* cnt, const int32_t* row_map,
                                       hipStream_t s) {
  const float sc = scale == 0.f ? 1.f / std::sqrt(static_cast<float>(cache->cfg.head_dim)) : scale;
  ca::AttnArgs a{};
  a.dtype = cache->cfg.dtype == CA_FP16 ? 0 : 1;
  a.H = cache->cfg.num_heads;
  a.D = cache->cfg.head_dim;
  a.C = cache->cfg.chunk_size;
  a.q = q;
  a.o = o;
  a.kpool = cache->cfg.k_pool;
  a.vpool = cache->cfg.v_pool;
  a.ss = cache->cfg.slot_stride;
  a.hs = cache->cfg.head_stride;
  a.slot_len = cache->d_slot_len;
  const size_t np = static_cast<size_t>(cache->work.n_parts);
  const size_t o_bytes = np * a.H * a.D * 4;
  if (o_bytes > 0xFFFFFFFFull)
    return fail(CA_ERR_INVALID, "ca_attention: partial-O workspace above 4 GiB (" +
                                    std::to_string(o_bytes) + " bytes); use longer segments");
  a.ws_o = reinterpret_cast<float*>(ws);
  a.ws_o_bytes = static_cast<uint32_t>(o_bytes);
  a.ws_ml = np ? reinterpret_cast<float*>(ws + align_up(o_bytes, 256)) : nullptr;
  a.qscale = sc * 1.4426950408889634f;
  a.cnt = cnt;
  a.row_map = row_map;
  hipError_t e = ca::launch_attention(a, cache->dw, s, cache->phase_mask, cache->side);
  if (e != hipSuccess) return hip_fail(e, "ca_attention launch");
  return CA_OK;
}

static ca_status attention_impl(ca_cache* cache, const void* q, void* o, float scale, void* ws,
                                size_t ws_bytes, void* stream, const int64_t* seq_ids,
                                int64_t n) {
  if (!cache) return fail(CA_ERR_INVALID, "ca_attention: null cache");
  if (cache->table_only) return fail(CA_ERR_INVALID, "ca_attention: table-only cache");
  if (seq_ids && n != cache->tree.num_seqs())
    return fail(CA_ERR_INVALID, "ca_attention_ordered: n differs from the number of live sequences");
  if (cache->tree.num_seqs() == 0) return CA_OK;
  ca_status st = check_attention_io(cache, q, o, scale);
  if (st != CA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  cache->ensure_work();
  const size_t need = cache->ws_bytes();
  if (cache->work.n_parts > 0 && (!ws || ws_bytes < need || (reinterpret_cast<uintptr_t>(ws) & 255)))
    return fail(CA_ERR_WORKSPACE, "ca_attention: workspace missing, misaligned or smaller than " +
                                      std::to_string(need) + " bytes");
  if (!cache->dw_valid && (st = cache->upload(s)) != CA_OK) return st;
  const int32_t* row_map = nullptr;
  if (seq_ids) {
    if ((st = cache->upload_row_map(seq_ids, n, s)) != CA_OK) return st;
    row_map = cache->d_rowmap;
  }
  if (cache->schedule == 3 && (st = cache->ensure_side()) != CA_OK) return st;
  st = ca_cache::ensure_counters(&cache->d_cnt, &cache->d_cnt_cap,
                                 static_cast<size_t>(cache->tree.num_seqs()) * cache->cfg.num_heads, s);
  if (st != CA_OK) return st;
  return launch_attention_call(cache, q, o, scale, static_cast<char*>(ws), cache->d_cnt, row_map, s);
}

ca_status ca_attention(ca_cache* cache, const void* q, void* o, float scale, void* ws,
                       size_t ws_bytes, void* stream) try {
  return attention_impl(cache, q, o, scale, ws, ws_bytes, stream, nullptr, 0);
} catch (...) {
  return on_exception("ca_attention");
}

ca_status ca_attention_ordered(ca_cache* cache, const void* q, void* o, const int64_t* seq_ids,
                               int64_t n, float scale, void* ws, size_t ws_bytes, void* stream) try {
  if (!seq_ids && n > 0) return fail(CA_ERR_INVALID, "ca_attention_ordered: null seq_ids");
  static const int64_t kNone = 0;
  return attention_impl(cache, q, o, scale, ws, ws_bytes, stream, seq_ids ? seq_ids : &kNone, n);
} catch (...) {
  return on_exception("ca_attention_ordered");
}

ca_status ca_attention_noalloc(ca_cache* cache, const void* q, void* o, float scale,
                               void* stream) try {
  if (!cache) return fail(CA_ERR_INVALID, "ca_attention_noalloc: null cache");
  if (cache->table_only) return fail(CA_ERR_INVALID, "ca_attention_noalloc: table-only cache");
  if (cache->tree.num_seqs() == 0) return CA_OK;
  ca_status st = check_attention_io(cache, q, o, scale);
  if (st != CA_OK) return st;
  // Everything the call needs must exist already: the kernel context on the
  // device (ca_prepare or an earlier attention call after the last tree or
  // tuning change) and, for the two-stream schedule, its stream.
  if (!cache->work_valid || cache->tree.dirty() || !cache->dw_valid)
    return fail(CA_ERR_INVALID,
                "ca_attention_noalloc: kernel context not current (call ca_prepare after the "
                "last tree or tuning change)");
  if (cache->schedule == 3 && !cache->side.stream)
    return fail(CA_ERR_INVALID, "ca_attention_noalloc: the two-stream schedule's stream does not "
                                "exist yet (one ca_attention call creates it)");
  if (!cache->scratch)
    return fail(CA_ERR_DEVICE, "ca_attention_noalloc: no device scratch: " + cache->scratch_error);
  const size_t counters = static_cast<size_t>(cache->tree.num_seqs()) * cache->cfg.num_heads;
  const size_t parts = cache->ws_bytes();
  if (counters * sizeof(int32_t) > ca::kScratchCounterBytes ||
      parts > ca::kScratchBytes - ca::kScratchCounterBytes)
    return fail(CA_ERR_WORKSPACE,
                "ca_attention_noalloc: the call needs " + std::to_string(counters) +
                    " (row, head) counters and " + std::to_string(parts) +
                    " bytes of partials; the device scratch holds " +
                    std::to_string(ca::kScratchCounterBytes / sizeof(int32_t)) + " and " +
                    std::to_string(ca::kScratchBytes - ca::kScratchCounterBytes) +
                    " (use ca_attention with a caller workspace)");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* cnt = reinterpret_cast<int32_t*>(cache->scratch);
  // the scratch keeps whatever the last call on this GPU left: the counters
  // are cleared by a kernel on the caller's stream before every call
  hipError_t e = ca::launch_fill_i32(cnt, static_cast<int64_t>(counters), 0, s);
  if (e != hipSuccess) return hip_fail(e, "ca_attention_noalloc counter clear");
  return launch_attention_call(cache, q, o, scale, cache->scratch + ca::kScratchCounterBytes, cnt,
                               nullptr, s);
} catch (...) {
  return on_exception("ca_attention_noalloc");
}

ca_status ca_prepare(ca_cache* cache, void* stream, int32_t* uploaded) try {
  if (uploaded) *uploaded = 0;
  if (!cache) return fail(CA_ERR_INVALID, "ca_prepare: null cache");
  cache->ensure_work();
  if (cache->table_only || cache->tree.num_seqs() == 0 || cache->dw_valid) return CA_OK;
  ca_status st = cache->upload(static_cast<hipStream_t>(stream));
  if (st != CA_OK) return st;
  if (uploaded) *uploaded = 1;
  return CA_OK;
} catch (...) {
  return on_exception("ca_prepare");
}

ca_status ca_prefill_attention(ca_cache* cache, int64_t seq_id, const void* q, void* o,
                               int64_t n_q, float scale, void* stream) try {
  if (!cache) return fail(CA_ERR_INVALID, "ca_prefill_attention: null cache");
  if (cache->table_only) return fail(CA_ERR_INVALID, "ca_prefill_attention: table-only cache");
  if (cache->cfg.dtype != CA_FP16)
    return fail(CA_ERR_INVALID, "ca_prefill_attention: fp16 caches only");
  const auto& seqs = cache->tree.seqs();
  auto it = seqs.find(seq_id);
  if (it == seqs.end()) return fail(CA_ERR_NOT_FOUND, "ca_prefill_attention: unknown sequence");
  const int64_t L = it->second.length;
  if (n_q < 0 || n_q > L) return fail(CA_ERR_INVALID, "ca_prefill_attention: need 0 <= n_q <= length");
  if (n_q == 0) return CA_OK;
  if (!q || !o) return fail(CA_ERR_INVALID, "ca_prefill_attention: null q/o");
  if ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(o)) & 15)
    return fail(CA_ERR_INVALID, "ca_prefill_attention: q/o must be 16-byte aligned");
  if (!(scale >= 0.f) || std::isinf(scale))
    return fail(CA_ERR_INVALID, "ca_prefill_attention: bad scale");
  if (L > INT32_MAX / 2) return fail(CA_ERR_INVALID, "ca_prefill_attention: sequence too long");
  hipStream_t s = static_cast<hipStream_t>(stream);

  // root -> leaf path: slots and start positions (a chunk may be shorter
  // than c). A short path goes to the kernel inside its arguments; a longer
  // one is uploaded through the pinned staging ring.
  std::vector<int32_t> path;
  for (int32_t id = it->second.term; id != ca::ChunkTree::kRoot; id = cache->tree.node(id).parent)
    path.push_back(id);
  const int32_t nc = static_cast<int32_t>(path.size());
  const bool inline_path = nc <= ca::kPrefillInlineChunks;
  const size_t bytes = (2 * static_cast<size_t>(nc) + 1) * sizeof(int32_t);
  std::vector<int32_t>& hp = cache->prefill_host_path;
  int32_t* slot = nullptr;
  char* h = nullptr;
  ca_status st = CA_OK;
  if (inline_path) {
    hp.resize(2 * static_cast<size_t>(nc) + 1);
    slot = hp.data();
  } else {
    if ((st = cache->prefill_stage.acquire(bytes, &h)) != CA_OK) return st;
    slot = reinterpret_cast<int32_t*>(h);
  }
  int32_t* start = slot + nc;
  int32_t pos = 0;
  for (int32_t k = 0; k < nc; ++k) {
    const ca::Node& nd = cache->tree.node(path[nc - 1 - k]);
    slot[k] = nd.slot;
    start[k] = pos;
    pos += static_cast<int32_t>(nd.tokens.size());
  }
  start[nc] = pos;
  if (pos != L) return fail(CA_ERR_INVALID, "ca_prefill_attention: inconsistent path");
  if (!inline_path) {
    if ((st = ensure_device(&cache->d_path, &cache->d_path_cap, bytes, s, "prefill path")) != CA_OK)
      return st;
    if ((st = cache->prefill_stage.copy(cache->d_path, bytes, s)) != CA_OK) return st;
  }

  ca::PrefillArgs a{};
  a.H = cache->cfg.num_heads;
  a.D = cache->cfg.head_dim;
  a.C = cache->cfg.chunk_size;
  a.q = q;
  a.o = o;
  a.kpool = cache->cfg.k_pool;
  a.vpool = cache->cfg.v_pool;
  a.ss = cache->cfg.slot_stride;
  a.hs = cache->cfg.head_stride;
  if (inline_path) {
    a.host_path = slot;
  } else {
    a.chunk_slot = reinterpret_cast<const int32_t*>(cache->d_path);
    a.chunk_start = a.chunk_slot + nc;
  }
  a.n_chunks = nc;
  a.n_q = static_cast<int>(n_q);
  const float sc = scale == 0.f ? 1.f / std::sqrt(static_cast<float>(a.D)) : scale;
  a.qscale = sc * 1.4426950408889634f;
  // Key-range split: when the (64-query tile, head) blocks alone would leave
  // compute units idle, cut each tile's units (64-row pieces of its chunks)
  // into parts of at least six units, up to about one block per CU (one
  // block fits a CU, so more blocks run in rounds): a part's time is mostly
  // its block's fixed latency (start, first loads, merge, partial stores),
  // so parts are kept long.
  const int64_t tiles = (n_q + 63) / 64 * static_cast<int64_t>(a.H);
  const int64_t units = static_cast<int64_t>(nc) * ((a.C + 63) / 64);
  int64_t split = 1;
  if (cache->prefill_split > 0)
    split = cache->prefill_split;
  else if (tiles < cache->num_cus)
    split = std::min<int64_t>({(cache->num_cus + tiles - 1) / tiles, std::max<int64_t>(1, units / 6), 16});
  a.n_split = static_cast<int>(split);
  if (split > 1) {
    const size_t ws = static_cast<size_t>(tiles * split) * ca::prefill_part_bytes(a.D);
    if ((st = ensure_device(reinterpret_cast<char**>(&cache->d_pf_ws), &cache->d_pf_ws_cap, ws, s,
                            "prefill partials")) != CA_OK)
      return st;
    if ((st = ca_cache::ensure_counters(&cache->d_pf_cnt, &cache->d_pf_cnt_cap,
                                        static_cast<size_t>(tiles), s)) != CA_OK)
      return st;
    a.ws = cache->d_pf_ws;
    a.ws_bytes = ws;
    a.cnt = cache->d_pf_cnt;
  }
  hipError_t e = ca::launch_prefill(a, s);
  if (e != hipSuccess) return hip_fail(e, "ca_prefill_attention launch");
  return CA_OK;
} catch (...) {
  return on_exception("ca_prefill_attention");
}

ca_status ca_export_tables(const ca_cache* cache, ca_tables* out) try {
  if (!cache || !out) return fail(CA_ERR_INVALID, "ca_export_tables: null argument");
  ca_cache* c = const_cast<ca_cache*>(cache);
  ca::build_tables(c->tree, &c->exported);
  const ca::Tables& T = c->exported;
  out->B = static_cast<int64_t>(T.row_seq.size());
  out->n_nodes = static_cast<int64_t>(T.node_slot.size());
  out->n_shared = static_cast<int64_t>(T.shr_node.size());
  out->row_seq = T.row_seq.data();
  out->node_slot = T.node_slot.data();
  out->node_len = T.node_len.data();
  out->node_row_begin = T.node_row_begin.data();
  out->node_row_end = T.node_row_end.data();
  out->node_parent = T.node_parent.data();
  out->node_start_pos = T.node_start_pos.data();
  out->shr_node = T.shr_node.data();
  out->shr_part_base = T.shr_part_base.data();
  out->priv_ptr = T.priv_ptr.data();
  out->priv_node = T.priv_node.data();
  out->shr_ptr = T.shr_ptr.data();
  out->shr_part = T.shr_part.data();
  return CA_OK;
} catch (...) {
  return on_exception("ca_export_tables");
}

ca_status ca_set_tuning(ca_cache* cache, int32_t seg_chunks, int32_t split_chunks,
                        int32_t phase_mask, int32_t schedule) {
  if (!cache) return fail(CA_ERR_INVALID, "ca_set_tuning: null cache");
  if (seg_chunks < -1 || seg_chunks > 64 || split_chunks < -1 || phase_mask < 0 || phase_mask > 7 ||
      schedule < -1 || schedule > 4)
    return fail(CA_ERR_INVALID, "ca_set_tuning: value out of range");
  bool rebuild = false;
  if (seg_chunks == -1) seg_chunks = 0;  // automatic
  else if (seg_chunks == 0) seg_chunks = cache->seg_chunks;
  if (seg_chunks != cache->seg_chunks) {
    cache->seg_chunks = seg_chunks;
    rebuild = true;
  }
  if (schedule >= 0 && schedule != cache->schedule) {
    cache->schedule = schedule;
    rebuild = true;
  }
  if (split_chunks >= 0 && split_chunks != cache->split_chunks) {
    cache->split_chunks = split_chunks;
    rebuild = true;
  }
  if (phase_mask > 0) cache->phase_mask = phase_mask;
  if (rebuild) cache->work_valid = false;
  return CA_OK;
}

ca_status ca_stats(const ca_cache* cache, int64_t* uploads, int64_t* slots_used,
                   int64_t* slots_total, int32_t* schedule, int32_t* seg_chunks,
                   int64_t* patches) try {
  if (!cache) return fail(CA_ERR_INVALID, "ca_stats: null cache");
  if (!cache->patch_error.empty()) return fail(CA_ERR_INVALID, cache->patch_error);
  if (patches) *patches = cache->patches;
  if (uploads) *uploads = cache->uploads;
  if (slots_used) *slots_used = cache->tree.pool().in_use();
  if (slots_total) *slots_total = cache->tree.pool().capacity();
  if (schedule) *schedule = cache->schedule;
  if (seg_chunks) {
    ca_cache* c = const_cast<ca_cache*>(cache);
    c->ensure_work();
    *seg_chunks = c->work.seg_chunks;
  }
  return CA_OK;
} catch (...) {
  return on_exception("ca_stats");
}

}  // extern "C"
