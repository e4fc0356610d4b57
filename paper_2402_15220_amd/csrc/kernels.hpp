// Launch interface of the gfx950 kernels (host side).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "tree.hpp"
#include "worklist.hpp"

namespace ca {

// Device views of the work lists (pointers into one uploaded blob).
struct DevWork {
  const CfSeg* segs = nullptr;
  const int32_t* seg_slots = nullptr;
  int32_t n_segs = 0;
  int32_t max_seg_rows = 0;
  const SfItem* items = nullptr;
  int32_t n_items = 0;
  const int32_t* priv_slot = nullptr;
  const int32_t* part_ptr = nullptr;
  const int32_t* parts = nullptr;
  const int32_t* mg_rows = nullptr;
  int32_t n_mg = 0;
  int schedule = 0;  // 0 sequential, 1 fused + merge epilogue, 2 fused + in-kernel merge,
                     // 3 concurrent streams + in-kernel merge, 4 serial reduction
  // schedule 4: host array, segments [seg_group_ptr[g], seg_group_ptr[g+1])
  // form the g-th chunk-first launch
  const int32_t* seg_group_ptr = nullptr;
  int32_t n_seg_groups = 0;
};

// Second stream and events for the concurrent schedule (default priority).
struct SideStream {
  hipStream_t stream = nullptr;
  hipEvent_t fork = nullptr;
  hipEvent_t join = nullptr;
};

struct AttnArgs {
  int dtype;  // 0 fp16, 1 fp32
  int H, D, C;
  const void* q;
  void* o;
  const void* kpool;
  const void* vpool;
  int64_t ss, hs;  // pool strides of a slot and of a head (elements)
  const int32_t* slot_len;
  float* ws_o;   // [n_parts][H][D]
  float* ws_ml;  // [n_parts][H][2] (running max in log2 units, sum)
  uint32_t ws_o_bytes;  // bytes of the ws_o region (below 4 GiB)
  float qscale;  // softmax scale * log2(e)
  int32_t* cnt;  // [B][H] arrival counters, zero between launches
  const int32_t* row_map = nullptr;  // [B] tree row -> row of q and o (null: tree order)
};

// Enqueue the attention kernels. `phase_mask` selects phases (bit 0
// chunk-first, bit 1 sequence-first, bit 2 merge). In the fused and
// concurrent schedules bits 0 and 1 together also finish every row.
hipError_t launch_attention(const AttnArgs& a, const DevWork& w, hipStream_t stream,
                            int phase_mask, const SideStream& side);

// Causal prefill attention of a sequence's last n_q tokens over its path
// (fp16 only). A path of at most kPrefillInlineChunks chunks is passed from
// host_path (slots, then starts) inside the kernel arguments; a longer one
// through the device arrays chunk_slot/chunk_start.
constexpr int kPrefillInlineChunks = 255;
struct PrefillArgs {
  int H, D, C;
  const void* q;
  void* o;
  const void* kpool;
  const void* vpool;
  int64_t ss, hs;              // pool strides of a slot and of a head (elements)
  const int32_t* host_path;    // host [n_chunks] slots then [n_chunks + 1] starts, or null
  const int32_t* chunk_slot;   // device [n_chunks] (paths longer than the inline limit)
  const int32_t* chunk_start;  // device [n_chunks + 1]
  int n_chunks;
  int n_q;
  float qscale;  // softmax scale * log2(e)
  // Key-range split of each (64-query tile, head): n_split parts in separate
  // blocks; for n_split > 1, ws holds tiles * n_split partials of
  // prefill_part_bytes(D) each and cnt one zeroed counter per tile
  // (tiles = ceil(n_q / 64) * H); the kernel leaves the counters at zero.
  int n_split = 1;
  float* ws = nullptr;
  size_t ws_bytes = 0;  // bytes of ws the launch may touch (below 4 GiB)
  int32_t* cnt = nullptr;
};
constexpr size_t prefill_part_bytes(int D) { return (64 * static_cast<size_t>(D) + 128) * 4; }
hipError_t launch_prefill(const PrefillArgs& a, hipStream_t stream);

// Device scratch of ca_attention_noalloc (scratch.hip): kScratchBytes per
// GPU; the first kScratchCounterBytes hold arrival counters, the rest the
// partial results. scratch_address() returns the current device's copy
// (hipGetSymbolAddress, taken once per device).
constexpr size_t kScratchBytes = size_t(16) << 20;
constexpr size_t kScratchCounterBytes = size_t(256) << 10;
hipError_t scratch_address(char** out);

// p[0 .. n) = value on `stream` (a kernel, not a memset node).
hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t value, hipStream_t stream);

// K/V row copies for tree operations (at most kKvJobsPerLaunch per call).
constexpr int kKvJobsPerLaunch = 64;
hipError_t launch_kv_jobs(const KvJob* jobs, int n, int dtype, int H, int D, int C, int64_t ss,
                          int64_t hs, const void* k, const void* v, void* kpool, void* vpool,
                          int32_t* slot_len, hipStream_t stream);

}  // namespace ca
