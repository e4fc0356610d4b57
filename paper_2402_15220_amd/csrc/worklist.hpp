// Work-list records shared by the host flattener and the HIP kernels. Plain
// int32 structs so they can be copied to the device as a byte blob.
#pragma once

#include <cstdint>

namespace ca {

// A chunk-first segment: n_chunks (<= 64) consecutive shared chunks of one
// run (slots at seg_slots[slot_off ...], root -> leaf) covering query rows
// [row_begin, row_end). Partial for row r is part_base + r - row_begin.
// Segment i's slots start at slot_off = i * kSegSlotStride (padded with its
// last slot), so a block can request them from its segment index alone,
// without waiting for the record.
constexpr int kSegSlotStride = 64;
struct CfSeg {
  int32_t slot_off;
  int32_t n_chunks;
  int32_t row_begin;
  int32_t row_end;
  int32_t part_base;
  int32_t pad0, pad1, pad2;
};

// A sequence-first item: row `row`, private chunks priv_slot[cb, ce).
// out_part < 0: the item owns the row's result; it merges the row's segment
// partials and writes o. Otherwise it writes partial out_part. The record
// also carries what the item's block would otherwise fetch through chains
// of dependent loads: the row's partial list parts[part_b, part_e) and the
// slots of its first kSfInline private chunks (slot[i] = priv_slot[cb + i]
// for i < n_inline = min(ce - cb, kSfInline)).
constexpr int kSfInline = 8;
struct SfItem {
  int32_t row;
  int32_t cb;
  int32_t ce;
  int32_t out_part;
  int32_t part_b;
  int32_t part_e;
  int32_t n_inline;
  int32_t pad;
  int32_t slot[kSfInline];
};

static_assert(sizeof(CfSeg) == 32, "CfSeg layout");
static_assert(sizeof(SfItem) == 64, "SfItem layout");

}  // namespace ca
