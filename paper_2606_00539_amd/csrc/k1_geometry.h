// Geometry of K1 (the gradient pass) and its work items, shared by the
// kernel and the runtime's work-list builder.
#pragma once

#include <stdint.h>

namespace gnmr {

// K1 geometry: a workgroup of 256 lanes reads one work item of 64 KiB with
// 16 outstanding 16-byte loads per lane.
constexpr int kK1Block = 256;
constexpr int kK1Unroll = 16;
constexpr int64_t kItemBytes = int64_t(kK1Block) * kK1Unroll * 16;
// MI355X: 256 compute units in 8 XCDs, each XCD with its own L2.
constexpr uint32_t kNumXcd = 8;

// One work item: elements [e0, e0 + count) of segment `seg`.  Items are
// ordered by unit, so the items of unit b are [unit_item_off[b],
// unit_item_off[b+1]).
struct Item {
  int64_t e0;
  int32_t seg;
  int32_t count;
};
static_assert(sizeof(Item) == 16, "Item layout");

}  // namespace gnmr
