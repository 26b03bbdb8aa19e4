// Plain types and integer mappings shared by the planner and the attention kernels: no
// matrix or memory intrinsics, so the planner can also be compiled for the host (the
// tests run it there against out-of-range and overflowing grouping arrays).
#pragma once
#include <hip/hip_runtime.h>

namespace pg {

// Tile descriptor produced by the planner.
//  q tiles : kind 0 = prefix query rows [row0,row1) of group `group` (packed prefix index);
//            kind 1 = response query rows [row0,row1) (packed suffix index), which may span
//                     several members of the group; aux = first response key any row sees
//                     (start of the member that owns row0).
//  kv tiles: kind 0 = prefix keys [row0,row1); kind 1 = response keys [row0,row1);
//            aux = end of the response rows that can see them (end of the member owning row1-1).
struct TileDesc {
  int kind, group, row0, row1, aux, work, chunk, nchunks;
};

// ---------------------------------------------------------------- XCD-aware block order
// MI355X has 8 XCDs with a private L2 each, and workgroup ids are handed to them
// round-robin (id % 8). Grids are ordered so that the workgroups that read the same
// key/value head run on the same XCD: with `units` work units (tiles, longest first)
// and `heads` heads per unit, of which `per_kv` consecutive heads share a kv head,
// block b of xcd = b % 8 takes the j-th (b / 8) slot of that XCD. When the number of
// kv heads is a multiple of 8, XCD x owns kv heads x, x+8, ...; when it divides 8,
// each kv head is spread over 8 / n_kv XCDs. Otherwise the plain order is used.
// Slots past the end map to unit >= units (the block exits).
constexpr int kXcds = 8;

struct BlockSlot {
  int unit, head;
};

__host__ __device__ inline long xcd_grid_blocks(long units, int heads, int per_kv) {
  const int n_kv = heads / per_kv;
  if (n_kv % kXcds == 0) return units * heads;
  if (kXcds % n_kv == 0) {
    const long x = kXcds / n_kv;
    return kXcds * ((units * per_kv + x - 1) / x);
  }
  return units * heads;
}

__device__ __forceinline__ BlockSlot xcd_slot(int b, int heads, int per_kv) {
  const int n_kv = heads / per_kv;
  BlockSlot s;
  if (n_kv % kXcds == 0) {
    const int xcd = b % kXcds, j = b / kXcds;
    const int per_xcd = heads / kXcds;  // heads owned by one XCD
    s.unit = j / per_xcd;
    const int sub = j % per_xcd;
    const int kv = xcd + kXcds * (sub / per_kv);
    s.head = kv * per_kv + sub % per_kv;
  } else if (kXcds % n_kv == 0) {
    const int xcd = b % kXcds, j = b / kXcds;
    const int x = kXcds / n_kv;
    const int kv = xcd % n_kv, part = xcd / n_kv;
    const int p = j * x + part;
    s.unit = p / per_kv;
    s.head = kv * per_kv + p % per_kv;
  } else {
    s.unit = b / heads;
    s.head = b % heads;
  }
  return s;
}

}  // namespace pg
