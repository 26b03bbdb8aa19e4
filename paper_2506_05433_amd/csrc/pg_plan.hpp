// Device-side planner: validates the grouping arrays and builds the tile lists
// that the attention kernels walk, ordered longest-first.
//
// Query tiles follow the two attention calls of Eq. (4): prefix query tiles
// (causal self-attention over the prefix) and response query tiles. Response
// rows of all members of a group are stacked into common tiles: every one of
// them sees the whole group prefix, so the prefix part of a tile is a dense
// rectangle regardless of member boundaries, and only the response part needs
// the per-member causal mask. Key/value tiles are the mirror image for the
// key-stationary gradient kernel.
#pragma once
#include <hip/hip_runtime.h>

#include "pg_types.hpp"

namespace pg {

struct PlanHeader {
  int error;     // nonzero when the grouping arrays are inconsistent
  int n_qtiles;  // number of query tiles
  int n_kvtiles; // number of key/value tiles
  int pad[61];
};

struct GroupInfoEx {
  int p0, p1, s0, s1, m0, m1, pad0, pad1;
};

__device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Inclusive scan of one value per thread over a block of NT threads.
template <int NT, typename V>
__device__ __forceinline__ V block_inclusive_scan(V v, V* tmp) {
  const int t = threadIdx.x;
  tmp[t] = v;
  __syncthreads();
  for (int off = 1; off < NT; off <<= 1) {
    V add = (t >= off) ? tmp[t - off] : 0;
    __syncthreads();
    tmp[t] += add;
    __syncthreads();
  }
  V r = tmp[t];
  __syncthreads();
  return r;
}

// Largest index i in [lo, hi) with a[i] <= x (a nondecreasing, a[lo] <= x).
__device__ __forceinline__ int upper_index(const int* a, int lo, int hi, int x) {
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (a[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

constexpr int kPlanThreads = 1024;

// Shared memory of the one-block planner steps.
struct PlanShared {
  int tmp[kPlanThreads];
  long long tmp64[kPlanThreads];
  long long members;  // running sum of group sizes
  int err;
  int carry[3];
};

// Response tiles of a group: its response rows stacked into b-row tiles across member
// boundaries, or (split) each member's rows tiled on their own. Stacking wastes no rows
// and lets every tile share the group's prefix; splitting gives more, shorter tiles, which
// is what a problem too small to fill the GPU needs (its time is the longest tile walk).
__device__ inline int response_tiles(const int* __restrict__ cu_s, const GroupInfoEx& gi, int b, int split) {
  if (!split) return ceil_div(gi.s1 - gi.s0, b);
  int n = 0;
  // unrolled so that several members' lengths are loaded at once (one thread walks a group's members)
#pragma unroll 4
  for (int m = gi.m0; m < gi.m1; ++m) n += ceil_div(cu_s[m + 1] - cu_s[m], b);
  return n;
}

// One block of kPlanThreads threads. Validates and computes per-group ranges and tile offsets.
__device__ inline void plan_groups_body(const int* __restrict__ cu_p, const int* __restrict__ cu_s,
                                        const int* __restrict__ gsz, int ng, int ns, int tp, int ts, int bm, int bkv,
                                        int kv_chunks, int split, long max_q, long max_kv, PlanHeader* hdr,
                                        GroupInfoEx* ginfo, int* qoff, int* kvoff, PlanShared& sh) {
  int* tmp = sh.tmp;
  int& err = sh.err;
  int* carry = sh.carry;
  const int t = threadIdx.x;
  if (t == 0) { err = 0; carry[0] = carry[1] = carry[2] = 0; sh.members = 0; }
  __syncthreads();
  int bad = 0;
  for (int g = t; g <= ng; g += kPlanThreads) {
    int v = cu_p[g];
    if (g == 0 && v != 0) bad = 1;
    if (g == ng && v != tp) bad = 1;
    if (g > 0 && v < cu_p[g - 1]) bad = 1;
    if (g < ng && (gsz[g] < 0 || gsz[g] > ns)) bad = 1;
  }
  for (int m = t; m <= ns; m += kPlanThreads) {
    int v = cu_s[m];
    if (m == 0 && v != 0) bad = 1;
    if (m == ns && v != ts) bad = 1;
    if (m > 0 && v < cu_s[m - 1]) bad = 1;
  }
  if (bad) atomicOr(&err, 1);
  __syncthreads();
  // member starts: exclusive scan of group sizes, in 64 bits so that no sum of sizes can wrap
  // around to n_suffixes; checked against it afterwards, and only then are the starts used to
  // index cu_suffix_lens
  for (int base = 0; base < ng; base += kPlanThreads) {
    const int g = base + t;
    const long long v = (g < ng && !err) ? gsz[g] : 0;
    const long long inc = block_inclusive_scan<kPlanThreads>(v, sh.tmp64);
    const long long m1 = sh.members + inc;
    if (g < ng) { ginfo[g].m0 = (int)(m1 - v); ginfo[g].m1 = (int)m1; }
    __syncthreads();
    if (t == kPlanThreads - 1) sh.members = m1;
    __syncthreads();
  }
  if (t == 0 && sh.members != ns) err = 1;
  __syncthreads();
  const int ok = !err;
  for (int base = 0; base < ng; base += kPlanThreads) {
    const int g = base + t;
    int nq = 0, nkv = 0;
    if (g < ng && ok) {
      GroupInfoEx gi = ginfo[g];
      gi.p0 = cu_p[g]; gi.p1 = cu_p[g + 1];
      gi.s0 = cu_s[gi.m0]; gi.s1 = cu_s[gi.m1];
      gi.pad0 = gi.pad1 = 0;
      ginfo[g] = gi;
      nq = ceil_div(gi.p1 - gi.p0, bm) + response_tiles(cu_s, gi, bm, split);
      nkv = ceil_div(gi.p1 - gi.p0, bkv) * kv_chunks + response_tiles(cu_s, gi, bkv, split);
    }
    const int iq = block_inclusive_scan<kPlanThreads>(nq, tmp);
    const int ikv = block_inclusive_scan<kPlanThreads>(nkv, tmp);
    if (g < ng) { qoff[g] = carry[1] + iq - nq; kvoff[g] = carry[2] + ikv - nkv; }
    __syncthreads();
    if (t == kPlanThreads - 1) { carry[1] += iq; carry[2] += ikv; }
    __syncthreads();
  }
  // the host sized the tile arrays from the totals; a list longer than that bound
  // can only come from inconsistent arrays, so it is treated as an error too
  if (t == 0 && ok && (carry[1] > max_q || carry[2] > max_kv)) err = 1;
  __syncthreads();
  if (t == 0) {
    const int ok = !err;
    qoff[ng] = ok ? carry[1] : 0;
    kvoff[ng] = ok ? carry[2] : 0;
    hdr->error = err;
    hdr->n_qtiles = ok ? carry[1] : 0;
    hdr->n_kvtiles = ok ? carry[2] : 0;
  }
}

__global__ void __launch_bounds__(kPlanThreads) plan_groups_kernel(
    const int* __restrict__ cu_p, const int* __restrict__ cu_s, const int* __restrict__ gsz,
    int ng, int ns, int tp, int ts, int bm, int bkv, int kv_chunks, int split, long max_q, long max_kv,
    PlanHeader* hdr, GroupInfoEx* ginfo, int* qoff, int* kvoff) {
  __shared__ PlanShared sh;
  plan_groups_body(cu_p, cu_s, gsz, ng, ns, tp, ts, bm, bkv, kv_chunks, split, max_q, max_kv, hdr, ginfo, qoff, kvoff,
                   sh);
}

// Descriptor of tile i (< the number of tiles). `which` 0 = query tiles, 1 = kv tiles.
// Returns the tile's work (the ranking key).
__device__ inline int plan_tile(int i, const int* __restrict__ cu_s, int ng, int bm, int bkv, int kv_chunks,
                                 int split, const GroupInfoEx* __restrict__ ginfo, const int* __restrict__ off,
                                 TileDesc* tiles, int which) {
  const int g = upper_index(off, 0, ng, i);  // off[ng] == n > i, groups with no tile share offsets
  // skip groups with zero tiles that share the offset of the next one
  const GroupInfoEx gi = ginfo[g];
  const int b = which ? bkv : bm;
  const int chunks = which ? kv_chunks : 1;
  int local = i - off[g];
  const int np = ceil_div(gi.p1 - gi.p0, b) * chunks;
  TileDesc d;
  d.group = g;
  d.chunk = 0;
  d.nchunks = 1;
  if (local < np) {
    d.kind = 0;
    d.chunk = local % chunks;
    d.nchunks = chunks;
    local /= chunks;
    d.row0 = gi.p0 + local * b;
    d.row1 = min(d.row0 + b, gi.p1);
    if (!which) {
      d.aux = 0;
      d.work = d.row1 - gi.p0;                          // keys seen by the last row
    } else {
      d.aux = 0;
      d.work = ((gi.p1 - d.row0) + (gi.s1 - gi.s0)) / chunks;  // query rows that see these keys
    }
  } else {
    d.kind = 1;
    int lo = gi.s0, hi = gi.s1;  // the rows the tile is cut from: the group's, or one member's
    local -= np;
    if (split) {
#pragma unroll 4
      for (int m = gi.m0; m < gi.m1; ++m) {
        const int t = ceil_div(cu_s[m + 1] - cu_s[m], b);
        if (local < t) {
          lo = cu_s[m];
          hi = cu_s[m + 1];
          break;
        }
        local -= t;
      }
    }
    d.row0 = lo + local * b;
    d.row1 = min(d.row0 + b, hi);
    if (!which) {
      const int m = upper_index(cu_s, gi.m0, gi.m1, d.row0);
      d.aux = cu_s[m];                                  // first response key of the tile
      d.work = (gi.p1 - gi.p0) + (d.row1 - d.aux);
    } else {
      const int m = upper_index(cu_s, gi.m0, gi.m1, d.row1 - 1);
      d.aux = cu_s[m + 1];                              // end of queries that see the keys
      d.work = d.aux - d.row0;
    }
  }
  tiles[i] = d;
  return d.work;
}

// One thread per (possible) tile: fills the descriptors.
__global__ void plan_tiles_kernel(const int* __restrict__ cu_s, int ng, int bm, int bkv, int kv_chunks, int split,
                                  int max_tiles, const PlanHeader* hdr, const GroupInfoEx* __restrict__ ginfo,
                                  const int* __restrict__ off, TileDesc* tiles, int which) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int n = which ? hdr->n_kvtiles : hdr->n_qtiles;
  if (i >= n || i >= max_tiles) return;
  plan_tile(i, cu_s, ng, bm, bkv, kv_chunks, split, ginfo, off, tiles, which);
}

// Longest-first order: order[rank] = tile, rank by (work desc, index asc). Deterministic.
__global__ void __launch_bounds__(256) plan_rank_kernel(const PlanHeader* hdr, const TileDesc* __restrict__ tiles,
                                                        int* order, int which) {
  __shared__ int w[1024];
  const int n = which ? hdr->n_kvtiles : hdr->n_qtiles;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if ((int)(blockIdx.x * blockDim.x) >= n) return;
  const int mine = i < n ? tiles[i].work : 0;
  int rank = 0;
  for (int base = 0; base < n; base += 1024) {
    __syncthreads();
    for (int k = threadIdx.x; k < 1024; k += blockDim.x) w[k] = (base + k < n) ? tiles[base + k].work : -1;
    __syncthreads();
    if (i < n) {
      const int lim = min(1024, n - base);
      for (int k = 0; k < lim; ++k) {
        const int o = w[k];
        rank += (o > mine) || (o == mine && base + k < i);
      }
    }
  }
  if (i < n) order[rank] = i;
}

// seg_start[r] = first row of the member that owns response row r.
__global__ void seg_start_kernel(const int* __restrict__ cu_s, int ns, int ts, const PlanHeader* hdr,
                                 int* seg_start) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= ts || hdr->error) return;
  seg_start[r] = cu_s[upper_index(cu_s, 0, ns, r)];
}

// Row map of the single-buffer layout of Eq. (2) (per group [P; R_1; ...; R_G], groups
// one after another): xrow[t] for packed prefix row t, xrow[total_prefix + s] for packed
// response row s. Prefix row t of group g is preceded by the responses of the earlier
// groups (s0 of g rows); response row s of group g by the prefixes of groups 0..g (p1).
__device__ inline void xrow_of(int row, const int* __restrict__ cu_p, const int* __restrict__ cu_s, int ng, int ns,
                               int tp, const GroupInfoEx* __restrict__ ginfo, int* xrow) {
  if (row < tp) {
    const int g = upper_index(cu_p, 0, ng, row);
    xrow[row] = row + ginfo[g].s0;
    return;
  }
  const int s = row - tp;
  const int m = upper_index(cu_s, 0, ns, s);
  int lo = 0, hi = ng;  // the group of member m: the last group whose members start at or before m
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (ginfo[mid].m0 <= m) lo = mid; else hi = mid;
  }
  xrow[row] = s + ginfo[lo].p1;
}

__global__ void xrow_kernel(const int* __restrict__ cu_p, const int* __restrict__ cu_s, int ng, int ns, int tp,
                            int ts, const PlanHeader* hdr, const GroupInfoEx* __restrict__ ginfo, int* xrow) {
  const int row = blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= tp + ts || hdr->error) return;
  xrow_of(row, cu_p, cu_s, ng, ns, tp, ginfo, xrow);
}

// Groups, tile descriptors and longest-first ranks in one block, for plans whose tile
// lists each fit in kPlanThreads entries (the host checks the bounds): the steps above in
// order, separated by block barriers instead of kernel boundaries, with the same results.
// Saves the launch and memory latency of two to four dependent one-block kernels per call.
// The per-row tables (seg_start_kernel, xrow_kernel) stay separate wide launches: one
// block would walk every row.
__global__ void __launch_bounds__(kPlanThreads) plan_fused_kernel(
    const int* __restrict__ cu_p, const int* __restrict__ cu_s, const int* __restrict__ gsz, int ng, int ns, int tp,
    int ts, int bm, int bkv, int kv_chunks, int split, long max_q, long max_kv, PlanHeader* hdr, GroupInfoEx* ginfo,
    int* qoff, int* kvoff, TileDesc* qtiles, int* qorder, TileDesc* kvtiles, int* kvorder, int* seg_start) {
  __shared__ PlanShared sh;
  plan_groups_body(cu_p, cu_s, gsz, ng, ns, tp, ts, bm, bkv, kv_chunks, split, max_q, max_kv, hdr, ginfo, qoff, kvoff,
                   sh);
  __syncthreads();
  const int t = threadIdx.x;
  // the tile counts the header now holds, taken from shared memory (both <= kPlanThreads, a host bound)
  const bool ok = !sh.err;
  const int nq = ok ? sh.carry[1] : 0, nkv = (kvtiles && ok) ? sh.carry[2] : 0;
  const int wq = t < nq ? plan_tile(t, cu_s, ng, bm, bkv, 1, split, ginfo, qoff, qtiles, 0) : -1;
  const int wkv = t < nkv ? plan_tile(t, cu_s, ng, bm, bkv, kv_chunks, split, ginfo, kvoff, kvtiles, 1) : -1;
  // the per-row member starts (what seg_start_kernel computes), when asked for
  if (seg_start && ok)
    for (int r = t; r < ts; r += kPlanThreads) seg_start[r] = cu_s[upper_index(cu_s, 0, ns, r)];
  // longest-first ranks, the rule of plan_rank_kernel: (work desc, index asc)
  for (int which = 0; which < 2; ++which) {
    const int n = which ? nkv : nq;
    int* order = which ? kvorder : qorder;
    sh.tmp[t] = which ? wkv : wq;
    __syncthreads();
    if (t < n) {
      const int mine = sh.tmp[t];
      int rank = 0;
      for (int k = 0; k < n; ++k) {
        const int o = sh.tmp[k];
        rank += (o > mine) || (o == mine && k < t);
      }
      order[rank] = t;
    }
    __syncthreads();
  }
}

}  // namespace pg
