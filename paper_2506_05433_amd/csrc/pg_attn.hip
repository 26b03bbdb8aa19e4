// C ABI of the grouped-attention library (declared in include/pg_attn.h):
// host-side argument checks, workspace layout, and the launch sequence.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/pg_attn.h"
#include "pg_bwd.hpp"
#include "pg_fwd.hpp"
#include "pg_plan.hpp"
#include "pg_last.hpp"
#include "pg_rope.hpp"

// Scratch of pg_attn_fwd_noalloc: the tile plan that pg_attn_fwd keeps in the caller's
// workspace. Every device the library runs on holds its own copy until the process ends.
// In host code `scratch` only names the symbol; its device address comes from
// hipGetSymbolAddress, once per device (scratch_ptr below).
__device__ __align__(256) char scratch[PG_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

long ceil_div_l(long a, long b) { return (a + b - 1) / b; }

// Workspace layout shared by the forward and backward calls.
struct Layout {
  size_t hdr, ginfo, qoff, kvoff, qtiles, qorder, kvtiles, kvorder, seg, dsum, part, xrow, total;
  long max_q, max_kv;
  int kv_chunks, split;
};

// Pieces each prefix key tile's query walk is split into for the dK/dV kernel: enough
// workgroups to balance the long prefix walks over the CUs (about 512 prefix pieces, i.e.
// two per CU), at most 8, and 1 when there are already that many prefix key tiles. More
// pieces balance better but each adds a full fp32 partial to write and reduce; measured on
// the single-group and large-group workloads, 512 beats 256 and 1024-4096. A piece keeps at
// least 16 64-row query tiles of the average walk (a group's rows, once per query head of
// the kv head): shorter pieces cost more in their fixed start-up and in the reduce launch
// than they save. A grid of at most 128 key tiles (half the CUs) runs as long as its
// longest walk whatever the total work, so there pieces of one such tile pay off.
int kv_chunks_for(int ng, int tp, int ts, int h_q, int h_kv) {
  if (tp <= 0 || h_kv <= 0) return 1;
  const long tiles = (ceil_div_l(tp, pg::kKvBN) + ng) * (long)h_kv;
  long c = ceil_div_l(512, tiles);
  const long walk = ceil_div_l((long)tp + ts, (long)(ng > 0 ? ng : 1) * 64) * (h_q / h_kv);
  const long min_piece = 2 * tiles <= 256 ? 1 : 16;
  if (c > walk / min_piece) c = walk / min_piece;
  return (int)(c < 1 ? 1 : (c > 8 ? 8 : c));
}

// Problems whose stacked query tiles x heads cannot fill the 256 CUs tile each member's
// responses on their own (see response_tiles in the planner): their time is the longest
// tile walk, not the total work.
constexpr long kSplitBelow = 256;

Layout make_layout(int ng, int ns, int tp, int ts, int h_q, int h_kv, int d, bool bwd) {
  Layout L{};
  L.kv_chunks = bwd ? kv_chunks_for(ng, tp, ts, h_q, h_kv) : 1;
  L.split = (ceil_div_l(tp, pg::kFwdBM) + ceil_div_l(ts, pg::kFwdBM) + ng) * (long)h_q < kSplitBelow ? 1 : 0;
  // bounds of the tile lists in either tiling (splitting adds at most one tile per member)
  L.max_q = ceil_div_l(tp, pg::kFwdBM) + ceil_div_l(ts, pg::kFwdBM) + 2L * ng + ns;
  L.max_kv = bwd ? (ceil_div_l(tp, pg::kKvBN) + ng) * L.kv_chunks + ceil_div_l(ts, pg::kKvBN) + ng + ns : 0;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += align_up(bytes); return o; };
  const size_t rows = (size_t)tp + (size_t)ts;  // sizes are non-negative ints: no overflow in 64 bits
  L.hdr = take(sizeof(pg::PlanHeader));
  L.ginfo = take(sizeof(pg::GroupInfoEx) * (size_t)(ng > 0 ? ng : 1));
  L.qoff = take(sizeof(int) * ((size_t)ng + 1));
  L.kvoff = take(sizeof(int) * ((size_t)ng + 1));
  L.qtiles = take(sizeof(pg::TileDesc) * (size_t)(L.max_q > 0 ? L.max_q : 1));
  L.qorder = take(sizeof(int) * (size_t)(L.max_q > 0 ? L.max_q : 1));
  L.kvtiles = take(sizeof(pg::TileDesc) * (size_t)(L.max_kv > 0 ? L.max_kv : 1));
  L.kvorder = take(sizeof(int) * (size_t)(L.max_kv > 0 ? L.max_kv : 1));
  L.seg = take(sizeof(int) * (size_t)(ts > 0 ? ts : 1));
  L.dsum = bwd ? take(sizeof(float) * (size_t)h_q * (rows > 0 ? rows : 1)) : off;
  L.part = (bwd && L.kv_chunks > 1) ? take(sizeof(float) * (size_t)L.kv_chunks * 2 * (size_t)tp * h_kv * d) : off;
  L.xrow = bwd ? take(sizeof(int) * (rows > 0 ? rows : 1)) : off;
  L.total = off;
  return L;
}


// ---------------------------------------------------------------- kernel timing
// Optional HIP-event brackets around each launch, recorded on the launch's own
// stream. Off unless pg_timing_start() was called.
namespace timing {
constexpr int kCap = 16384;
struct Rec {
  int kernel;
  hipEvent_t a, b;
};
std::mutex mu;
bool on = false;
int n = 0;
thread_local bool suppressed = false;  // set by calls that must not create events
std::vector<Rec> recs;

int begin(int kernel, hipStream_t st) {
  if (suppressed) return -1;
  std::lock_guard<std::mutex> g(mu);
  if (!on || n >= kCap) return -1;
  if ((int)recs.size() <= n) {
    Rec r{kernel, nullptr, nullptr};
    if (hipEventCreate(&r.a) != hipSuccess || hipEventCreate(&r.b) != hipSuccess) return -1;
    recs.push_back(r);
  }
  recs[n].kernel = kernel;
  if (hipEventRecord(recs[n].a, st) != hipSuccess) return -1;
  return n++;
}

void end(int idx, hipStream_t st) {
  if (idx < 0) return;
  std::lock_guard<std::mutex> g(mu);
  (void)hipEventRecord(recs[idx].b, st);
}
}  // namespace timing

struct Timed {
  int idx;
  hipStream_t st;
  Timed(int kernel, hipStream_t s) : idx(timing::begin(kernel, s)), st(s) {}
  ~Timed() { timing::end(idx, st); }
};

struct Common {
  int dtype, ng, ns, tp, ts, h_q, h_kv, d;
  float scale;
};

int check_common(const Common& c, const int32_t* cu_p, const int32_t* cu_s, const int32_t* gsz) {
  if (c.dtype != PG_BF16 && c.dtype != PG_FP32) return fail(PG_EUNSUPPORTED, "dtype %d is not PG_BF16 or PG_FP32", c.dtype);
  if (c.ng < 0 || c.ns < 0 || c.tp < 0 || c.ts < 0)
    return fail(PG_EINVAL, "negative size (n_groups=%d n_suffixes=%d total_prefix=%d total_suffix=%d)", c.ng, c.ns,
                c.tp, c.ts);
  if (c.ng == 0 && (c.tp != 0 || c.ns != 0)) return fail(PG_EINVAL, "no groups but nonzero prefix rows or members");
  if (c.ns == 0 && c.ts != 0) return fail(PG_EINVAL, "no members but nonzero total_suffix");
  if (c.h_q <= 0 || c.h_kv <= 0 || c.h_q % c.h_kv != 0)
    return fail(PG_EINVAL, "h_q=%d must be a positive multiple of h_kv=%d", c.h_q, c.h_kv);
  if (c.d != 64 && c.d != 128) return fail(PG_EUNSUPPORTED, "head_dim=%d (supported: 64, 128)", c.d);
  // a staged tile's byte range (at most 128 rows of h * head_dim fp32) must stay below 2^31
  if ((long)c.h_q * c.d > 65536) return fail(PG_EUNSUPPORTED, "h_q*head_dim=%ld exceeds 65536", (long)c.h_q * c.d);
  if (!(std::isfinite(c.scale) && c.scale > 0.f)) return fail(PG_EINVAL, "softmax_scale must be finite and > 0");
  const long rows = (long)c.tp + c.ts;
  if (rows * c.h_q > 0x7fffffffL || (long)c.tp * c.h_q * c.d > (1L << 40))
    return fail(PG_EUNSUPPORTED, "problem too large for 32-bit row*head indexing");
  if (c.ng > 0 && (!cu_p || !gsz)) return fail(PG_EINVAL, "cu_prefix_lens/group_sizes is NULL");
  if (c.ns > 0 && !cu_s) return fail(PG_EINVAL, "cu_suffix_lens is NULL");
  if (c.ng > 0 && !cu_s) return fail(PG_EINVAL, "cu_suffix_lens is NULL");
  return PG_OK;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(PG_EHIP, "%s: %s", what, hipGetErrorString(e));
}

int device_ready() {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  return PG_OK;
}

// Device address of `scratch` on the current device, looked up on the device's first call.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(PG_EUNSUPPORTED, "device id %d (at most %d devices)", dev, kMaxDevices);
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(PG_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return PG_OK;
}

bool debug_validate() {
  const char* v = getenv("PG_DEBUG_VALIDATE");
  return v && v[0] == '1';
}

// PG_PLAN_MULTI=1 runs the multi-kernel planner even where the one-block planner applies
// (the two must give the same plan; a test compares them).
bool plan_multi() {
  const char* v = getenv("PG_PLAN_MULTI");
  return v && v[0] == '1';
}

// Launch check after the planner, and the PG_DEBUG_VALIDATE readback of its verdict.
int finish_plan(const pg::PlanHeader* hdr, hipStream_t st) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "planner launch");
  if (debug_validate()) {
    pg::PlanHeader h;
    e = hipMemcpyAsync(&h, hdr, sizeof(h), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "PG_DEBUG_VALIDATE readback");
    if (h.error) return fail(PG_EINVAL, "grouping arrays are inconsistent (checked on the device)");
  }
  return PG_OK;
}

void launch_plan_tiles(const Common& c, const Layout& L, char* ws, const int32_t* cu_p, const int32_t* cu_s,
                       const int32_t* gsz, hipStream_t st, bool bwd);

constexpr int kFusedSegRows = 8192;

// Runs the planner kernels. `bwd` also builds the key/value tile list.
int launch_plan(const Common& c, const Layout& L, char* ws, const int32_t* cu_p, const int32_t* cu_s,
                const int32_t* gsz, hipStream_t st, bool bwd, bool xl) {
  Timed tm(PG_K_PLAN, st);
  auto* hdr = (pg::PlanHeader*)(ws + L.hdr);
  auto* gi = (pg::GroupInfoEx*)(ws + L.ginfo);
  int* qoff = (int*)(ws + L.qoff);
  int* kvoff = (int*)(ws + L.kvoff);
  auto* qt = (pg::TileDesc*)(ws + L.qtiles);
  int* qo = (int*)(ws + L.qorder);
  // the one-block planner also fills the per-row member starts when there are few rows (one
  // launch less; over many rows one block is slower than the wide kernel)
  const bool one_block = L.max_q <= pg::kPlanThreads && (!bwd || L.max_kv <= pg::kPlanThreads) && !plan_multi();
  const bool fused_seg = one_block && c.ts <= kFusedSegRows;
  if (one_block) {
    // every tile list fits one block: groups, tiles and ranks in one launch
    hipLaunchKernelGGL(pg::plan_fused_kernel, dim3(1), dim3(pg::kPlanThreads), 0, st, cu_p, cu_s, gsz, c.ng, c.ns,
                       c.tp, c.ts, pg::kFwdBM, pg::kKvBN, L.kv_chunks, L.split, L.max_q,
                       bwd ? L.max_kv : 0x7fffffffL, hdr, gi, qoff, kvoff, qt, qo,
                       bwd ? (pg::TileDesc*)(ws + L.kvtiles) : nullptr, (int*)(ws + L.kvorder),
                       fused_seg ? (int*)(ws + L.seg) : nullptr);
  } else {
    launch_plan_tiles(c, L, ws, cu_p, cu_s, gsz, st, bwd);
  }
  if (c.ts > 0 && !fused_seg) {
    hipLaunchKernelGGL(pg::seg_start_kernel, dim3((unsigned)ceil_div_l(c.ts, 256)), dim3(256), 0, st, cu_s, c.ns,
                       c.ts, hdr, (int*)(ws + L.seg));
  }
  if (bwd && xl && c.tp + c.ts > 0) {
    hipLaunchKernelGGL(pg::xrow_kernel, dim3((unsigned)ceil_div_l((long)c.tp + c.ts, 256)), dim3(256), 0, st, cu_p,
                       cu_s, c.ng, c.ns, c.tp, c.ts, hdr, gi, (int*)(ws + L.xrow));
  }
  return finish_plan(hdr, st);
}

// The multi-kernel planner: groups, then tiles and ranks of each list.
void launch_plan_tiles(const Common& c, const Layout& L, char* ws, const int32_t* cu_p, const int32_t* cu_s,
                       const int32_t* gsz, hipStream_t st, bool bwd) {
  auto* hdr = (pg::PlanHeader*)(ws + L.hdr);
  auto* gi = (pg::GroupInfoEx*)(ws + L.ginfo);
  int* qoff = (int*)(ws + L.qoff);
  int* kvoff = (int*)(ws + L.kvoff);
  hipLaunchKernelGGL(pg::plan_groups_kernel, dim3(1), dim3(pg::kPlanThreads), 0, st, cu_p, cu_s, gsz, c.ng, c.ns,
                     c.tp, c.ts, pg::kFwdBM, pg::kKvBN, L.kv_chunks, L.split, L.max_q, bwd ? L.max_kv : 0x7fffffffL,
                     hdr, gi, qoff, kvoff);
  auto* qt = (pg::TileDesc*)(ws + L.qtiles);
  int* qo = (int*)(ws + L.qorder);
  if (L.max_q > 0) {
    const int blocks = (int)ceil_div_l(L.max_q, 256);
    hipLaunchKernelGGL(pg::plan_tiles_kernel, dim3(blocks), dim3(256), 0, st, cu_s, c.ng, pg::kFwdBM, pg::kKvBN,
                       1, L.split, (int)L.max_q, hdr, gi, qoff, qt, 0);
    hipLaunchKernelGGL(pg::plan_rank_kernel, dim3(blocks), dim3(256), 0, st, hdr, qt, qo, 0);
  }
  if (bwd && L.max_kv > 0) {
    auto* kt = (pg::TileDesc*)(ws + L.kvtiles);
    int* ko = (int*)(ws + L.kvorder);
    const int blocks = (int)ceil_div_l(L.max_kv, 256);
    hipLaunchKernelGGL(pg::plan_tiles_kernel, dim3(blocks), dim3(256), 0, st, cu_s, c.ng, pg::kFwdBM, pg::kKvBN,
                       L.kv_chunks, L.split, (int)L.max_kv, hdr, gi, kvoff, kt, 1);
    hipLaunchKernelGGL(pg::plan_rank_kernel, dim3(blocks), dim3(256), 0, st, hdr, kt, ko, 1);
  }
}

template <typename T, int D>
void launch_fwd(const pg::FwdArgs& a, long max_q, hipStream_t st) {
  const long blocks = pg::xcd_grid_blocks(max_q, a.h_q, a.h_q / a.h_kv);
  Timed tm(PG_K_FWD, st);
  if (blocks > 0) hipLaunchKernelGGL((pg::fwd_kernel<T, D>), dim3((unsigned)blocks), dim3(pg::kFwdThreads), 0, st, a);
}

template <typename T, int D>
void launch_bwd(const pg::BwdArgs& a, long max_q, long max_kv, hipStream_t st) {
  // dQ first: it also writes Dsum, which the dK/dV kernel reads
  if (max_q > 0) {
    Timed tm(PG_K_DQ, st);
    const long blocks = pg::xcd_grid_blocks(max_q, a.h_q, a.h_q / a.h_kv);
    hipLaunchKernelGGL((pg::dq_kernel<T, D>), dim3((unsigned)blocks), dim3(pg::kDqThreads), 0, st, a);
  }
  if (max_kv > 0) {
    {
      Timed tm(PG_K_DKDV, st);
      const long blocks = pg::xcd_grid_blocks(max_kv, a.h_kv, 1);
      hipLaunchKernelGGL((pg::dkdv_kernel<T, D>), dim3((unsigned)blocks), dim3(pg::kKvThreads), 0, st, a);
    }
    if (a.kv_chunks > 1 && a.total_prefix > 0) {
      Timed tm(PG_K_KV_REDUCE, st);
      const long n = 2L * a.total_prefix * a.h_kv * D / 4;
      hipLaunchKernelGGL((pg::kv_reduce_kernel<T, D>), dim3((unsigned)ceil_div_l(n, 256)), dim3(256), 0, st, a);
    }
  }
}



// The calls' bodies after argument checks; xl selects the single-buffer layout of Eq. (2)
// (the caller then passes the same buffer for the prefix and response sides).
int fwd_impl(const Common& c, const int32_t* cu_p, const int32_t* cu_s, const int32_t* gsz, const void* q_pre,
             const void* k_pre, const void* v_pre, const void* q_suf, const void* k_suf, const void* v_suf,
             void* o_pre, void* o_suf, float* lse_pre, float* lse_suf, bool xl, void* workspace,
             size_t workspace_bytes, void* stream) {
  const Layout L = make_layout(c.ng, c.ns, c.tp, c.ts, c.h_q, c.h_kv, c.d, false);
  if (!workspace || workspace_bytes < L.total)
    return fail(PG_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace_bytes, L.total);
  int rc = device_ready();
  if (rc) return rc;
  if (c.ng == 0) return PG_OK;
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  if ((rc = launch_plan(c, L, ws, cu_p, cu_s, gsz, st, false, xl))) return rc;
  pg::FwdArgs a{};
  a.q_pre = q_pre; a.k_pre = k_pre; a.v_pre = v_pre; a.q_suf = q_suf; a.k_suf = k_suf; a.v_suf = v_suf;
  a.o_pre = o_pre; a.o_suf = o_suf; a.lse_pre = lse_pre; a.lse_suf = lse_suf;
  a.hdr = (const pg::PlanHeader*)(ws + L.hdr);
  a.ginfo = (const pg::GroupInfoEx*)(ws + L.ginfo);
  a.qtiles = (const pg::TileDesc*)(ws + L.qtiles);
  a.qorder = (const int*)(ws + L.qorder);
  a.seg_start = (const int*)(ws + L.seg);
  a.h_q = c.h_q; a.h_kv = c.h_kv; a.total_prefix = c.tp; a.total_suffix = c.ts;
  a.scale_log2 = c.scale * pg::kLog2e;
  a.xl = xl ? 1 : 0;
  if (c.dtype == PG_BF16) {
    if (c.d == 128) launch_fwd<pg::bf16, 128>(a, L.max_q, st); else launch_fwd<pg::bf16, 64>(a, L.max_q, st);
  } else {
    if (c.d == 128) launch_fwd<float, 128>(a, L.max_q, st); else launch_fwd<float, 64>(a, L.max_q, st);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "forward launch");
  return PG_OK;
}

// in: q_pre, k_pre, v_pre, q_suf, k_suf, v_suf, o_pre, o_suf, lse_pre, lse_suf, do_pre, do_suf;
// out: dq_pre, dk_pre, dv_pre, dq_suf, dk_suf, dv_suf.
int bwd_impl(const Common& c, const int32_t* cu_p, const int32_t* cu_s, const int32_t* gsz, const void* const* in,
             void* const* out, bool xl, void* workspace, size_t workspace_bytes, void* stream) {
  const Layout L = make_layout(c.ng, c.ns, c.tp, c.ts, c.h_q, c.h_kv, c.d, true);
  if (!workspace || workspace_bytes < L.total)
    return fail(PG_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace_bytes, L.total);
  int rc = device_ready();
  if (rc) return rc;
  if (c.ng == 0) return PG_OK;
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  if ((rc = launch_plan(c, L, ws, cu_p, cu_s, gsz, st, true, xl))) return rc;
  pg::BwdArgs a{};
  a.q_pre = in[0]; a.k_pre = in[1]; a.v_pre = in[2]; a.q_suf = in[3]; a.k_suf = in[4]; a.v_suf = in[5];
  a.o_pre = in[6]; a.o_suf = in[7]; a.lse_pre = (const float*)in[8]; a.lse_suf = (const float*)in[9];
  a.do_pre = in[10]; a.do_suf = in[11];
  a.dq_pre = out[0]; a.dk_pre = out[1]; a.dv_pre = out[2]; a.dq_suf = out[3]; a.dk_suf = out[4]; a.dv_suf = out[5];
  a.dsum = (float*)(ws + L.dsum);
  a.part = (float*)(ws + L.part);
  a.kv_chunks = L.kv_chunks;
  a.hdr = (const pg::PlanHeader*)(ws + L.hdr);
  a.ginfo = (const pg::GroupInfoEx*)(ws + L.ginfo);
  a.qtiles = (const pg::TileDesc*)(ws + L.qtiles);
  a.qorder = (const int*)(ws + L.qorder);
  a.kvtiles = (const pg::TileDesc*)(ws + L.kvtiles);
  a.kvorder = (const int*)(ws + L.kvorder);
  a.seg_start = (const int*)(ws + L.seg);
  a.h_q = c.h_q; a.h_kv = c.h_kv; a.total_prefix = c.tp; a.total_suffix = c.ts;
  a.scale = c.scale;
  a.scale_log2 = c.scale * pg::kLog2e;
  a.xl = xl ? 1 : 0;
  a.xrow = (const int*)(ws + L.xrow);
  if (c.dtype == PG_BF16) {
    if (c.d == 128) launch_bwd<pg::bf16, 128>(a, L.max_q, L.max_kv, st);
    else launch_bwd<pg::bf16, 64>(a, L.max_q, L.max_kv, st);
  } else {
    if (c.d == 128) launch_bwd<float, 128>(a, L.max_q, L.max_kv, st);
    else launch_bwd<float, 64>(a, L.max_q, L.max_kv, st);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "backward launch");
  return PG_OK;
}


// ---------------------------------------------------------------- final-token forward
struct LastLayout {
  size_t hdr, ginfo, qoff, kvoff, blocks, nblk, part_o, part_ml, total;
  int mpw, nb_max, nch;
};

LastLayout last_layout(int ng, int ns, int h_q, int h_kv, int d) {
  LastLayout L{};
  const int ratio = (h_kv > 0 && h_q >= h_kv) ? h_q / h_kv : 1;
  L.mpw = ratio <= pg::kLastRows ? pg::kLastRows / ratio : 1;
  L.nb_max = (int)std::min<long>(ns, ceil_div_l(ns, L.mpw) + ng);
  const long units = (long)(L.nb_max > 0 ? L.nb_max : 1) * (h_kv > 0 ? h_kv : 1);
  L.nch = (int)std::max<long>(1, std::min<long>(pg::kLastMaxChunks, ceil_div_l(1024, units)));
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += align_up(bytes); return o; };
  L.hdr = take(sizeof(pg::PlanHeader));
  L.ginfo = take(sizeof(pg::GroupInfoEx) * (size_t)(ng > 0 ? ng : 1));
  L.qoff = take(sizeof(int) * ((size_t)ng + 1));
  L.kvoff = take(sizeof(int) * ((size_t)ng + 1));
  L.blocks = take(sizeof(pg::LastBlock) * (size_t)(L.nb_max > 0 ? L.nb_max : 1));
  L.nblk = take(sizeof(int));
  const size_t slots = (size_t)(L.nb_max > 0 ? L.nb_max : 1) * (h_kv > 0 ? h_kv : 1) * L.nch * pg::kLastRows;
  L.part_o = take(sizeof(float) * slots * (size_t)(d > 0 ? d : 1));
  L.part_ml = take(sizeof(float) * slots * 2);
  L.total = off;
  return L;
}

// ---------------------------------------------------------------- rotary embedding
// Workspace of the rope / positions calls: the planner's header and per-group ranges.
struct RopeLayout {
  size_t hdr, ginfo, qoff, kvoff, total;
};

RopeLayout rope_layout(int ng) {
  RopeLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += align_up(bytes); return o; };
  L.hdr = take(sizeof(pg::PlanHeader));
  L.ginfo = take(sizeof(pg::GroupInfoEx) * (size_t)(ng > 0 ? ng : 1));
  L.qoff = take(sizeof(int) * ((size_t)ng + 1));
  L.kvoff = take(sizeof(int) * ((size_t)ng + 1));
  L.total = off;
  return L;
}

int check_grouping(int ng, int ns, int tp, int ts, const int32_t* cu_p, const int32_t* cu_s, const int32_t* gsz) {
  if (ng < 0 || ns < 0 || tp < 0 || ts < 0)
    return fail(PG_EINVAL, "negative size (n_groups=%d n_suffixes=%d total_prefix=%d total_suffix=%d)", ng, ns,
                tp, ts);
  if (ng == 0 && (tp != 0 || ns != 0)) return fail(PG_EINVAL, "no groups but nonzero prefix rows or members");
  if (ns == 0 && ts != 0) return fail(PG_EINVAL, "no members but nonzero total_suffix");
  if ((long)tp + ts > 0x7fffffffL) return fail(PG_EUNSUPPORTED, "more than 2^31-1 rows");
  if (ng > 0 && (!cu_p || !gsz || !cu_s)) return fail(PG_EINVAL, "a grouping array is NULL");
  return PG_OK;
}

// Validates the grouping arrays on the device and fills the per-group ranges the row ->
// position mapping reads (the first planner kernel of the attention calls).
int launch_rope_plan(const RopeLayout& L, char* ws, int ng, int ns, int tp, int ts, const int32_t* cu_p,
                     const int32_t* cu_s, const int32_t* gsz, hipStream_t st) {
  auto* hdr = (pg::PlanHeader*)(ws + L.hdr);
  hipLaunchKernelGGL(pg::plan_groups_kernel, dim3(1), dim3(pg::kPlanThreads), 0, st, cu_p, cu_s, gsz, ng, ns, tp,
                     ts, pg::kFwdBM, pg::kKvBN, 1, 0, 0x7fffffffL, 0x7fffffffL, hdr,
                     (pg::GroupInfoEx*)(ws + L.ginfo), (int*)(ws + L.qoff), (int*)(ws + L.kvoff));
  return finish_plan(hdr, st);
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

extern "C" {

size_t pg_attn_fwd_workspace_size(int n_groups, int n_suffixes, int total_prefix, int total_suffix, int h_q,
                                  int h_kv, int head_dim) {
  if (n_groups < 0 || n_suffixes < 0 || total_prefix < 0 || total_suffix < 0 || h_q < 0 || h_kv < 0 ||
      head_dim < 0)
    return 0;
  return make_layout(n_groups, n_suffixes, total_prefix, total_suffix, h_q, h_kv, head_dim, false).total;
}

size_t pg_attn_bwd_workspace_size(int n_groups, int n_suffixes, int total_prefix, int total_suffix, int h_q,
                                  int h_kv, int head_dim) {
  if (n_groups < 0 || n_suffixes < 0 || total_prefix < 0 || total_suffix < 0 || h_q < 0 || h_kv < 0 ||
      head_dim < 0)
    return 0;
  return make_layout(n_groups, n_suffixes, total_prefix, total_suffix, h_q, h_kv, head_dim, true).total;
}

const char* pg_status_string(int s) {
  switch (s) {
    case PG_OK: return "PG_OK";
    case PG_EINVAL: return "PG_EINVAL: invalid argument";
    case PG_EUNSUPPORTED: return "PG_EUNSUPPORTED: unsupported configuration";
    case PG_EWORKSPACE: return "PG_EWORKSPACE: workspace missing or too small";
    case PG_EHIP: return "PG_EHIP: HIP runtime error";
    default: return "unknown pg_status";
  }
}

const char* pg_last_error(void) { return g_last_error.c_str(); }

int pg_plan_status(const void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  const void* hdr = workspace;
  if (!workspace) {
    void* p = nullptr;
    const int rc = scratch_ptr(&p);
    if (rc) return rc;
    hdr = p;  // every planned call puts the plan header at offset 0
  } else if (workspace_bytes < sizeof(pg::PlanHeader)) {
    return fail(PG_EWORKSPACE, "workspace of %zu bytes cannot hold a plan header", workspace_bytes);
  }
  int err = 0;
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipMemcpyAsync(&err, hdr, sizeof(int), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "plan status readback");
  return err ? fail(PG_EINVAL, "grouping arrays are inconsistent (checked on the device)") : PG_OK;
}

int pg_attn_fwd(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                int h_q, int h_kv, int head_dim, float softmax_scale,
                const void* q_pre, const void* k_pre, const void* v_pre,
                const void* q_suf, const void* k_suf, const void* v_suf,
                void* o_pre, void* o_suf, float* lse_pre, float* lse_suf,
                void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  const Common c{dtype, n_groups, n_suffixes, total_prefix, total_suffix, h_q, h_kv, head_dim, softmax_scale};
  int rc = check_common(c, cu_prefix_lens, cu_suffix_lens, group_sizes);
  if (rc) return rc;
  if (total_prefix > 0 && (!q_pre || !k_pre || !v_pre || !o_pre || !lse_pre))
    return fail(PG_EINVAL, "a prefix tensor pointer is NULL");
  if (total_suffix > 0 && (!q_suf || !k_suf || !v_suf || !o_suf || !lse_suf))
    return fail(PG_EINVAL, "a suffix tensor pointer is NULL");
  return fwd_impl(c, cu_prefix_lens, cu_suffix_lens, group_sizes, q_pre, k_pre, v_pre, q_suf, k_suf, v_suf, o_pre,
                  o_suf, lse_pre, lse_suf, false, workspace, workspace_bytes, stream);
}

int pg_attn_fwd_noalloc(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                        const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                        int h_q, int h_kv, int head_dim, float softmax_scale,
                        const void* q_pre, const void* k_pre, const void* v_pre,
                        const void* q_suf, const void* k_suf, const void* v_suf,
                        void* o_pre, void* o_suf, float* lse_pre, float* lse_suf, void* stream) {
  g_last_error.clear();
  const Common c{dtype, n_groups, n_suffixes, total_prefix, total_suffix, h_q, h_kv, head_dim, softmax_scale};
  int rc = check_common(c, cu_prefix_lens, cu_suffix_lens, group_sizes);
  if (rc) return rc;
  if (total_prefix > 0 && (!q_pre || !k_pre || !v_pre || !o_pre || !lse_pre))
    return fail(PG_EINVAL, "a prefix tensor pointer is NULL");
  if (total_suffix > 0 && (!q_suf || !k_suf || !v_suf || !o_suf || !lse_suf))
    return fail(PG_EINVAL, "a suffix tensor pointer is NULL");
  const size_t need = make_layout(n_groups, n_suffixes, total_prefix, total_suffix, h_q, h_kv, head_dim, false).total;
  if (need > (size_t)PG_NOALLOC_SCRATCH_BYTES)
    return fail(PG_EUNSUPPORTED, "the plan needs %zu bytes of scratch, more than the %u held for pg_attn_fwd_noalloc",
                need, (unsigned)PG_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((rc = scratch_ptr(&ws))) return rc;
  // no timing brackets: they may create events
  const bool was = timing::suppressed;
  timing::suppressed = true;
  rc = fwd_impl(c, cu_prefix_lens, cu_suffix_lens, group_sizes, q_pre, k_pre, v_pre, q_suf, k_suf, v_suf, o_pre,
                o_suf, lse_pre, lse_suf, false, ws, (size_t)PG_NOALLOC_SCRATCH_BYTES, stream);
  timing::suppressed = was;
  return rc;
}

int pg_attn_fwd_xours(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                      const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                      int h_q, int h_kv, int head_dim, float softmax_scale,
                      const void* q, const void* k, const void* v, void* o, float* lse,
                      void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  const Common c{dtype, n_groups, n_suffixes, total_prefix, total_suffix, h_q, h_kv, head_dim, softmax_scale};
  int rc = check_common(c, cu_prefix_lens, cu_suffix_lens, group_sizes);
  if (rc) return rc;
  if (total_prefix + total_suffix > 0 && (!q || !k || !v || !o || !lse))
    return fail(PG_EINVAL, "a tensor pointer is NULL");
  return fwd_impl(c, cu_prefix_lens, cu_suffix_lens, group_sizes, q, k, v, q, k, v, o, o, lse, lse, true, workspace,
                  workspace_bytes, stream);
}

int pg_attn_bwd(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                int h_q, int h_kv, int head_dim, float softmax_scale,
                const void* q_pre, const void* k_pre, const void* v_pre,
                const void* q_suf, const void* k_suf, const void* v_suf,
                const void* o_pre, const void* o_suf, const float* lse_pre, const float* lse_suf,
                const void* do_pre, const void* do_suf,
                void* dq_pre, void* dk_pre, void* dv_pre,
                void* dq_suf, void* dk_suf, void* dv_suf,
                void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  const Common c{dtype, n_groups, n_suffixes, total_prefix, total_suffix, h_q, h_kv, head_dim, softmax_scale};
  int rc = check_common(c, cu_prefix_lens, cu_suffix_lens, group_sizes);
  if (rc) return rc;
  if (total_prefix > 0 && (!q_pre || !k_pre || !v_pre || !o_pre || !lse_pre || !do_pre || !dq_pre || !dk_pre ||
                           !dv_pre))
    return fail(PG_EINVAL, "a prefix tensor pointer is NULL");
  if (total_suffix > 0 && (!q_suf || !k_suf || !v_suf || !o_suf || !lse_suf || !do_suf || !dq_suf || !dk_suf ||
                           !dv_suf))
    return fail(PG_EINVAL, "a suffix tensor pointer is NULL");
  const void* in[12] = {q_pre, k_pre, v_pre, q_suf, k_suf, v_suf, o_pre, o_suf, lse_pre, lse_suf, do_pre, do_suf};
  void* out[6] = {dq_pre, dk_pre, dv_pre, dq_suf, dk_suf, dv_suf};
  return bwd_impl(c, cu_prefix_lens, cu_suffix_lens, group_sizes, in, out, false, workspace, workspace_bytes, stream);
}

int pg_attn_bwd_xours(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                      const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                      int h_q, int h_kv, int head_dim, float softmax_scale,
                      const void* q, const void* k, const void* v, const void* o, const float* lse,
                      const void* d_o, void* dq, void* dk, void* dv,
                      void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  const Common c{dtype, n_groups, n_suffixes, total_prefix, total_suffix, h_q, h_kv, head_dim, softmax_scale};
  int rc = check_common(c, cu_prefix_lens, cu_suffix_lens, group_sizes);
  if (rc) return rc;
  if (total_prefix + total_suffix > 0 && (!q || !k || !v || !o || !lse || !d_o || !dq || !dk || !dv))
    return fail(PG_EINVAL, "a tensor pointer is NULL");
  const void* in[12] = {q, k, v, q, k, v, o, o, lse, lse, d_o, d_o};
  void* out[6] = {dq, dk, dv, dq, dk, dv};
  return bwd_impl(c, cu_prefix_lens, cu_suffix_lens, group_sizes, in, out, true, workspace, workspace_bytes, stream);
}

int pg_timing_start(void) {
  std::lock_guard<std::mutex> g(timing::mu);
  timing::on = true;
  timing::n = 0;
  return PG_OK;
}

int pg_timing_stop(void) {
  std::lock_guard<std::mutex> g(timing::mu);
  timing::on = false;
  return PG_OK;
}

int pg_timing_get(int kernel, int* launches, double* total_ms) {
  if (!launches || !total_ms) return fail(PG_EINVAL, "NULL output pointer");
  std::lock_guard<std::mutex> g(timing::mu);
  int cnt = 0;
  double tot = 0.0;
  for (int i = 0; i < timing::n; ++i) {
    const timing::Rec& r = timing::recs[i];
    if (r.kernel != kernel) continue;
    hipError_t e = hipEventSynchronize(r.b);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) return hip_fail(e, "timing event");
    ++cnt;
    tot += ms;
  }
  *launches = cnt;
  *total_ms = tot;
  return PG_OK;
}

size_t pg_attn_fwd_last_workspace_size(int n_groups, int n_suffixes, int total_prefix, int total_suffix, int h_q,
                                       int h_kv, int head_dim) {
  (void)total_prefix; (void)total_suffix;
  if (n_groups < 0 || n_suffixes < 0 || total_prefix < 0 || total_suffix < 0 || h_q < 0 || h_kv < 0 ||
      head_dim < 0)
    return 0;
  return last_layout(n_groups, n_suffixes, h_q, h_kv, head_dim).total;
}

int pg_attn_fwd_last(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                     const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                     int h_q, int h_kv, int head_dim, float softmax_scale,
                     const void* q_pre, const void* k_pre, const void* v_pre,
                     const void* q_suf, const void* k_suf, const void* v_suf,
                     void* o_last, float* lse_last, void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  const Common c{dtype, n_groups, n_suffixes, total_prefix, total_suffix, h_q, h_kv, head_dim, softmax_scale};
  int rc = check_common(c, cu_prefix_lens, cu_suffix_lens, group_sizes);
  if (rc) return rc;
  if (h_q / h_kv > pg::kLastRows) return fail(PG_EUNSUPPORTED, "h_q / h_kv = %d exceeds %d", h_q / h_kv, pg::kLastRows);
  if (total_prefix > 0 && (!q_pre || !k_pre || !v_pre)) return fail(PG_EINVAL, "a prefix tensor pointer is NULL");
  if (total_suffix > 0 && (!q_suf || !k_suf || !v_suf)) return fail(PG_EINVAL, "a suffix tensor pointer is NULL");
  if (n_suffixes > 0 && (!o_last || !lse_last)) return fail(PG_EINVAL, "o_last or lse_last is NULL");
  const LastLayout L = last_layout(n_groups, n_suffixes, h_q, h_kv, head_dim);
  if (!workspace || workspace_bytes < L.total)
    return fail(PG_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace_bytes, L.total);
  if ((rc = device_ready())) return rc;
  if (n_suffixes == 0) return PG_OK;
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  pg::LastArgs a{};
  a.q_pre = q_pre; a.k_pre = k_pre; a.v_pre = v_pre; a.q_suf = q_suf; a.k_suf = k_suf; a.v_suf = v_suf;
  a.o_last = o_last; a.lse_last = lse_last;
  a.cu_s = cu_suffix_lens;
  a.hdr = (const pg::PlanHeader*)(ws + L.hdr);
  a.ginfo = (const pg::GroupInfoEx*)(ws + L.ginfo);
  a.blocks = (const pg::LastBlock*)(ws + L.blocks);
  a.n_blocks = (const int*)(ws + L.nblk);
  a.part_o = (float*)(ws + L.part_o);
  a.part_ml = (float*)(ws + L.part_ml);
  a.h_q = h_q; a.h_kv = h_kv; a.ns = n_suffixes; a.nch = L.nch; a.nb_max = L.nb_max; a.mpw = L.mpw;
  a.scale_log2 = softmax_scale * pg::kLog2e;
  {
    Timed tp(PG_K_PLAN, st);
    const RopeLayout R{L.hdr, L.ginfo, L.qoff, L.kvoff, 0};
    if ((rc = launch_rope_plan(R, ws, n_groups, n_suffixes, total_prefix, total_suffix, cu_prefix_lens,
                               cu_suffix_lens, group_sizes, st)))
      return rc;
    hipLaunchKernelGGL(pg::plan_last_kernel, dim3(1), dim3(pg::kPlanThreads), 0, st, a.hdr, a.ginfo, n_groups, L.mpw,
                       L.nb_max, (pg::LastBlock*)(ws + L.blocks), (int*)(ws + L.nblk));
  }
  const long blocks = pg::xcd_grid_blocks((long)L.nb_max * L.nch, h_kv, 1);
  const long merge = (long)(head_dim == 128 ? pg::merge_groups<128>() : pg::merge_groups<64>()) * L.nb_max * h_kv;
  if (blocks > INT32_MAX || merge > INT32_MAX)
    return fail(PG_EUNSUPPORTED, "%d responses x %d kv heads exceed the launch grid", n_suffixes, h_kv);
  const dim3 gc((unsigned)blocks), gm((unsigned)merge), tc(pg::kLastThreads), tm_(pg::kMergeThreads);
  Timed tm(PG_K_LAST, st);
  if (dtype == PG_BF16) {
    if (head_dim == 128) {
      hipLaunchKernelGGL((pg::last_kernel<pg::bf16, 128>), gc, tc, 0, st, a);
      hipLaunchKernelGGL((pg::last_merge_kernel<pg::bf16, 128>), gm, tm_, 0, st, a);
    } else {
      hipLaunchKernelGGL((pg::last_kernel<pg::bf16, 64>), gc, tc, 0, st, a);
      hipLaunchKernelGGL((pg::last_merge_kernel<pg::bf16, 64>), gm, tm_, 0, st, a);
    }
  } else {
    if (head_dim == 128) {
      hipLaunchKernelGGL((pg::last_kernel<float, 128>), gc, tc, 0, st, a);
      hipLaunchKernelGGL((pg::last_merge_kernel<float, 128>), gm, tm_, 0, st, a);
    } else {
      hipLaunchKernelGGL((pg::last_kernel<float, 64>), gc, tc, 0, st, a);
      hipLaunchKernelGGL((pg::last_merge_kernel<float, 64>), gm, tm_, 0, st, a);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "final-token forward launch");
  return PG_OK;
}

size_t pg_rope_workspace_size(int n_groups) {
  if (n_groups < 0) return 0;
  return rope_layout(n_groups).total;
}

int pg_rope(int dtype, int n_groups, int n_suffixes, int total_prefix, int total_suffix,
            const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
            int h_q, int h_kv, int head_dim, int rotary_dim, double base, int flags,
            const void* q_pre, const void* q_suf, const void* k_pre, const void* k_suf,
            void* q_pre_out, void* q_suf_out, void* k_pre_out, void* k_suf_out,
            void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  int rc = check_grouping(n_groups, n_suffixes, total_prefix, total_suffix, cu_prefix_lens, cu_suffix_lens,
                          group_sizes);
  if (rc) return rc;
  if (dtype != PG_BF16 && dtype != PG_FP32) return fail(PG_EUNSUPPORTED, "dtype %d is not PG_BF16 or PG_FP32", dtype);
  if (head_dim != 64 && head_dim != 128) return fail(PG_EUNSUPPORTED, "head_dim=%d (supported: 64, 128)", head_dim);
  if (h_q < 0 || h_kv < 0 || h_q + h_kv == 0) return fail(PG_EINVAL, "h_q=%d h_kv=%d: need h_q + h_kv > 0", h_q, h_kv);
  if ((long)(h_q + h_kv) * head_dim > 65536)
    return fail(PG_EUNSUPPORTED, "(h_q + h_kv) * head_dim exceeds 65536");
  if (rotary_dim < 16 || rotary_dim > head_dim || rotary_dim % 16 != 0)
    return fail(PG_EUNSUPPORTED, "rotary_dim=%d (a multiple of 16 in [16, head_dim=%d])", rotary_dim, head_dim);
  if (!(std::isfinite(base) && base > 0.0)) return fail(PG_EINVAL, "base must be finite and > 0");
  if (flags & ~(PG_ROPE_INVERSE | PG_ROPE_INTERLEAVED)) return fail(PG_EINVAL, "unknown flags 0x%x", flags);
  const void* ins[4] = {q_pre, q_suf, k_pre, k_suf};
  void* outs[4] = {q_pre_out, q_suf_out, k_pre_out, k_suf_out};
  for (int t = 0; t < 4; ++t) {
    const bool used = (t < 2 ? h_q : h_kv) > 0 && (t % 2 == 0 ? total_prefix : total_suffix) > 0;
    if (!used) continue;
    if (!ins[t] || !outs[t]) return fail(PG_EINVAL, "a tensor pointer is NULL");
    if (!aligned16(ins[t]) || !aligned16(outs[t])) return fail(PG_EINVAL, "tensor pointers must be 16-byte aligned");
  }
  const RopeLayout L = rope_layout(n_groups);
  if (!workspace || workspace_bytes < L.total)
    return fail(PG_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace_bytes, L.total);
  if ((rc = device_ready())) return rc;
  const int rows = total_prefix + total_suffix;
  if (rows == 0) return PG_OK;
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  pg::RopeArgs a{};
  a.cu_p = cu_prefix_lens; a.cu_s = cu_suffix_lens;
  a.hdr = (const pg::PlanHeader*)(ws + L.hdr);
  a.ginfo = (const pg::GroupInfoEx*)(ws + L.ginfo);
  a.ng = n_groups; a.ns = n_suffixes; a.tp = total_prefix; a.ts = total_suffix;
  a.h_q = h_q; a.h_kv = h_kv; a.rot = rotary_dim; a.flags = flags;
  a.log2_base = std::log2(base);
  for (int t = 0; t < 4; ++t) { a.src[t] = ins[t]; a.dst[t] = outs[t]; }
  {
    Timed tp(PG_K_PLAN, st);
    if ((rc = launch_rope_plan(L, ws, n_groups, n_suffixes, total_prefix, total_suffix, cu_prefix_lens,
                               cu_suffix_lens, group_sizes, st)))
      return rc;
  }
  const dim3 grid((unsigned)rows), block(pg::kRopeThreads);
  Timed tm(PG_K_ROPE, st);
  if (dtype == PG_BF16) {
    if (head_dim == 128) hipLaunchKernelGGL((pg::rope_kernel<pg::bf16, 128>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((pg::rope_kernel<pg::bf16, 64>), grid, block, 0, st, a);
  } else {
    if (head_dim == 128) hipLaunchKernelGGL((pg::rope_kernel<float, 128>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((pg::rope_kernel<float, 64>), grid, block, 0, st, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "rope launch");
  return PG_OK;
}

int pg_grouped_positions(int n_groups, int n_suffixes, int total_prefix, int total_suffix,
                         const int32_t* cu_prefix_lens, const int32_t* cu_suffix_lens, const int32_t* group_sizes,
                         int32_t* pos_pre, int32_t* pos_suf, void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  int rc = check_grouping(n_groups, n_suffixes, total_prefix, total_suffix, cu_prefix_lens, cu_suffix_lens,
                          group_sizes);
  if (rc) return rc;
  if ((total_prefix > 0 && !pos_pre) || (total_suffix > 0 && !pos_suf))
    return fail(PG_EINVAL, "a position array is NULL");
  const RopeLayout L = rope_layout(n_groups);
  if (!workspace || workspace_bytes < L.total)
    return fail(PG_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace_bytes, L.total);
  if ((rc = device_ready())) return rc;
  const int rows = total_prefix + total_suffix;
  if (rows == 0) return PG_OK;
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  if ((rc = launch_rope_plan(L, ws, n_groups, n_suffixes, total_prefix, total_suffix, cu_prefix_lens,
                             cu_suffix_lens, group_sizes, st)))
    return rc;
  pg::RopeArgs a{};
  a.cu_p = cu_prefix_lens; a.cu_s = cu_suffix_lens;
  a.hdr = (const pg::PlanHeader*)(ws + L.hdr);
  a.ginfo = (const pg::GroupInfoEx*)(ws + L.ginfo);
  a.ng = n_groups; a.ns = n_suffixes; a.tp = total_prefix; a.ts = total_suffix;
  a.pos_out[0] = pos_pre; a.pos_out[1] = pos_suf;
  hipLaunchKernelGGL(pg::positions_kernel, dim3((unsigned)ceil_div_l(rows, 256)), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "positions launch");
  return PG_OK;
}

}  // extern "C"
