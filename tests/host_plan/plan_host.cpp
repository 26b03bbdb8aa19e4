// The device planner (pg_plan.hpp) compiled for the host and run on grouping arrays read
// from stdin, so the tests can check its plans and its handling of inconsistent arrays
// under AddressSanitizer (every array is allocated at exactly the size the library's host
// code gives it, so a read past the end is reported).
//
// stdin: mode (0 = one-block planner, 1 = multi-kernel planner), ng, ns, tp, ts, bm, bkv,
//        kv_chunks, split, max_q, max_kv, then cu_prefix_lens[ng+1], cu_suffix_lens[ns+1],
//        group_sizes[ng].
// stdout: error n_qtiles n_kvtiles, then one line per query tile in rank order
//         ("q kind group row0 row1 aux work chunk nchunks"), the same for kv tiles ("k ..."),
//         then "s" followed by the per-row member starts (when the plan is valid).
#include <cstdio>
#include <memory>

#include "pg_plan.hpp"

using namespace pg;

int main() {
  int mode, ng, ns, tp, ts, bm, bkv, kvc, split;
  long max_q, max_kv;
  if (scanf("%d %d %d %d %d %d %d %d %d %ld %ld", &mode, &ng, &ns, &tp, &ts, &bm, &bkv, &kvc, &split, &max_q,
            &max_kv) != 11)
    return 2;
  std::unique_ptr<int[]> cu_p(new int[ng + 1]), cu_s(new int[ns + 1]), gsz(new int[ng > 0 ? ng : 1]);
  for (int i = 0; i <= ng; ++i) if (scanf("%d", &cu_p[i]) != 1) return 2;
  for (int i = 0; i <= ns; ++i) if (scanf("%d", &cu_s[i]) != 1) return 2;
  for (int i = 0; i < ng; ++i) if (scanf("%d", &gsz[i]) != 1) return 2;
  PlanHeader hdr{};
  std::unique_ptr<GroupInfoEx[]> gi(new GroupInfoEx[ng > 0 ? ng : 1]);
  std::unique_ptr<int[]> qoff(new int[ng + 1]), kvoff(new int[ng + 1]);
  const long nq_cap = max_q > 0 ? max_q : 1, nkv_cap = max_kv > 0 ? max_kv : 1;
  std::unique_ptr<TileDesc[]> qt(new TileDesc[nq_cap]), kt(new TileDesc[nkv_cap]);
  std::unique_ptr<int[]> qo(new int[nq_cap]), ko(new int[nkv_cap]);
  std::unique_ptr<int[]> seg(new int[ts > 0 ? ts : 1]);
  if (mode == 0) {
    host_launch(1, kPlanThreads, [&] {
      plan_fused_kernel(cu_p.get(), cu_s.get(), gsz.get(), ng, ns, tp, ts, bm, bkv, kvc, split, max_q, max_kv, &hdr,
                        gi.get(), qoff.get(), kvoff.get(), qt.get(), qo.get(), kt.get(), ko.get(), seg.get());
    });
  } else {
    host_launch(1, kPlanThreads, [&] {
      plan_groups_kernel(cu_p.get(), cu_s.get(), gsz.get(), ng, ns, tp, ts, bm, bkv, kvc, split, max_q, max_kv, &hdr,
                         gi.get(), qoff.get(), kvoff.get());
    });
    const unsigned bq = (unsigned)((max_q + 255) / 256), bk = (unsigned)((max_kv + 255) / 256);
    if (max_q > 0) {
      host_launch(bq, 256, [&] {
        plan_tiles_kernel(cu_s.get(), ng, bm, bkv, 1, split, (int)max_q, &hdr, gi.get(), qoff.get(), qt.get(), 0);
      });
      host_launch(bq, 256, [&] { plan_rank_kernel(&hdr, qt.get(), qo.get(), 0); });
    }
    if (max_kv > 0) {
      host_launch(bk, 256, [&] {
        plan_tiles_kernel(cu_s.get(), ng, bm, bkv, kvc, split, (int)max_kv, &hdr, gi.get(), kvoff.get(), kt.get(), 1);
      });
      host_launch(bk, 256, [&] { plan_rank_kernel(&hdr, kt.get(), ko.get(), 1); });
    }
  }
  if (mode == 1 && ts > 0) {
    host_launch((unsigned)((ts + 1023) / 1024), 1024, [&] { seg_start_kernel(cu_s.get(), ns, ts, &hdr, seg.get()); });
  }
  printf("%d %d %d\n", hdr.error, hdr.n_qtiles, hdr.n_kvtiles);
  if (hdr.error) return 0;
  for (int r = 0; r < hdr.n_qtiles; ++r) {
    const TileDesc& d = qt[qo[r]];
    printf("q %d %d %d %d %d %d %d %d\n", d.kind, d.group, d.row0, d.row1, d.aux, d.work, d.chunk, d.nchunks);
  }
  for (int r = 0; r < hdr.n_kvtiles; ++r) {
    const TileDesc& d = kt[ko[r]];
    printf("k %d %d %d %d %d %d %d %d\n", d.kind, d.group, d.row0, d.row1, d.aux, d.work, d.chunk, d.nchunks);
  }
  printf("s");
  for (int r = 0; r < ts; ++r) printf(" %d", seg[r]);
  printf("\n");
  return 0;
}
