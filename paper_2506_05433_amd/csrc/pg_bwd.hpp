// Backward kernels (vector-Jacobian product of the forward, Lemma 1 / Appendix A.1).
//
//   dq_kernel      : query-stationary (the forward's tiling), recomputing P and dP. It runs
//                    first and also forms Dsum[h][row] = <dO_row, O_row> (the softmax-Jacobian
//                    row term) for its rows, which the dK/dV kernel then reads.
//   dkdv_kernel    : key-stationary. A workgroup owns 128 keys of one key/value head
//                    (32 per wave, kept in registers) and walks, in a fixed order, every
//                    query row that sees them: for each query head sharing the kv head,
//                    the causal prefix rows and then every response row of every member
//                    of the group. The prefix dK/dV of a group is therefore the G-way sum
//                    of the members' contributions taken in member order inside one
//                    workgroup: deterministic, no atomics.
//
// Products per (query tile, key tile), all on 32x32 MFMA tiles:
//   dkdv: S = Q K^T and dP = dO V^T with queries as rows (A = Q, dO from LDS, B = K, V
//         from registers); dV^T += dO^T P and dK^T += Q^T dS take P and dS straight
//         from the accumulators as B operands and dO^T, Q^T through transposing LDS reads.
//   dq  : S^T = K Q^T and dP^T = V dO^T with queries as columns; dQ^T += K^T dS^T.
#pragma once
#include "pg_common.hpp"
#include "pg_plan.hpp"

namespace pg {

struct BwdArgs {
  const void *q_pre, *k_pre, *v_pre, *q_suf, *k_suf, *v_suf;
  const void *o_pre, *o_suf, *do_pre, *do_suf;
  const float *lse_pre, *lse_suf;
  void *dq_pre, *dk_pre, *dv_pre, *dq_suf, *dk_suf, *dv_suf;
  float* dsum;  // [h_q][total_prefix + total_suffix]
  float* part;  // [kv_chunks][2 (dK, dV)][total_prefix][h_kv][D] fp32 partials, when kv_chunks > 1
  int kv_chunks;
  const PlanHeader* hdr;
  const GroupInfoEx* ginfo;
  const TileDesc *qtiles, *kvtiles;
  const int *qorder, *kvorder;
  const int* seg_start;
  int h_q, h_kv, total_prefix, total_suffix;
  float scale, scale_log2;
  // 1: single-buffer layout of Eq. (2) (see FwdArgs::xl); xrow maps packed rows (prefix
  // rows, then response rows) to tensor rows for the kernels that sweep rows
  int xl;
  const int* xrow;
};

// ------------------------------------------------------------------ dK, dV (key-stationary)
// A workgroup owns 128 keys of one kv head, split into four groups of 32. Each key
// group is served by two waves (on one SIMD, or on two when the key tile is ragged):
//   P-wave : S = Q K^T, P = exp(S*scale - lse) (masked), dV^T += dO^T P; it hands P
//            (bf16 operand fragments) to its partner through LDS;
//   G-wave : one query tile behind, dP = dO V^T, dS = P (dP - Dsum), dK^T += Q^T dS.
// Each wave therefore holds one kv operand and one accumulator (about half the
// registers of a wave doing all four products), so two waves fit per SIMD and one's
// exp/VALU work overlaps the other's matrix instructions. Query tiles are
// triple-buffered in LDS (P-waves read tile i, G-waves tile i-1; the G-waves load tile
// i+1 through registers and write it to LDS after their work on tile i-1).
constexpr int kKvGroups = 4;                 // 32-key groups per workgroup
constexpr int kKvBN = 32 * kKvGroups;        // keys per workgroup
constexpr int kKvThreads = 128 * kKvGroups;  // a P-wave and a G-wave per key group

template <typename T>
struct KvTileRows {  // query rows per staged tile
  static constexpr int value = sizeof(T) == 2 ? 64 : 32;
};

template <typename T, int D>
__global__ void __launch_bounds__(kKvThreads, 512 / kKvThreads) dkdv_kernel(const BwdArgs a) {
  using E = Elt<T>;
  using Frag = typename E::Frag;
  constexpr int BQ = KvTileRows<T>::value;  // query rows per staged tile
  constexpr int QB = BQ / 32;               // 32-row halves
  constexpr int NT = BQ / 16;               // 16-wide k steps over the tile's queries
  constexpr int KK = D / 16, DB = D / 32;
  constexpr int NBUF = 3;
  constexpr int TILE = LdsTile<T, D>::bytes(BQ);
  __shared__ __attribute__((aligned(16))) char smem[NBUF][2][TILE];  // [buffer][Q, dO]
  __shared__ __attribute__((aligned(16))) float s_lse[NBUF][BQ];     // lse * log2(e), +inf for padding
  __shared__ __attribute__((aligned(16))) float s_dsum[NBUF][BQ];
  __shared__ __attribute__((aligned(16))) int s_seg[NBUF][BQ];
  __shared__ __attribute__((aligned(16))) Frag s_p[2][kKvGroups][NT][64];  // P handoff [buffer][group][k step][lane]

  const BlockSlot slot = xcd_slot(blockIdx.x, a.h_kv, 1);
  const int rank = slot.unit, kvh = slot.head;
  if (rank >= a.hdr->n_kvtiles) return;
  const TileDesc td = a.kvtiles[a.kvorder[rank]];
  const GroupInfoEx gi = a.ginfo[td.group];
  const bool kv_suffix = td.kind == 1;
  // tensor row offsets of this group's prefix and response rows (single-buffer layout)
  const int xo_pre = a.xl ? gi.s0 : 0, xo_suf = a.xl ? gi.p1 : 0;
  const int xk = kv_suffix ? xo_suf : xo_pre;
  const int lse_ld_pre = a.xl ? a.total_prefix + a.total_suffix : a.total_prefix;
  const int lse_ld_suf = a.xl ? a.total_prefix + a.total_suffix : a.total_suffix;
  const int ratio = a.h_q / a.h_kv;
  const int rows_all = a.total_prefix + a.total_suffix;

  const int tid = threadIdx.x, wave = uniform(tid >> 6), lane = tid & 63;
  const int n = lane & 31, hh = lane >> 5;
  const bool pwave = wave < kKvGroups;
  // Key group of the wave. Waves run on SIMD wave % 4. With all four key groups holding keys,
  // the P- and G-wave of a group share a SIMD; a ragged key tile (fewer groups) pairs the
  // G-wave of group g with SIMD (g + 2) % 4 instead, so that its active waves spread over
  // all four SIMDs.
  const bool ragged = td.row1 - td.row0 <= kKvBN - 32;
  const int grp = (pwave || !ragged) ? wave % kKvGroups : (wave + kKvGroups / 2) % kKvGroups;
  const int wk0 = td.row0 + 32 * grp;             // first key of this key group
  const bool wave_active = wk0 < td.row1;
  const int wk1 = min(wk0 + 32, td.row1) - 1;     // last valid key of the group
  const int key = wk0 + n;
  const bool kvalid = key < td.row1;
  const int key_c = kvalid ? key : td.row1 - 1;

  // P-waves keep K, G-waves keep V (the B operand of their first product)
  Frag kv[KK];
  {
    const T* B = (const T*)(pwave ? (kv_suffix ? a.k_suf : a.k_pre) : (kv_suffix ? a.v_suf : a.v_pre));
    const size_t off = ((size_t)(key_c + xk) * a.h_kv + kvh) * D + 8 * hh;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) kv[kk] = E::global_row(B + off + 16 * kk, kvalid);
    // wait for them here, on every path: otherwise the compiler, unsure whether they landed,
    // waits for all outstanding loads (the next tile's copies included) before the first
    // product of every tile
    __builtin_amdgcn_s_waitcnt(0);
  }
  f32x16 acc[DB];  // dV^T (P-wave) or dK^T (G-wave)
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x16{};

  // Query ranges that see these keys, in fixed order:
  //   prefix keys  : response rows [s0, s1) (dense), then prefix rows [row0, p1) (causal);
  //   response keys: response rows [row0, aux) (causal within each member).
  // The dense response range comes first so that the workgroups of all prefix key
  // tiles of a kv head, which start together, stream the same query tiles in step
  // and share them in L2.
  const int rc_lo = td.row0;                       // causal range
  const int rc_hi = kv_suffix ? td.aux : gi.p1;
  const int rd_lo = kv_suffix ? 0 : gi.s0;         // dense range
  const int rd_hi = kv_suffix ? 0 : gi.s1;
  const int nd = (rd_hi - rd_lo + BQ - 1) / BQ;
  const int nc = (rc_hi - rc_lo + BQ - 1) / BQ;
  const int per_head = nd + nc;
  // this workgroup's piece [it0, it1) of the walk (a prefix key tile may be split in chunks)
  const int walk = per_head * ratio;
  const int it0 = (int)((long)walk * td.chunk / td.nchunks);
  const int it1 = (int)((long)walk * (td.chunk + 1) / td.nchunks);
  const float c = a.scale_log2;

  struct TileInfo {
    int hq, q0, qend;
    bool qsuf, causal;
  };
  // tile `it` is position j of query head hd's walk; the loop advances (hd, j) by one
  // tile per iteration instead of dividing
  auto info = [&](int hd, int j) {
    TileInfo ti;
    ti.hq = kvh * ratio + hd;
    ti.causal = j >= nd;  // prefix keys x prefix rows, or response keys x response rows
    ti.qsuf = ti.causal ? kv_suffix : true;
    ti.q0 = ti.causal ? rc_lo + (j - nd) * BQ : rd_lo + j * BQ;
    ti.qend = ti.causal ? rc_hi : rd_hi;
    return ti;
  };
  // visibility of a tile to this key group: skip (no pair visible) / full (all visible)
  auto visibility = [&](const TileInfo& ti, int buf, bool& skip, bool& full) {
    skip = false;
    full = true;  // padding rows need no mask: their lse is +inf
    if (ti.causal) {
      skip = ti.q0 + BQ - 1 < wk0;                   // every query precedes every key
      full = ti.q0 >= wk1;                            // every query sees every key
      if (kv_suffix) {
        const int last = min(ti.q0 + BQ, ti.qend) - 1 - ti.q0;
        skip = skip || (s_seg[buf][0] > wk1);         // queries all belong to later members
        full = full && (s_seg[buf][last] <= wk0);
      }
    }
  };

  // Query tiles are staged through registers, not copied straight into LDS: with the three
  // buffers in one LDS array indexed at run time, a direct copy into one of them would make
  // every read of another wait for the copy to land. The G-waves stage them (and the per-row
  // values below): with the G-waves issuing first, the P-waves were the longer chain of a
  // tile and the G-waves waited for them at the barrier, so the copies go there (measured
  // faster than any other split of the staging between the roles).
  TileLoader<T, BQ, D, kKvThreads / 2> ldq, ldo;
  ldq.init(a.h_q * D, wave - kKvGroups, lane);  // used by the G-waves only
  ldo.init(a.h_q * D, wave - kKvGroups, lane);
  FragOffsets<T, D> fo;
  fo.init(lane);
  // per-row values of the next tile: loaded with its copies, used only in commit() (a use
  // right after the load would wait for the copies issued before it as well)
  float pf_lse = 0.f, pf_dsum = 0.f;
  int pf_seg = 0;
  const int rl = tid - 64 * kKvGroups;  // row of this lane of the first G-wave
  const bool row_lane = rl >= 0 && rl < BQ;
  auto issue = [&](const TileInfo& ti, int it) {  // `it` selects the buffer
    const T* Qs = (const T*)(ti.qsuf ? a.q_suf : a.q_pre);
    const T* Gs = (const T*)(ti.qsuf ? a.do_suf : a.do_pre);
    const size_t off = ((size_t)(ti.q0 + (ti.qsuf ? xo_suf : xo_pre)) * a.h_q + ti.hq) * D;
    if (!pwave) {
      ldq.load(smem[it % NBUF][0], Qs + off, a.h_q * D, ti.qend - ti.q0);
      ldo.load(smem[it % NBUF][1], Gs + off, a.h_q * D, ti.qend - ti.q0);
    }
    if (row_lane) {
      const int q = min(ti.q0 + rl, ti.qend - 1);  // padding rows read the last row; commit() drops them
      const float* L = ti.qsuf ? a.lse_suf : a.lse_pre;
      const int ld = ti.qsuf ? lse_ld_suf : lse_ld_pre;
      pf_lse = L[(size_t)ti.hq * ld + q + (ti.qsuf ? xo_suf : xo_pre)];
      pf_dsum = a.dsum[(size_t)ti.hq * rows_all + (ti.qsuf ? a.total_prefix : 0) + q];
      if (ti.qsuf) pf_seg = a.seg_start[q];
    }
  };
  auto commit = [&](const TileInfo& ti, int buf) {
    if (!pwave) {
      ldq.store(smem[buf][0]);
      ldo.store(smem[buf][1]);
    }
    if (row_lane) {
      const bool v = ti.q0 + rl < ti.qend;
      s_lse[buf][rl] = v ? pf_lse * kLog2e : INFINITY;  // padding rows: P = 0
      s_dsum[buf][rl] = v ? pf_dsum : 0.f;
      s_seg[buf][rl] = (v && ti.qsuf) ? pf_seg : 0;
    }
  };

  // The walk: every wave stages its share of tile it+1, works on its tile, and meets the
  // others at one barrier per tile. The two roles run this skeleton as separate loops
  // (`work` is the role's body), so each keeps its accumulator in place; both loops
  // execute the same barriers, and the role is uniform per wave.
  auto walk_tiles = [&](auto&& work) {
    int cur_hd = it0 / (per_head > 0 ? per_head : 1), cur_j = it0 - cur_hd * per_head;
    TileInfo ti_cur = info(cur_hd, cur_j), ti_prev = ti_cur;  // tiles it and it - 1
    if (it1 > it0) { issue(ti_cur, it0 % NBUF); commit(ti_cur, it0 % NBUF); }
    ldq.wait();
    __syncthreads();
    for (int it = it0; it <= it1; ++it) {
      int nxt_hd = cur_hd, nxt_j = cur_j + 1;
      if (nxt_j == per_head) { nxt_j = 0; ++nxt_hd; }
      const TileInfo ti_next = info(nxt_hd, nxt_j);
      if (it + 1 < it1) issue(ti_next, it + 1);
      work(it, ti_cur, ti_prev);
      if (it + 1 < it1) commit(ti_next, (it + 1) % NBUF);
      ti_prev = ti_cur;
      ti_cur = ti_next;
      cur_hd = nxt_hd;
      cur_j = nxt_j;
      ldq.wait();
      __syncthreads();
    }
  };

  // The G-waves (one tile behind, the longer chain of each tile) issue first when both waves
  // of a SIMD are ready.
  if (!pwave) __builtin_amdgcn_s_setprio(1);
  if (pwave) {
    walk_tiles([&](int it, const TileInfo& ti, const TileInfo&) {
      if (!(it < it1 && wave_active)) return;
      // ---------------- P-wave on tile it
      const int buf = it % NBUF;
      bool skip, full;
      visibility(ti, buf, skip, full);
      if (!skip) {
        const char* Qt = smem[buf][0];
        const char* Gt = smem[buf][1];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          f32x16 sc = f32x16{};
#pragma unroll
          for (int kk = 0; kk < KK; ++kk)
            sc = E::mma(fo.row(Qt, 32 * qb, kk), kv[kk], sc);
          // P = exp2(S*c - lse*log2e); rows are queries, the lane's column is its key
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const f32x4 l4 = *(const f32x4*)&s_lse[buf][32 * qb + 8 * i + 4 * hh];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) sc[4 * i + jj] = fast_exp2(fmaf(sc[4 * i + jj], c, -l4[jj]));
          }
          if (!full) {
            // boundary tile: query offset o = 8i + jj of register r = 4i + jj sees the lane's
            // key iff o >= lim (causal) and the key is not before the query's member start
            asm volatile("");
            const int lim = key_c - (ti.q0 + 32 * qb + 4 * hh);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              int4 g4 = int4{0, 0, 0, 0};
              if (kv_suffix) g4 = *(const int4*)&s_seg[buf][32 * qb + 8 * i + 4 * hh];
              const int gs[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
              for (int jj = 0; jj < 4; ++jj) {
                const int o = 8 * i + jj;
                const bool ok = (o >= lim) & (key_c >= gs[jj]);
                sc[4 * i + jj] = ok ? sc[4 * i + jj] : 0.f;
              }
            }
          }
          // hand P to the G-wave and accumulate dV^T += dO^T P over these 32 queries
#pragma unroll
          for (int t2 = 0; t2 < 2; ++t2) {
            const int t = 2 * qb + t2;
            const Frag pf = E::acc_to_frag(sc, t2);
            s_p[it & 1][grp][t][lane] = pf;
#pragma unroll
            for (int db = 0; db < DB; ++db) acc[db] = E::mma(fo.tr(Gt, t, db), pf, acc[db]);
          }
        }
      }
    });
  } else {
    walk_tiles([&](int it, const TileInfo&, const TileInfo& ti) {
      if (!(it > it0 && wave_active)) return;
      // ---------------- G-wave on tile it-1
      const int buf = (it - 1) % NBUF;
      bool skip, full;
      visibility(ti, buf, skip, full);
      if (!skip) {
        const char* Qt = smem[buf][0];
        const char* Gt = smem[buf][1];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          f32x16 dp = f32x16{};
#pragma unroll
          for (int kk = 0; kk < KK; ++kk)
            dp = E::mma(fo.row(Gt, 32 * qb, kk), kv[kk], dp);
#pragma unroll
          for (int t2 = 0; t2 < 2; ++t2) {
            const int t = 2 * qb + t2;
            const Frag pf = s_p[(it - 1) & 1][grp][t][lane];
            // registers 8 t2 + e, e = 0..7, hold query rows 32 qb + 8 (2 t2 + e/4) + 4 hh + e%4
            const f32x4 d0 = *(const f32x4*)&s_dsum[buf][32 * qb + 16 * t2 + 4 * hh];
            const f32x4 d1 = *(const f32x4*)&s_dsum[buf][32 * qb + 16 * t2 + 8 + 4 * hh];
            float ds[8];
#pragma unroll
            for (int e = 0; e < 8; ++e)
              ds[e] = E::frag_elem(pf, e) * (dp[8 * t2 + e] - (e < 4 ? d0[e] : d1[e - 4]));
            const Frag dsf = E::to_frag(ds);
#pragma unroll
            for (int db = 0; db < DB; ++db) acc[db] = E::mma(fo.tr(Qt, t, db), dsf, acc[db]);
          }
        }
      }
    });
  }

  if (!wave_active || !kvalid) return;
  const float sc = pwave ? 1.f : a.scale;
  if (td.nchunks > 1) {
    // fp32 partial of this chunk; kv_reduce_kernel adds the chunks in order
    float* out = a.part + (((size_t)td.chunk * 2 + (pwave ? 1 : 0)) * a.total_prefix + key) * a.h_kv * D +
                 (size_t)kvh * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d0 = 32 * db + 8 * i + 4 * hh;
        *(f32x4*)(out + d0) = f32x4{acc[db][4 * i] * sc, acc[db][4 * i + 1] * sc, acc[db][4 * i + 2] * sc,
                                    acc[db][4 * i + 3] * sc};
      }
    return;
  }
  T* out = (T*)(pwave ? (kv_suffix ? a.dv_suf : a.dv_pre) : (kv_suffix ? a.dk_suf : a.dk_pre)) +
           ((size_t)(key + xk) * a.h_kv + kvh) * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d0 = 32 * db + 8 * i + 4 * hh;
      E::store4(out + d0, acc[db][4 * i] * sc, acc[db][4 * i + 1] * sc, acc[db][4 * i + 2] * sc,
                acc[db][4 * i + 3] * sc);
    }
}

// dK_pre, dV_pre = sum over the kv_chunks partials, in chunk order (deterministic).
template <typename T, int D>
__global__ void __launch_bounds__(256) kv_reduce_kernel(const BwdArgs a) {
  const long n4 = (long)a.total_prefix * a.h_kv * D / 4;  // float4 groups per tensor
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= 2 * n4) return;
  const int which = i >= n4;  // 0: dK, 1: dV
  const long e = i - which * n4;
  const size_t stride = (size_t)2 * a.total_prefix * a.h_kv * D;  // floats per chunk
  const float* src = a.part + (size_t)which * a.total_prefix * a.h_kv * D + 4 * e;
  f32x4 s = *(const f32x4*)src;
  for (int c = 1; c < a.kv_chunks; ++c) s += *(const f32x4*)(src + c * stride);
  long de = e;  // destination float4 index: the packed prefix row mapped to its tensor row
  if (a.xl) {
    const long per_row = (long)a.h_kv * D / 4;
    const long t = e / per_row;
    de = (long)a.xrow[t] * per_row + (e - t * per_row);
  }
  T* dst = (T*)(which ? a.dv_pre : a.dk_pre) + 4 * de;
  Elt<T>::store4(dst, s[0], s[1], s[2], s[3]);
}

// ------------------------------------------------------------------ dQ (query-stationary)
constexpr int kDqBM = 128;
constexpr int kDqBN = 64;
constexpr int kDqThreads = 256;

template <typename T, int D>
__global__ void __launch_bounds__(kDqThreads, 2) dq_kernel(const BwdArgs a) {
  using E = Elt<T>;
  using Frag = typename E::Frag;
  constexpr int BN = kDqBN;
  constexpr int KK = D / 16, DB = D / 32;
  constexpr int TILE = LdsTile<T, D>::bytes(BN);
  // two K/V buffers as distinct LDS objects, named statically by a loop unrolled by two
  // (the forward kernel explains why)
  __shared__ __attribute__((aligned(16))) char sK0[TILE], sV0[TILE], sK1[TILE], sV1[TILE];

  const BlockSlot slot = xcd_slot(blockIdx.x, a.h_q, a.h_q / a.h_kv);
  const int rank = slot.unit, head = slot.head;
  if (rank >= a.hdr->n_qtiles) return;
  const TileDesc td = a.qtiles[a.qorder[rank]];
  const GroupInfoEx gi = a.ginfo[td.group];
  const int kvh = head / (a.h_q / a.h_kv);
  const bool suffix = td.kind == 1;
  const int rows_all = a.total_prefix + a.total_suffix;
  // tensor row offsets of this group's prefix and response rows (single-buffer layout)
  const int xo_pre = a.xl ? gi.s0 : 0, xo_suf = a.xl ? gi.p1 : 0;
  const int xq = suffix ? xo_suf : xo_pre;

  const int tid = threadIdx.x, wave = uniform(tid >> 6), lane = tid & 63;
  const int n = lane & 31, hh = lane >> 5;
  const int wq0 = td.row0 + 32 * wave;
  const bool wave_active = wq0 < td.row1;
  const int wq1 = min(wq0 + 32, td.row1) - 1;
  const int qrow = wq0 + n;
  const bool qvalid = qrow < td.row1;
  const int qrow_c = qvalid ? qrow : td.row1 - 1;

  const T* Q = (const T*)(suffix ? a.q_suf : a.q_pre);
  const T* G = (const T*)(suffix ? a.do_suf : a.do_pre);
  Frag qf[KK], gf[KK];
  {
    const size_t off = ((size_t)(qrow_c + xq) * a.h_q + head) * D + 8 * hh;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      qf[kk] = E::global_row(Q + off + 16 * kk, qvalid);
      gf[kk] = E::global_row(G + off + 16 * kk, qvalid);
    }
  }
  const float* L = suffix ? a.lse_suf : a.lse_pre;
  const int ld = a.xl ? rows_all : (suffix ? a.total_suffix : a.total_prefix);
  const float lse2 = L[(size_t)head * ld + qrow_c + xq] * kLog2e;
  // Dsum = <dO, O> of the lane's query: the lane holds half of the row (the dO fragments
  // above), its partner lane (lane ^ 32) the other half. Stored for the dK/dV kernel.
  float dsum;
  {
    const T* O = (const T*)(suffix ? a.o_suf : a.o_pre);
    const size_t off = ((size_t)(qrow_c + xq) * a.h_q + head) * D + 8 * hh;
    float part = 0.f;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const Frag of = E::global_row(O + off + 16 * kk, qvalid);
#pragma unroll
      for (int e = 0; e < 8; ++e) part = fmaf(E::frag_elem(of, e), E::frag_elem(gf[kk], e), part);
    }
    dsum = wave_swap32_sum(part);
    if (qvalid && hh == 0) a.dsum[(size_t)head * rows_all + (suffix ? a.total_prefix : 0) + qrow] = dsum;
  }
  const int seg_q = suffix ? a.seg_start[qrow_c] : 0;
  const int seg_w_lo = (suffix && wave_active) ? a.seg_start[wq0] : 0;
  const int seg_w_hi = (suffix && wave_active) ? a.seg_start[wq1] : 0;

  const int kA0 = gi.p0, kA1 = suffix ? gi.p1 : td.row1;
  const int kB0 = suffix ? td.aux : 0, kB1 = suffix ? td.row1 : 0;
  const int nA = (kA1 - kA0 + BN - 1) / BN;
  const int nB = (kB1 - kB0 + BN - 1) / BN;
  const int ntiles = nA + nB;
  const T* Kp = (const T*)a.k_pre; const T* Vp = (const T*)a.v_pre;
  const T* Ks = (const T*)a.k_suf; const T* Vs = (const T*)a.v_suf;
  const int kvstride = a.h_kv * D;

  Stager<T, BN, D, kDqThreads> ldk, ldv;
  ldk.init(kvstride, wave, lane);
  ldv.init(kvstride, wave, lane);
  FragOffsets<T, D> fo;
  fo.init(lane);
  auto issue = [&](int j, char* kdst, char* vdst) {
    const bool segA = j < nA;
    const int k0 = segA ? kA0 + j * BN : kB0 + (j - nA) * BN;
    const int kend = segA ? kA1 : kB1;
    const size_t kx = (size_t)(k0 + (segA ? xo_pre : xo_suf));
    ldk.load(kdst, (segA ? Kp : Ks) + kx * kvstride + kvh * D, kvstride, kend - k0);
    ldv.load(vdst, (segA ? Vp : Vs) + kx * kvstride + kvh * D, kvstride, kend - k0);
  };

  f32x16 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x16{};
  const float c = a.scale_log2;

  // one key tile: start the copy of tile j + 1 into (Kn, Vn), work on (Kt, Vt), publish
  auto step = [&](int j, const char* Kt, const char* Vt, char* Kn, char* Vn) {
    if (j + 1 < ntiles) issue(j + 1, Kn, Vn);
    const bool segA = j < nA;
    const int k0 = segA ? kA0 + j * BN : kB0 + (j - nA) * BN;
    const int kend = segA ? kA1 : kB1;
    bool skip, full;
    const bool cross = segA && suffix;  // response queries x prefix keys: no causal mask
    if (cross) {
      skip = false;
      full = k0 + BN <= kend;
    } else {
      skip = k0 > wq1;
      if (!segA) skip = skip || (k0 + BN <= seg_w_lo);
      full = (k0 + BN - 1 <= wq0) && (k0 + BN <= kend);
      if (!segA) full = full && (k0 >= seg_w_hi);
    }
    if (wave_active && !skip) {
      // two blocks of 32 keys, one after the other
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          s = E::mma(fo.row(Kt, 32 * kb, kk), qf[kk], s);
          dp = E::mma(fo.row(Vt, 32 * kb, kk), gf[kk], dp);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[r] = fast_exp2(fmaf(s[r], c, -lse2));
        }
        if (!full) {  // boundary tile: zero the invisible keys (see the forward kernel)
          asm volatile("");
          const int base = k0 + 32 * kb + 4 * hh;
          int hi = kend - base;
          if (!cross) hi = min(hi, qrow_c + 1 - base);
          const int lo = segA ? -(1 << 30) : seg_q - base;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int o = 8 * (r >> 2) + (r & 3);
            s[r] = ((o >= lo) & (o < hi)) ? s[r] : 0.f;
          }
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) dp[r] = s[r] * (dp[r] - dsum);
        // dQ^T += K^T dS^T over these 32 keys (two k steps of 16)
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
          const Frag dsf = E::acc_to_frag(dp, t2);
#pragma unroll
          for (int db = 0; db < DB; ++db)
            acc[db] = E::mma(fo.tr(Kt, (2 * kb + t2), db), dsf, acc[db]);
        }
      }
    }
    if (j + 1 < ntiles) {
      ldk.store(Kn);
      ldv.store(Vn);
    }
    ldk.wait();
    __syncthreads();
  };

  if (ntiles > 0) {
    issue(0, sK0, sV0);
    ldk.store(sK0);
    ldv.store(sV0);
  }
  ldk.wait();
  __syncthreads();
  for (int j = 0; j < ntiles; j += 2) {
    step(j, sK0, sV0, sK1, sV1);
    if (j + 1 < ntiles) step(j + 1, sK1, sV1, sK0, sV0);
  }

  if (!wave_active || !qvalid) return;
  T* dQ = (T*)(suffix ? a.dq_suf : a.dq_pre) + ((size_t)(qrow + xq) * a.h_q + head) * D;
  const float sc = a.scale;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d0 = 32 * db + 8 * i + 4 * hh;
      E::store4(dQ + d0, acc[db][4 * i] * sc, acc[db][4 * i + 1] * sc, acc[db][4 * i + 2] * sc, acc[db][4 * i + 3] * sc);
    }
}

}  // namespace pg
