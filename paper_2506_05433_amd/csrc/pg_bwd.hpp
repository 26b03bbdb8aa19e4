// Backward kernels (vector-Jacobian product of the forward, Lemma 1 / Appendix A.1).
//
//   bwd_dot_kernel : Dsum[h][row] = <dO_row, O_row> (the softmax-Jacobian row term).
//   dkdv_kernel    : key-stationary. A workgroup owns 128 keys of one key/value head
//                    (32 per wave, kept in registers) and walks, in a fixed order, every
//                    query row that sees them: for each query head sharing the kv head,
//                    the causal prefix rows and then every response row of every member
//                    of the group. The prefix dK/dV of a group is therefore the G-way sum
//                    of the members' contributions taken in member order inside one
//                    workgroup: deterministic, no atomics.
//   dq_kernel      : query-stationary (the forward's tiling), recomputing P and dP.
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
  const PlanHeader* hdr;
  const GroupInfoEx* ginfo;
  const TileDesc *qtiles, *kvtiles;
  const int *qorder, *kvorder;
  const int* seg_start;
  int h_q, h_kv, total_prefix, total_suffix;
  float scale, scale_log2;
};

// ------------------------------------------------------------------ Dsum = rowsum(dO * O)
template <typename T, int D>
__global__ void __launch_bounds__(256) bwd_dot_kernel(const BwdArgs a) {
  // 16 lanes per (row, head); 16 rows-heads per 256-thread block
  constexpr int EPL = D / 16;  // elements per lane
  const int rows = a.total_prefix + a.total_suffix;
  const long item = (long)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int sub = threadIdx.x & 15;
  if (item >= (long)rows * a.h_q) return;
  const int row = (int)(item / a.h_q), head = (int)(item % a.h_q);
  const bool pre = row < a.total_prefix;
  const int r = pre ? row : row - a.total_prefix;
  const T* O = (const T*)(pre ? a.o_pre : a.o_suf) + ((size_t)r * a.h_q + head) * D + sub * EPL;
  const T* G = (const T*)(pre ? a.do_pre : a.do_suf) + ((size_t)r * a.h_q + head) * D + sub * EPL;
  float acc = 0.f;
#pragma unroll
  for (int e = 0; e < EPL; ++e) acc += (float)O[e] * (float)G[e];
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, 16);
  if (sub == 0) a.dsum[(size_t)head * rows + row] = acc;
}

// ------------------------------------------------------------------ dK, dV (key-stationary)
constexpr int kKvBN = 128;  // keys per workgroup (32 per wave)
constexpr int kKvBQ = 64;   // query rows per staged tile
constexpr int kKvThreads = 256;

template <typename T, int D>
__global__ void __launch_bounds__(kKvThreads) dkdv_kernel(const BwdArgs a) {
  using E = Elt<T>;
  using Frag = typename E::Frag;
  constexpr int BQ = kKvBQ;
  constexpr int KK = D / 16, DB = D / 32;
  constexpr int TILE = LdsTile<T, D>::bytes(BQ);
  __shared__ __attribute__((aligned(16))) char smem[2][2][TILE];  // [buffer][Q, dO]
  __shared__ __attribute__((aligned(16))) float s_lse[2][BQ];     // lse * log2(e), +inf for padding
  __shared__ __attribute__((aligned(16))) float s_dsum[2][BQ];
  __shared__ int s_seg[2][BQ];

  const BlockSlot slot = xcd_slot(blockIdx.x, a.h_kv, 1);
  const int rank = slot.unit, kvh = slot.head;
  if (rank >= a.hdr->n_kvtiles) return;
  const TileDesc td = a.kvtiles[a.kvorder[rank]];
  const GroupInfoEx gi = a.ginfo[td.group];
  const bool kv_suffix = td.kind == 1;
  const int ratio = a.h_q / a.h_kv;
  const int rows_all = a.total_prefix + a.total_suffix;

  const int tid = threadIdx.x, wave = uniform(tid >> 6), lane = tid & 63;
  const int n = lane & 31, hh = lane >> 5;
  const int wk0 = td.row0 + 32 * wave;            // first key of this wave
  const bool wave_active = wk0 < td.row1;
  const int wk1 = min(wk0 + 32, td.row1) - 1;     // last valid key of this wave
  const int key = wk0 + n;
  const bool kvalid = key < td.row1;
  const int key_c = kvalid ? key : td.row1 - 1;

  const T* Kb = (const T*)(kv_suffix ? a.k_suf : a.k_pre);
  const T* Vb = (const T*)(kv_suffix ? a.v_suf : a.v_pre);
  Frag kf[KK], vf[KK];
  {
    const size_t off = ((size_t)key_c * a.h_kv + kvh) * D + 8 * hh;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      kf[kk] = E::global_row(Kb + off + 16 * kk, kvalid);
      vf[kk] = E::global_row(Vb + off + 16 * kk, kvalid);
    }
  }
  f32x16 dk[DB], dv[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) { dk[db] = f32x16{}; dv[db] = f32x16{}; }

  // Query ranges that see these keys, in fixed order:
  //   prefix keys  : prefix rows [row0, p1) (causal), then response rows [s0, s1) (dense)
  //   response keys: response rows [row0, aux) (causal within each member)
  const int r1_lo = td.row0;
  const int r1_hi = kv_suffix ? td.aux : gi.p1;
  const int r2_lo = kv_suffix ? 0 : gi.s0;
  const int r2_hi = kv_suffix ? 0 : gi.s1;
  const int n1 = (r1_hi - r1_lo + BQ - 1) / BQ;
  const int n2 = (r2_hi - r2_lo + BQ - 1) / BQ;
  const int per_head = n1 + n2;
  const int total = per_head * ratio;
  const float c = a.scale_log2;

  TileLoader<T, BQ, D, kKvThreads> ldq, ldo;
  float pf_lse = 0.f, pf_dsum = 0.f;
  int pf_seg = 0;
  auto issue = [&](int it) {
    const int hq = kvh * ratio + it / per_head;
    const int j = it % per_head;
    const bool first = j < n1;
    // first range: prefix rows for prefix keys, response rows for response keys
    const bool qsuf = first ? kv_suffix : true;
    const int q0 = first ? r1_lo + j * BQ : r2_lo + (j - n1) * BQ;
    const int qend = first ? r1_hi : r2_hi;
    const T* Qs = (const T*)(qsuf ? a.q_suf : a.q_pre);
    const T* Gs = (const T*)(qsuf ? a.do_suf : a.do_pre);
    const size_t off = ((size_t)q0 * a.h_q + hq) * D;
    ldq.load(Qs + off, a.h_q * D, qend - q0, tid);
    ldo.load(Gs + off, a.h_q * D, qend - q0, tid);
    if (tid < BQ) {
      const int q = q0 + tid;
      const bool v = q < qend;
      const float* L = qsuf ? a.lse_suf : a.lse_pre;
      const int tot = qsuf ? a.total_suffix : a.total_prefix;
      pf_lse = v ? L[(size_t)hq * tot + q] * kLog2e : INFINITY;
      pf_dsum = v ? a.dsum[(size_t)hq * rows_all + (qsuf ? a.total_prefix : 0) + q] : 0.f;
      pf_seg = (v && qsuf) ? a.seg_start[q] : 0;
    }
  };
  auto commit = [&](int buf) {
    ldq.store(smem[buf][0], tid);
    ldo.store(smem[buf][1], tid);
    if (tid < BQ) { s_lse[buf][tid] = pf_lse; s_dsum[buf][tid] = pf_dsum; s_seg[buf][tid] = pf_seg; }
  };

  if (total > 0) { issue(0); commit(0); }
  __syncthreads();

  for (int it = 0; it < total; ++it) {
    const int buf = it & 1;
    if (it + 1 < total) issue(it + 1);
    const int j = it % per_head;
    const bool first = j < n1;
    const bool qsuf = first ? kv_suffix : true;
    const int q0 = first ? r1_lo + j * BQ : r2_lo + (j - n1) * BQ;
    const int qend = first ? r1_hi : r2_hi;
    // masking mode: causal when queries and keys are on the same side
    const bool causal = first;  // prefix keys x prefix rows, or response keys x response rows
    bool skip = false, full = true;  // padding rows need no mask: their lse is +inf
    if (causal) {
      skip = q0 + BQ - 1 < wk0;                      // every query precedes every key
      full = full && (q0 >= wk1);                    // every query sees every key
      if (kv_suffix) {
        const int seg_lo = s_seg[buf][0];
        const int last = min(q0 + BQ, qend) - 1 - q0;
        const int seg_hi = s_seg[buf][last];
        skip = skip || (seg_lo > wk1);               // queries all belong to later members
        full = full && (seg_hi <= wk0);
      }
    }
    if (wave_active && !skip) {
      const char* Qt = smem[buf][0];
      const char* Gt = smem[buf][1];
      // two halves of 32 query rows, one after the other (keeps S and dP of 32 rows live)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          s = E::mma(E::template lds_row<D>(Qt, 32 * qb + n, 2 * kk + hh), kf[kk], s);
          dp = E::mma(E::template lds_row<D>(Gt, 32 * qb + n, 2 * kk + hh), vf[kk], dp);
        }
        // P = exp2(S*c - lse*log2e) (0 on padding rows, whose lse is +inf);
        // dS = P * (dP - Dsum); rows are queries, the lane's column is its key.
        // The mask is only evaluated on tiles that straddle a boundary, branch-free.
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const f32x4 l4 = *(const f32x4*)&s_lse[buf][32 * qb + 8 * i + 4 * hh];
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) s[4 * i + jj] = fast_exp2(fmaf(s[4 * i + jj], c, -l4[jj]));
        }
        if (!full) {
          // boundary tile: query offset o = 8i + jj of register r = 4i + jj sees the lane's
          // key iff o >= lim (causal) and the key is not before the query's member start
          asm volatile("");
          const int lim = key_c - (q0 + 32 * qb + 4 * hh);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            int4 g4 = int4{0, 0, 0, 0};
            if (kv_suffix) g4 = *(const int4*)&s_seg[buf][32 * qb + 8 * i + 4 * hh];
            const int gs[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              const int o = 8 * i + jj;
              const bool ok = (o >= lim) & (key_c >= gs[jj]);
              s[4 * i + jj] = ok ? s[4 * i + jj] : 0.f;
            }
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const f32x4 d4 = *(const f32x4*)&s_dsum[buf][32 * qb + 8 * i + 4 * hh];
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) dp[4 * i + jj] = s[4 * i + jj] * (dp[4 * i + jj] - d4[jj]);
        }
        // dV^T += dO^T P ; dK^T += Q^T dS over these 32 queries (two k steps of 16)
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
          const int t = 2 * qb + t2;
          const Frag pfr = E::acc_to_frag(s, t2);
          const Frag dsf = E::acc_to_frag(dp, t2);
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            dv[db] = E::mma(E::template lds_tr<D>(Gt, 16 * t, 32 * db, lane), pfr, dv[db]);
            dk[db] = E::mma(E::template lds_tr<D>(Qt, 16 * t, 32 * db, lane), dsf, dk[db]);
          }
        }
      }
    }
    if (it + 1 < total) commit(buf ^ 1);
    __syncthreads();
  }

  if (!wave_active || !kvalid) return;
  T* dK = (T*)(kv_suffix ? a.dk_suf : a.dk_pre) + ((size_t)key * a.h_kv + kvh) * D;
  T* dV = (T*)(kv_suffix ? a.dv_suf : a.dv_pre) + ((size_t)key * a.h_kv + kvh) * D;
  const float sc = a.scale;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d0 = 32 * db + 8 * i + 4 * hh;
      E::store4(dK + d0, dk[db][4 * i] * sc, dk[db][4 * i + 1] * sc, dk[db][4 * i + 2] * sc, dk[db][4 * i + 3] * sc);
      E::store4(dV + d0, dv[db][4 * i], dv[db][4 * i + 1], dv[db][4 * i + 2], dv[db][4 * i + 3]);
    }
}

// ------------------------------------------------------------------ dQ (query-stationary)
constexpr int kDqBM = 128;
constexpr int kDqBN = 64;
constexpr int kDqThreads = 256;

template <typename T, int D>
#ifndef PG_DQ_MIN_BLOCKS
#define PG_DQ_MIN_BLOCKS 2
#endif
__global__ void __launch_bounds__(kDqThreads, PG_DQ_MIN_BLOCKS) dq_kernel(const BwdArgs a) {
  using E = Elt<T>;
  using Frag = typename E::Frag;
  constexpr int BN = kDqBN;
  constexpr int KK = D / 16, DB = D / 32;
  constexpr int TILE = LdsTile<T, D>::bytes(BN);
  __shared__ __attribute__((aligned(16))) char smem[2][2][TILE];  // [buffer][K, V]

  const BlockSlot slot = xcd_slot(blockIdx.x, a.h_q, a.h_q / a.h_kv);
  const int rank = slot.unit, head = slot.head;
  if (rank >= a.hdr->n_qtiles) return;
  const TileDesc td = a.qtiles[a.qorder[rank]];
  const GroupInfoEx gi = a.ginfo[td.group];
  const int kvh = head / (a.h_q / a.h_kv);
  const bool suffix = td.kind == 1;
  const int rows_all = a.total_prefix + a.total_suffix;

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
    const size_t off = ((size_t)qrow_c * a.h_q + head) * D + 8 * hh;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      qf[kk] = E::global_row(Q + off + 16 * kk, qvalid);
      gf[kk] = E::global_row(G + off + 16 * kk, qvalid);
    }
  }
  const float* L = suffix ? a.lse_suf : a.lse_pre;
  const int tot = suffix ? a.total_suffix : a.total_prefix;
  const float lse2 = L[(size_t)head * tot + qrow_c] * kLog2e;
  const float dsum = a.dsum[(size_t)head * rows_all + (suffix ? a.total_prefix : 0) + qrow_c];
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

  TileLoader<T, BN, D, kDqThreads> ldk, ldv;
  auto issue = [&](int j) {
    const bool segA = j < nA;
    const int k0 = segA ? kA0 + j * BN : kB0 + (j - nA) * BN;
    const int kend = segA ? kA1 : kB1;
    ldk.load((segA ? Kp : Ks) + (size_t)k0 * kvstride + kvh * D, kvstride, kend - k0, tid);
    ldv.load((segA ? Vp : Vs) + (size_t)k0 * kvstride + kvh * D, kvstride, kend - k0, tid);
  };

  f32x16 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x16{};
  const float c = a.scale_log2;

  if (ntiles > 0) {
    issue(0);
    ldk.store(smem[0][0], tid);
    ldv.store(smem[0][1], tid);
  }
  __syncthreads();

  for (int j = 0; j < ntiles; ++j) {
    const int buf = j & 1;
    if (j + 1 < ntiles) issue(j + 1);
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
      const char* Kt = smem[buf][0];
      const char* Vt = smem[buf][1];
      // two blocks of 32 keys, one after the other
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          s = E::mma(E::template lds_row<D>(Kt, 32 * kb + n, 2 * kk + hh), qf[kk], s);
          dp = E::mma(E::template lds_row<D>(Vt, 32 * kb + n, 2 * kk + hh), gf[kk], dp);
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
            acc[db] = E::mma(E::template lds_tr<D>(Kt, 16 * (2 * kb + t2), 32 * db, lane), dsf, acc[db]);
        }
      }
    }
    if (j + 1 < ntiles) {
      ldk.store(smem[buf ^ 1][0], tid);
      ldv.store(smem[buf ^ 1][1], tid);
    }
    __syncthreads();
  }

  if (!wave_active || !qvalid) return;
  T* dQ = (T*)(suffix ? a.dq_suf : a.dq_pre) + ((size_t)qrow * a.h_q + head) * D;
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
