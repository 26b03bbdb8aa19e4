// Forward kernel: flash-style tiled online softmax over the grouped layout (Eq. (4)).
//
// One workgroup = one query tile (up to 128 rows, 32 per wave) of one query head.
// The key/value stream of a tile is:
//   prefix query tile  : prefix keys [p0, row1)               (causal)
//   response query tile: prefix keys [p0, p1)                 (dense: every response row sees them)
//                        then response keys [aux, row1)        (causal inside each member)
// so the two attention calls of Eq. (4) become one online softmax per row. Key
// tiles no row of a wave can see are skipped by that wave, and masking code runs
// only on tiles that straddle a boundary.
//
// Per 64-key tile, each wave computes S^T = K Q^T (keys x queries) so that every
// lane owns one query column: the running max/sum of a row live in one lane pair
// (l, l^32). P^T is then directly the B operand of O^T += V^T P^T; V^T comes from
// the row-major LDS tile through transposing reads.
#pragma once
#include "pg_common.hpp"
#include "pg_plan.hpp"

namespace pg {

struct FwdArgs {
  const void *q_pre, *k_pre, *v_pre, *q_suf, *k_suf, *v_suf;
  void *o_pre, *o_suf;
  float *lse_pre, *lse_suf;
  const PlanHeader* hdr;
  const GroupInfoEx* ginfo;
  const TileDesc* qtiles;
  const int* qorder;
  const int* seg_start;
  int h_q, h_kv, total_prefix, total_suffix;
  float scale_log2;  // softmax_scale * log2(e)
  // 1: every tensor is one buffer in the layout of Eq. (2) (per group [P; R_1; ...; R_G],
  // groups one after another; *_pre and *_suf point at the same buffer, lse is
  // [h_q, total_prefix + total_suffix]); 0: separate prefix and response buffers.
  int xl;
};

constexpr int kFwdBM = 128;  // query rows per workgroup
constexpr int kFwdBN = 64;   // keys per tile
constexpr int kFwdThreads = 256;

template <typename T, int D>
#ifndef PG_FWD_MIN_BLOCKS
#define PG_FWD_MIN_BLOCKS 2
#endif
__global__ void __launch_bounds__(kFwdThreads, PG_FWD_MIN_BLOCKS) fwd_kernel(const FwdArgs a) {
  using E = Elt<T>;
  using Frag = typename E::Frag;
  constexpr int BN = kFwdBN;
  constexpr int KK = D / 16;  // k steps over head_dim
  constexpr int DB = D / 32;  // 32-wide blocks of head_dim
  constexpr int TILE = LdsTile<T, D>::bytes(BN);
  // Two K/V buffers as four distinct LDS objects: the loop below is unrolled by two so
  // that every access names its buffer statically, which lets the compiler see that the
  // copy into one buffer cannot overlap the reads of the other (with one array indexed
  // by j & 1 it has to wait for the copy to land before the first read of the tile).
  __shared__ __attribute__((aligned(16))) char sK0[TILE], sV0[TILE], sK1[TILE], sV1[TILE];

  const BlockSlot slot = xcd_slot(blockIdx.x, a.h_q, a.h_q / a.h_kv);
  const int rank = slot.unit, head = slot.head;
  if (rank >= a.hdr->n_qtiles) return;
  const TileDesc td = a.qtiles[a.qorder[rank]];
  const GroupInfoEx gi = a.ginfo[td.group];
  const int kvh = head / (a.h_q / a.h_kv);
  const bool suffix = td.kind == 1;
  // tensor row offsets of this group's prefix and response rows (single-buffer layout)
  const int xo_pre = a.xl ? gi.s0 : 0, xo_suf = a.xl ? gi.p1 : 0;
  const int xq = suffix ? xo_suf : xo_pre;

  const int tid = threadIdx.x, wave = uniform(tid >> 6), lane = tid & 63;
  const int n = lane & 31, hh = lane >> 5;
  const int wq0 = td.row0 + 32 * wave;             // first row of this wave
  const bool wave_active = wq0 < td.row1;
  const int wq1 = min(wq0 + 32, td.row1) - 1;      // last valid row of this wave
  const int qrow = wq0 + n;
  const bool qvalid = qrow < td.row1;
  const int qrow_c = qvalid ? qrow : td.row1 - 1;

  const T* Q = (const T*)(suffix ? a.q_suf : a.q_pre);
  Frag qf[KK];
  {
    const T* qp = Q + ((size_t)(qrow_c + xq) * a.h_q + head) * D + 8 * hh;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qf[kk] = E::global_row(qp + 16 * kk, qvalid);
  }
  const int seg_q = suffix ? a.seg_start[qrow_c] : 0;
  const int seg_w_lo = (suffix && wave_active) ? a.seg_start[wq0] : 0;
  const int seg_w_hi = (suffix && wave_active) ? a.seg_start[wq1] : 0;

  // key segments: A = prefix keys, B = response keys
  const int kA0 = gi.p0, kA1 = suffix ? gi.p1 : td.row1;
  const int kB0 = suffix ? td.aux : 0, kB1 = suffix ? td.row1 : 0;
  const int nA = (kA1 - kA0 + BN - 1) / BN;
  const int nB = (kB1 - kB0 + BN - 1) / BN;
  const int ntiles = nA + nB;

  const T* Kp = (const T*)a.k_pre; const T* Vp = (const T*)a.v_pre;
  const T* Ks = (const T*)a.k_suf; const T* Vs = (const T*)a.v_suf;
  const int kvstride = a.h_kv * D;

  Stager<T, BN, D, kFwdThreads> ldk, ldv;
  ldk.init(kvstride, wave, lane);
  ldv.init(kvstride, wave, lane);
  FragOffsets<T, D> fo;
  fo.init(lane);
  auto issue = [&](int j, char* kdst, char* vdst) {
    const bool segA = j < nA;
    const int k0 = segA ? kA0 + j * BN : kB0 + (j - nA) * BN;
    const int kend = segA ? kA1 : kB1;
    const size_t kx = (size_t)(k0 + (segA ? xo_pre : xo_suf));
    const T* kb = (segA ? Kp : Ks) + kx * kvstride + kvh * D;
    const T* vb = (segA ? Vp : Vs) + kx * kvstride + kvh * D;
    ldk.load(kdst, kb, kvstride, kend - k0);
    ldv.load(vdst, vb, kvstride, kend - k0);
  };

  f32x16 acc_o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc_o[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  const float c = a.scale_log2;

  // one key tile: start the copy of tile j + 1 into (Kn, Vn), work on (Kt, Vt), publish
  auto step = [&](int j, const char* Kt, const char* Vt, char* Kn, char* Vn) {
    if (j + 1 < ntiles) issue(j + 1, Kn, Vn);
    const bool segA = j < nA;
    const int k0 = segA ? kA0 + j * BN : kB0 + (j - nA) * BN;
    const int kend = segA ? kA1 : kB1;
    // visibility of this key tile to this wave
    bool skip, full;
    const bool cross = segA && suffix;  // response queries x prefix keys: no causal mask
    if (cross) {
      skip = false;
      full = k0 + BN <= kend;
    } else {
      // causal (prefix self-attention, or responses inside a member)
      skip = k0 > wq1;
      if (!segA) skip = skip || (k0 + BN <= seg_w_lo);
      full = (k0 + BN - 1 <= wq0) && (k0 + BN <= kend);
      if (!segA) full = full && (k0 >= seg_w_hi);
    }
    if (wave_active && !skip) {
      f32x16 s[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        s[kb] = f32x16{};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
          s[kb] = E::mma(fo.row(Kt, 32 * kb, kk), qf[kk], s[kb]);
      }
      // Mask, only on tiles that straddle a boundary (a real branch: the empty asm keeps
      // the compiler from turning it into selects executed on every tile). Key offset
      // o = 32kb + 8(r/4) + r%4 of register r is a compile-time constant; the lane's
      // visible offsets are [lo, hi).
      if (!full) {
        asm volatile("");
        const int base = k0 + 4 * hh;
        int hi = kend - base;
        if (!cross) hi = min(hi, qrow_c + 1 - base);
        const int lo = segA ? -(1 << 30) : seg_q - base;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int o = 32 * kb + 8 * (r >> 2) + (r & 3);
            s[kb][r] = ((o >= lo) & (o < hi)) ? s[kb][r] : -INFINITY;
          }
      }
      float tmax = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, s[kb][r]);
      tmax = wave_swap32_max(tmax) * c;  // c > 0: max(c*s) = c*max(s)
      // Lazy running max: a row keeps its max until a tile exceeds it by more than
      // 2^8, so most tiles need no rescale of O (p <= 256 is harmless in fp32/bf16;
      // the log-sum-exp is exact for any choice of m).
      const float m_new = (tmax > m_run + 8.f) ? tmax : m_run;
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      float psum = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = fast_exp2(fmaf(s[kb][r], c, -m_use));
          s[kb][r] = p;
          psum += p;
        }
      }
      if (__any(m_new != m_run)) {
        const float alpha = fast_exp2(m_run - m_use);
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) acc_o[db] *= alpha;
      }
      l_run += psum;
      m_run = m_new;
      // O^T += V^T P^T over the 64 keys (4 k steps of 16)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const Frag pf = E::acc_to_frag(s[t >> 1], t & 1);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const Frag vf = fo.tr(Vt, t, db);
          acc_o[db] = E::mma(vf, pf, acc_o[db]);
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

  if (!wave_active) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = 1.f / l_tot;
  if (qvalid) {
    T* O = (T*)(suffix ? a.o_suf : a.o_pre);
    T* op = O + ((size_t)(qrow + xq) * a.h_q + head) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d0 = 32 * db + 8 * i + 4 * hh;
        E::store4(op + d0, acc_o[db][4 * i] * inv, acc_o[db][4 * i + 1] * inv, acc_o[db][4 * i + 2] * inv,
                  acc_o[db][4 * i + 3] * inv);
      }
    if (hh == 0) {
      const float lse = (m_run + fast_log2(l_tot)) * kLn2;
      float* L = suffix ? a.lse_suf : a.lse_pre;
      const int ld = a.xl ? a.total_prefix + a.total_suffix : (suffix ? a.total_suffix : a.total_prefix);
      L[(size_t)head * ld + qrow + xq] = lse;
    }
  }
}

}  // namespace pg
