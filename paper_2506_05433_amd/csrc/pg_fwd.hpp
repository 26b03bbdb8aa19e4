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
// the row-major LDS tile through transposing reads. The leading tiles that every row
// of the workgroup sees run software-pipelined (the scores of tile j+1 are computed
// next to the exponentials of tile j); the rest take the masked path.
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
__global__ void __launch_bounds__(kFwdThreads, 2) fwd_kernel(const FwdArgs a) {
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
  // source rows of key tile j: (pointer to its first row of this kv head, valid rows)
  auto tile_src = [&](int j, const T* pre, const T* suf, int& rows) {
    const bool segA = j < nA;
    const int k0 = segA ? kA0 + j * BN : kB0 + (j - nA) * BN;
    rows = (segA ? kA1 : kB1) - k0;
    return (segA ? pre : suf) + (size_t)(k0 + (segA ? xo_pre : xo_suf)) * kvstride + kvh * D;
  };
  auto issue_k = [&](int j, char* kdst) {
    int rows;
    const T* src = tile_src(j, Kp, Ks, rows);
    ldk.load(kdst, src, kvstride, rows);
  };
  auto issue_v = [&](int j, char* vdst) {
    int rows;
    const T* src = tile_src(j, Vp, Vs, rows);
    ldv.load(vdst, src, kvstride, rows);
  };

  f32x16 acc_o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc_o[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  const float c = a.scale_log2;

  // S^T = K Q^T for one 64-key tile
  auto s_product = [&](const char* Kt, f32x16 (&s)[2]) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x16{};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) s[kb] = E::mma(fo.row(Kt, 32 * kb, kk), qf[kk], s[kb]);
    }
  };
  // Lazy running max of one tile's (masked) scores: a row keeps its max until a tile
  // exceeds it by more than 2^8, so most tiles need no rescale of O and l (p <= 256 is
  // harmless in fp32/bf16; the log-sum-exp is exact for any choice of m).
  auto tile_max = [&](const f32x16 (&s)[2]) {
    float tmax = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, s[kb][r]);
    tmax = wave_swap32_max(tmax) * c;  // c > 0: max(c*s) = c*max(s)
    const float m_new = (tmax > m_run + 8.f) ? tmax : m_run;
    if (__any(m_new != m_run)) {
      const float alpha = fast_exp2(m_run - ((m_new == -INFINITY) ? 0.f : m_new));
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) acc_o[db] *= alpha;
    }
    m_run = m_new;
  };
  // P = exp2(S*c - m) against the row's current max, l += rowsum(P), O^T += V^T P^T
  auto exp_pv = [&](f32x16 (&s)[2], const char* Vt) {
    const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
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
    l_run += psum;
    Frag pf[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) pf[t] = E::acc_to_frag(s[t >> 1], t & 1);
    // O^T += V^T P^T over the 64 keys (4 k steps of 16)
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int db = 0; db < DB; ++db) acc_o[db] = E::mma(fo.tr(Vt, t, db), pf[t], acc_o[db]);
  };

  // Tiles [0, nfull) are visible to every row of the workgroup (no mask, no skip): the
  // dense prefix of a response tile, and the prefix keys left of a prefix tile's
  // diagonal. They run software-pipelined: iteration j computes the scores of tile j + 1
  // while it exponentiates those of tile j and adds P V, with no branch in between, so
  // each wave interleaves matrix and vector instructions instead of alternating between
  // them (both waves of a SIMD meet at every barrier, so they would otherwise run the same
  // phase at the same time); the max of tile j + 1 and the rare rescale follow. K runs two
  // tiles ahead of V: iteration j reads K(j + 1) and V(j) and copies K(j + 2), V(j + 1).
  // The arithmetic is the same, in the same order, as for a boundary tile.
  const int nfull = suffix ? (kA1 - kA0) / BN : (td.row0 - kA0 + 1) / BN;
  // the remaining tiles: per-wave skip and masks at the boundaries
  auto step = [&](int j, const char* Kt, const char* Vt, char* Kn, char* Vn) {
    if (j + 1 < ntiles) {
      issue_k(j + 1, Kn);
      issue_v(j + 1, Vn);
    }
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
      s_product(Kt, s);
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
      tile_max(s);
      exp_pv(s, Vt);
    }
    if (j + 1 < ntiles) {
      ldk.store(Kn);
      ldv.store(Vn);
    }
    ldk.wait();
    __syncthreads();
  };
  auto pipe_step = [&](int j, f32x16 (&s_cur)[2], f32x16 (&s_nxt)[2], const char* Kt1, const char* Vt,
                       char* Kn2, char* Vn1) {
    const bool k2 = j + 2 <= nfull && j + 2 < ntiles, v1 = j + 1 < ntiles;
    if (k2) issue_k(j + 2, Kn2);
    if (v1) issue_v(j + 1, Vn1);
    if (wave_active) {
      // the scores of tile j + 1 (unused when j + 1 == nfull: the buffer then holds an
      // earlier tile or nothing, and the boundary loop recomputes them)
      s_product(Kt1, s_nxt);
      exp_pv(s_cur, Vt);
      if (j + 1 < nfull) tile_max(s_nxt);
    }
    if (k2) ldk.store(Kn2);
    if (v1) ldv.store(Vn1);
    ldk.wait();
    __syncthreads();
  };

  if (ntiles > 0) {
    issue_k(0, sK0);
    issue_v(0, sV0);
    ldk.store(sK0);
    ldv.store(sV0);
  }
  ldk.wait();
  __syncthreads();
  if (nfull > 0) {
    f32x16 sa[2], sb[2];
    const bool k1 = 1 < ntiles;
    if (k1) issue_k(1, sK1);
    if (wave_active) {
      s_product(sK0, sa);
      tile_max(sa);
    }
    if (k1) ldk.store(sK1);
    ldk.wait();
    __syncthreads();
    for (int j = 0; j < nfull; j += 2) {
      pipe_step(j, sa, sb, sK1, sV0, sK0, sV1);
      if (j + 1 < nfull) pipe_step(j + 1, sb, sa, sK0, sV1, sK1, sV0);
    }
  }
  for (int j = nfull; j < ntiles; ++j) {
    const bool odd = j & 1;
    step(j, odd ? sK1 : sK0, odd ? sV1 : sV0, odd ? sK0 : sK1, odd ? sV0 : sV1);
  }

  if (!wave_active) return;
  const float l_tot = wave_swap32_sum(l_run);
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
