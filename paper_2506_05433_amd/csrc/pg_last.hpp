// Forward of the final token of every member only: the multi-QA judge use of the
// shared-prefix layout (Section 2, "Further discussion"). A long response is the
// shared prefix, each short question is a member, and predictions are taken from
// the hidden state at each question's final token, so at the attention layer
// only those query rows are needed: the final row of [P; R_i] attends to the
// whole prefix and to its own question.
//
// MI355X layout of the work: for one group and one key/value head, the final
// queries of up to 128 (member, query head) pairs form one MFMA tile, so a staged
// prefix key/value tile serves every member and every head of the GQA group at
// once. With few queries and a long prefix that alone gives few workgroups, so
// the key stream of each member block is cut into `nch` contiguous chunks run by
// separate workgroups (flash-decoding); each writes its unnormalised output and
// its softmax state (running max, sum) and last_merge_kernel combines the chunks
// in chunk order (deterministic). The inner loop is the forward kernel's.
#pragma once
#include "pg_common.hpp"
#include "pg_plan.hpp"

namespace pg {

constexpr int kLastRows = 128;  // (member, head) rows per workgroup: 4 waves x 32
constexpr int kLastThreads = 256;
constexpr int kLastMaxChunks = 32;  // key chunks per member block (merged in one pass)

struct LastBlock {
  int group, m_first, m_count, pad;
};

struct LastArgs {
  const void *q_pre, *k_pre, *v_pre, *q_suf, *k_suf, *v_suf;
  void* o_last;     // [n_suffixes, h_q, D]
  float* lse_last;  // [h_q, n_suffixes]
  const int* cu_s;
  const PlanHeader* hdr;
  const GroupInfoEx* ginfo;
  const LastBlock* blocks;
  const int* n_blocks;
  float* part_o;   // [block][kv head][chunk][kLastRows][D] unnormalised outputs
  float* part_ml;  // [block][kv head][chunk][kLastRows][2] running max (log2 units) and sum
  int h_q, h_kv, ns, nch, nb_max, mpw;
  float scale_log2;
};

// Member blocks: group g's members in runs of at most mpw, groups in order (one block of
// kPlanThreads threads; groups processed in passes with a running offset).
__global__ void __launch_bounds__(kPlanThreads) plan_last_kernel(const PlanHeader* hdr, const GroupInfoEx* ginfo,
                                                                 int ng, int mpw, int nb_max, LastBlock* blocks,
                                                                 int* n_blocks) {
  __shared__ int tmp[kPlanThreads];
  __shared__ int carry;
  const int t = threadIdx.x;
  if (t == 0) carry = 0;
  __syncthreads();
  const bool ok = !hdr->error;
  for (int base = 0; base < ng; base += kPlanThreads) {
    const int g = base + t;
    const int members = (g < ng && ok) ? ginfo[g].m1 - ginfo[g].m0 : 0;
    const int nb = (members + mpw - 1) / mpw;
    const int inc = block_inclusive_scan<kPlanThreads>(nb, tmp);
    const int first = carry + inc - nb;
    for (int k = 0; k < nb; ++k) {
      if (first + k < nb_max) {
        LastBlock b;
        b.group = g;
        b.m_first = ginfo[g].m0 + k * mpw;
        b.m_count = min(mpw, members - k * mpw);
        b.pad = 0;
        blocks[first + k] = b;
      }
    }
    __syncthreads();
    if (t == kPlanThreads - 1) carry += inc;
    __syncthreads();
  }
  if (t == 0) *n_blocks = ok ? min(carry, nb_max) : 0;
}

template <typename T, int D>
__global__ void __launch_bounds__(kLastThreads, 2) last_kernel(const LastArgs a) {
  using E = Elt<T>;
  using Frag = typename E::Frag;
  constexpr int BN = 64;
  constexpr int KK = D / 16, DB = D / 32;
  constexpr int TILE = LdsTile<T, D>::bytes(BN);
  // two K/V buffers as distinct LDS objects, named statically by a loop unrolled by two (a
  // copy into one buffer then never makes reads of the other wait for it)
  __shared__ __attribute__((aligned(16))) char sK0[TILE], sV0[TILE], sK1[TILE], sV1[TILE];

  const BlockSlot slot = xcd_slot(blockIdx.x, a.h_kv, 1);
  const int unit = slot.unit, kvh = slot.head;
  const int b = unit / a.nch, chunk = unit - b * a.nch;
  if (b >= *a.n_blocks) return;
  const LastBlock blk = a.blocks[b];
  const GroupInfoEx gi = a.ginfo[blk.group];
  const int ratio = a.h_q / a.h_kv;
  const int rows = blk.m_count * ratio;

  const int tid = threadIdx.x, wave = uniform(tid >> 6), lane = tid & 63;
  const int n = lane & 31, hh = lane >> 5;
  const int r = 32 * wave + n;                      // this lane's (member, head) row
  const bool rvalid = r < rows;
  const int rc = rvalid ? r : 0;
  const int member = blk.m_first + rc / ratio, head = kvh * ratio + rc % ratio;
  const int ms0 = a.cu_s[member], ms1 = a.cu_s[member + 1];
  // the final token of [P; R_i]: the last response row, else the last prefix row
  const bool has_suf = ms1 > ms0, has_pre = gi.p1 > gi.p0;
  const bool qvalid = rvalid && (has_suf || has_pre);
  const T* qp = has_suf ? (const T*)a.q_suf + ((size_t)(ms1 - 1) * a.h_q + head) * D
                        : (const T*)a.q_pre + ((size_t)(has_pre ? gi.p1 - 1 : 0) * a.h_q + head) * D;
  Frag qf[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) qf[kk] = E::global_row(qp + 8 * hh + 16 * kk, qvalid);
  // the members whose rows this wave holds, and the response keys they see
  const int wr0 = 32 * wave, wr1 = min(32 * wave + 32, rows);
  const bool wave_active = wr0 < rows;
  const int wlo = wave_active ? a.cu_s[blk.m_first + wr0 / ratio] : 0;
  const int whi = wave_active ? a.cu_s[blk.m_first + (wr1 - 1) / ratio + 1] : 0;

  // key stream: the prefix (dense for every row), then the block's responses (own member only)
  const int kA0 = gi.p0, kA1 = gi.p1;
  const int kB0 = a.cu_s[blk.m_first], kB1 = a.cu_s[blk.m_first + blk.m_count];
  const int nA = (kA1 - kA0 + BN - 1) / BN, nB = (kB1 - kB0 + BN - 1) / BN;
  const int ntot = nA + nB;
  const int j0 = (int)((long)ntot * chunk / a.nch), j1 = (int)((long)ntot * (chunk + 1) / a.nch);

  const T* Kp = (const T*)a.k_pre; const T* Vp = (const T*)a.v_pre;
  const T* Ks = (const T*)a.k_suf; const T* Vs = (const T*)a.v_suf;
  const int kvstride = a.h_kv * D;
  Stager<T, BN, D, kLastThreads> ldk, ldv;
  ldk.init(kvstride, wave, lane);
  ldv.init(kvstride, wave, lane);
  FragOffsets<T, D> fo;
  fo.init(lane);
  auto issue = [&](int j, char* kdst, char* vdst) {
    const bool segA = j < nA;
    const int k0 = segA ? kA0 + j * BN : kB0 + (j - nA) * BN;
    const int kend = segA ? kA1 : kB1;
    ldk.load(kdst, (segA ? Kp : Ks) + (size_t)k0 * kvstride + kvh * D, kvstride, kend - k0);
    ldv.load(vdst, (segA ? Vp : Vs) + (size_t)k0 * kvstride + kvh * D, kvstride, kend - k0);
  };

  f32x16 acc_o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc_o[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  const float c = a.scale_log2;

  // one key tile: start the copy of tile j + 1 into (Kn, Vn), work on (Kt, Vt), publish
  auto step = [&](int j, const char* Kt, const char* Vt, char* Kn, char* Vn) {
    if (j + 1 < j1) issue(j + 1, Kn, Vn);
    const bool segA = j < nA;
    const int k0 = segA ? kA0 + j * BN : kB0 + (j - nA) * BN;
    const int kend = segA ? kA1 : kB1;
    const bool skip = !segA && (k0 >= whi || k0 + BN <= wlo);
    const bool full = segA && (k0 + BN <= kend);
    if (wave_active && !skip) {
      f32x16 s[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        s[kb] = f32x16{};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) s[kb] = E::mma(fo.row(Kt, 32 * kb, kk), qf[kk], s[kb]);
      }
      if (!full) {
        // visible key offsets [lo, hi) of the lane's row: the ragged end of the prefix, or its
        // own member's response keys
        asm volatile("");
        const int base = k0 + 4 * hh;
        const int lo = segA ? -(1 << 30) : ms0 - base;
        const int hi = segA ? kend - base : min(ms1, kend) - base;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int o = 32 * kb + 8 * (e >> 2) + (e & 3);
            s[kb][e] = ((o >= lo) & (o < hi)) ? s[kb][e] : -INFINITY;
          }
      }
      float tmax = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) tmax = fmaxf(tmax, s[kb][e]);
      tmax = wave_swap32_max(tmax) * c;
      const float m_new = (tmax > m_run + 8.f) ? tmax : m_run;
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      float psum = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = fast_exp2(fmaf(s[kb][e], c, -m_use));
          s[kb][e] = p;
          psum += p;
        }
      if (__any(m_new != m_run)) {
        const float alpha = fast_exp2(m_run - m_use);
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) acc_o[db] *= alpha;
      }
      l_run += psum;
      m_run = m_new;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const Frag pf = E::acc_to_frag(s[t >> 1], t & 1);
#pragma unroll
        for (int db = 0; db < DB; ++db) acc_o[db] = E::mma(fo.tr(Vt, t, db), pf, acc_o[db]);
      }
    }
    if (j + 1 < j1) {
      ldk.store(Kn);
      ldv.store(Vn);
    }
    ldk.wait();
    __syncthreads();
  };

  if (j1 > j0) {
    issue(j0, sK0, sV0);
    ldk.store(sK0);
    ldv.store(sV0);
  }
  ldk.wait();
  __syncthreads();
  for (int j = j0; j < j1; j += 2) {
    step(j, sK0, sV0, sK1, sV1);
    if (j + 1 < j1) step(j + 1, sK1, sV1, sK0, sV0);
  }

  if (!rvalid) return;
  const float l_tot = wave_swap32_sum(l_run);
  const size_t slotrow = ((size_t)((b * a.h_kv + kvh) * a.nch + chunk)) * kLastRows + r;
  float* po = a.part_o + slotrow * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d0 = 32 * db + 8 * i + 4 * hh;
      *(f32x4*)(po + d0) = f32x4{acc_o[db][4 * i], acc_o[db][4 * i + 1], acc_o[db][4 * i + 2], acc_o[db][4 * i + 3]};
    }
  if (hh == 0) {
    a.part_ml[2 * slotrow] = m_run;
    a.part_ml[2 * slotrow + 1] = l_tot;
  }
}

// Combines the chunks of one (member block, kv head) in chunk order and writes o_last and
// lse_last: with M the largest chunk max, o = sum_c 2^(m_c - M) o_c / sum_c 2^(m_c - M) l_c.
// A row whose sequence is empty (no prefix, no response) gets o = 0 and lse = -inf.
// One thread per (row, 4 output columns), kMergeThreads / (D/4) rows per workgroup, so the
// merge of even a single member block spreads over hundreds of workgroups; the threads of a
// row each recompute its (M, L) from the same cached chunk states.
constexpr int kMergeThreads = 128;
template <int D>
constexpr int merge_groups() { return kLastRows / (kMergeThreads / (D / 4)); }  // row groups per block

template <typename T, int D>
__global__ void __launch_bounds__(kMergeThreads) last_merge_kernel(const LastArgs a) {
  constexpr int Q = D / 4;                 // float4 groups per row
  constexpr int RPW = kMergeThreads / Q;   // rows per workgroup
  constexpr int G = merge_groups<D>();
  const int bk = blockIdx.x / G, rg = blockIdx.x - bk * G;
  const int b = bk / a.h_kv, kvh = bk - b * a.h_kv;
  if (b >= *a.n_blocks) return;
  const LastBlock blk = a.blocks[b];
  const int ratio = a.h_q / a.h_kv;
  const int r = rg * RPW + (int)threadIdx.x / Q, q = (int)threadIdx.x % Q;
  if (r >= blk.m_count * ratio) return;
  const size_t first = (size_t)(b * a.h_kv + kvh) * a.nch * kLastRows + r;  // slot row of chunk 0
  // Every chunk's state and output block is loaded up front (the loops run over the fixed
  // maximum with clamped indices, so all loads are in flight together); chunks past nch get
  // max -inf and weight 0, which leaves the sums unchanged.
  const int last = a.nch - 1;
  float mc[kLastMaxChunks], lc[kLastMaxChunks];
#pragma unroll
  for (int ch = 0; ch < kLastMaxChunks; ++ch) {
    const size_t sr = first + (size_t)min(ch, last) * kLastRows;
    mc[ch] = ch <= last ? a.part_ml[2 * sr] : -INFINITY;
    lc[ch] = a.part_ml[2 * sr + 1];
  }
  float M = -INFINITY;
#pragma unroll
  for (int ch = 0; ch < kLastMaxChunks; ++ch) M = fmaxf(M, mc[ch]);
  float L = 0.f;
  if (M != -INFINITY) {
#pragma unroll
    for (int ch = 0; ch < kLastMaxChunks; ++ch) L += lc[ch] * fast_exp2(mc[ch] - M);
  }
  const float inv = (M == -INFINITY) ? 0.f : 1.f / L;
  f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ch = 0; ch < kLastMaxChunks; ++ch) {
    const size_t sr = first + (size_t)min(ch, last) * kLastRows;
    const float w = (M == -INFINITY) ? 0.f : fast_exp2(mc[ch] - M) * inv;
    o += w * *(const f32x4*)(a.part_o + sr * D + 4 * q);
  }
  const int member = blk.m_first + r / ratio, head = kvh * ratio + r % ratio;
  Elt<T>::store4((T*)a.o_last + ((size_t)member * a.h_q + head) * D + 4 * q, o[0], o[1], o[2], o[3]);
  if (q == 0) a.lse_last[(size_t)head * a.ns + member] = (M == -INFINITY) ? -INFINITY : (M + fast_log2(L)) * kLn2;
}

}  // namespace pg
