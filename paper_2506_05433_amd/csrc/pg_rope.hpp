// Rotary position embedding with grouped position ids: the step before the
// attention kernels (Algorithm 1 takes q and k already rotary-encoded).
//
// Position rule (Section 2, "Algorithm implementation", after Eq. (4)): a token
// keeps the position it has in the Repeated-Prefix Forward, so prefix row t of
// a group is at t and row j of any member's response is at P + j. Positions are
// derived in the kernel from the grouping arrays; no position tensor is built.
//
// One workgroup per packed row rotates every head of q and of k on that row:
// the row's rotary_dim / 2 angles are computed once, in float64 (positions run
// to tens of thousands of radians, where a float32 angle would be off by up to
// ~1e-3), and kept in LDS as float32 cos / sin for all heads. The work is a
// streaming read and write of q and k, so the kernel is HBM-bound; rows are
// read and written in 16-byte (bf16) or 32-byte (fp32) chunks of 8 elements.
#pragma once
#include "pg_common.hpp"
#include "pg_plan.hpp"

namespace pg {

enum : int { kRopeInverse = 1, kRopeInterleaved = 2 };

struct RopeArgs {
  const int* cu_p;
  const int* cu_s;
  const PlanHeader* hdr;
  const GroupInfoEx* ginfo;
  int ng, ns, tp, ts;
  int h_q, h_kv, rot, flags;
  double log2_base;
  const void* src[4];  // q_pre, q_suf, k_pre, k_suf
  void* dst[4];
  int* pos_out[2];     // positions mode: pos_pre, pos_suf
};

constexpr int kRopeThreads = 256;

// Position of packed row `row` (the prefix rows of all groups, then all response rows).
__device__ inline int grouped_position(const RopeArgs& a, int row) {
  if (row < a.tp) {
    const int g = upper_index(a.cu_p, 0, a.ng, row);  // the last group starting at or before row
    return row - a.cu_p[g];
  }
  const int s = row - a.tp;
  const int m = upper_index(a.cu_s, 0, a.ns, s);
  int lo = 0, hi = a.ng;  // the group of member m: the last group whose members start at or before m
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (a.ginfo[mid].m0 <= m) lo = mid; else hi = mid;
  }
  return (a.ginfo[lo].p1 - a.ginfo[lo].p0) + (s - a.cu_s[m]);
}

template <typename T>
struct Chunk8;
template <>
struct Chunk8<bf16> {
  __device__ __forceinline__ static void load(const bf16* p, float (&x)[8]) {
    const bf16x8 v = *(const bf16x8*)p;
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = (float)v[e];
  }
  __device__ __forceinline__ static void store(bf16* p, const float (&x)[8]) {
    bf16x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (bf16)x[e];
    *(bf16x8*)p = v;
  }
};
template <>
struct Chunk8<float> {
  __device__ __forceinline__ static void load(const float* p, float (&x)[8]) {
    const f32x4 u = *(const f32x4*)p, w = *(const f32x4*)(p + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) { x[e] = u[e]; x[4 + e] = w[e]; }
  }
  __device__ __forceinline__ static void store(float* p, const float (&x)[8]) {
    *(f32x4*)p = f32x4{x[0], x[1], x[2], x[3]};
    *(f32x4*)(p + 4) = f32x4{x[4], x[5], x[6], x[7]};
  }
};

template <typename T, int D>
__global__ void __launch_bounds__(kRopeThreads) rope_kernel(const RopeArgs a) {
  __shared__ float s_cos[D / 2], s_sin[D / 2];
  if (a.hdr->error) return;
  const int row = blockIdx.x;
  const int pos = grouped_position(a, row);
  const int half = a.rot / 2;
  const bool inverse = a.flags & kRopeInverse;
  const bool inter = a.flags & kRopeInterleaved;
  for (int i = threadIdx.x; i < half; i += kRopeThreads) {
    const double ang = (double)pos * exp2(-2.0 * (double)i / (double)a.rot * a.log2_base);
    double sn, cs;
    sincos(ang, &sn, &cs);
    s_cos[i] = (float)cs;
    s_sin[i] = (float)(inverse ? -sn : sn);
  }
  __syncthreads();

  const bool pre = row < a.tp;
  const int r = pre ? row : row - a.tp;
  // work items of one head, in 8-element chunks: rotated chunks (half-split: chunk c with its
  // partner c + half/8; interleaved: 4 pairs) then the pass-through tail
  const int n_rot = inter ? a.rot / 8 : half / 8;
  const int per_head = n_rot + (D - a.rot) / 8;
  const int items = (a.h_q + a.h_kv) * per_head;
  for (int it = threadIdx.x; it < items; it += kRopeThreads) {
    const int head = it / per_head, c = it - head * per_head;
    const bool is_q = head < a.h_q;
    const int h = is_q ? head : head - a.h_q, nh = is_q ? a.h_q : a.h_kv;
    const int t = (is_q ? 0 : 2) + (pre ? 0 : 1);
    const size_t off = ((size_t)r * nh + h) * D;
    const T* src = (const T*)a.src[t] + off;
    T* dst = (T*)a.dst[t] + off;
    float x[8], y[8];
    if (c >= n_rot) {  // dimensions past rotary_dim: copied unchanged
      const int e0 = a.rot + 8 * (c - n_rot);
      Chunk8<T>::load(src + e0, x);
      Chunk8<T>::store(dst + e0, x);
    } else if (inter) {  // pairs (2i, 2i+1), i = 4c .. 4c+3
      Chunk8<T>::load(src + 8 * c, x);
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const float cs = s_cos[4 * c + p], sn = s_sin[4 * c + p];
        y[2 * p] = x[2 * p] * cs - x[2 * p + 1] * sn;
        y[2 * p + 1] = x[2 * p + 1] * cs + x[2 * p] * sn;
      }
      Chunk8<T>::store(dst + 8 * c, y);
    } else {  // pairs (i, i + half), i = 8c .. 8c+7
      Chunk8<T>::load(src + 8 * c, x);
      Chunk8<T>::load(src + half + 8 * c, y);
      float u[8], w[8];
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        const float cs = s_cos[8 * c + p], sn = s_sin[8 * c + p];
        u[p] = x[p] * cs - y[p] * sn;
        w[p] = y[p] * cs + x[p] * sn;
      }
      Chunk8<T>::store(dst + 8 * c, u);
      Chunk8<T>::store(dst + half + 8 * c, w);
    }
  }
}

// Positions only: pos_pre [total_prefix], pos_suf [total_suffix].
__global__ void __launch_bounds__(256) positions_kernel(const RopeArgs a) {
  if (a.hdr->error) return;
  const int row = blockIdx.x * 256 + threadIdx.x;
  if (row >= a.tp + a.ts) return;
  const int pos = grouped_position(a, row);
  if (row < a.tp) a.pos_out[0][row] = pos;
  else a.pos_out[1][row - a.tp] = pos;
}

}  // namespace pg
