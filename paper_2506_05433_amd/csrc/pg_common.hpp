// Shared device helpers for the grouped-attention kernels (gfx950, wave64).
//
// Matrix products use the CDNA4 matrix cores through 32x32 output tiles:
//   bf16: v_mfma_f32_32x32x16_bf16 (one instruction per 16-wide k step),
//   fp32: v_mfma_f32_32x32x2_f32   (eight instructions per 16-wide k step).
// Operand convention for one 32x32 tile C[m][n] += sum_k A[m][k] B[k][n]:
//   lane l holds row m = l%32 of A and column n = l%32 of B; lane half
//   h = l/32 holds the eight k values 8h..8h+7 of a 16-wide k step;
//   accumulator register r of lane l holds C[8(r/4) + 4h + r%4][l%32].
// Any consistent relabelling of k inside a step is harmless because A and B
// use the same one; the kernels exploit that when a product's B operand is
// taken straight from a previous accumulator (see acc_to_frag).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pg {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Tile descriptor produced by the planner.
//  q tiles : kind 0 = prefix query rows [row0,row1) of group `group` (packed prefix index);
//            kind 1 = response query rows [row0,row1) (packed suffix index), which may span
//                     several members of the group; aux = first response key any row sees
//                     (start of the member that owns row0).
//  kv tiles: kind 0 = prefix keys [row0,row1); kind 1 = response keys [row0,row1);
//            aux = end of the response rows that can see them (end of the member owning row1-1).
struct TileDesc {
  int kind, group, row0, row1, aux, work, pad0, pad1;
};

// Per-group ranges: prefix rows [p0,p1), response rows [s0,s1).
struct GroupInfo {
  int p0, p1, s0, s1;
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

__device__ __forceinline__ float wave_swap32_max(float v) {
  return fmaxf(v, __shfl_xor(v, 32));
}

// ---------------------------------------------------------------- element traits
template <typename T>
struct Elt;

template <>
struct Elt<bf16> {
  using Frag = bf16x8;  // the 8 k values of one lane in a 16-wide k step
  static constexpr int kBytes = 2;
  __device__ __forceinline__ static f32x16 mma(const Frag& a, const Frag& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  // 8 consecutive elements at an LDS byte address (16-byte aligned)
  __device__ __forceinline__ static Frag lds_row(const char* p) { return *(const Frag*)p; }
  // transposed operand from a row-major LDS tile: element s of the result is
  // tile[row(s)][col] with row(s) = r0 + s (s<4) or r0 + 8 + (s-4) (s>=4), where
  // r0 = base_row + 4*h and col = base_col + l%32 (see the ds_read_tr16_b64 note).
  __device__ __forceinline__ static Frag lds_tr(const char* tile, int pitch, int base_row, int base_col, int lane) {
    const int g16 = (lane & 31) >> 4, j = lane & 15, h = lane >> 5;
    const int row = base_row + 4 * h + (j >> 2);
    const int col = base_col + 16 * g16 + 4 * (j & 3);
    const char* p0 = tile + row * pitch + col * 2;
    const char* p1 = p0 + 8 * pitch;
    i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p0));
    i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p1));
    // whole-vector shuffle + bit cast (element-wise bf16 inserts are lowered badly)
    i16x8 ab = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
    Frag f = __builtin_bit_cast(Frag, ab);
    return f;
  }
  // 8 consecutive elements from global memory (16-byte aligned), zero when !valid
  __device__ __forceinline__ static Frag global_row(const bf16* p, bool valid) {
    if (!valid) return Frag{};
    uint4 u = *(const uint4*)p;
    return __builtin_bit_cast(Frag, u);
  }
  // accumulator registers [8*half, 8*half+8) as the B operand of the next product
  __device__ __forceinline__ static Frag acc_to_frag(const f32x16& acc, int half) {
    Frag f;
#pragma unroll
    for (int s = 0; s < 8; ++s) f[s] = (bf16)acc[8 * half + s];
    return f;
  }
  __device__ __forceinline__ static void store4(bf16* p, float a, float b, float c, float d) {
    bf16x4 v = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
    *(bf16x4*)p = v;
  }
};

template <>
struct Elt<float> {
  struct Frag {
    float v[8];
  };
  static constexpr int kBytes = 4;
  __device__ __forceinline__ static f32x16 mma(const Frag& a, const Frag& b, f32x16 c) {
#pragma unroll
    for (int s = 0; s < 8; ++s) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v[s], b.v[s], c, 0, 0, 0);
    return c;
  }
  __device__ __forceinline__ static Frag lds_row(const char* p) {
    f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 16);
    Frag f;
    f.v[0] = a[0]; f.v[1] = a[1]; f.v[2] = a[2]; f.v[3] = a[3];
    f.v[4] = b[0]; f.v[5] = b[1]; f.v[6] = b[2]; f.v[7] = b[3];
    return f;
  }
  __device__ __forceinline__ static Frag lds_tr(const char* tile, int pitch, int base_row, int base_col, int lane) {
    const int h = lane >> 5;
    const int col = base_col + (lane & 31);
    Frag f;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int row = base_row + 4 * h + (s & 3) + 8 * (s >> 2);
      f.v[s] = *(const float*)(tile + row * pitch + col * 4);
    }
    return f;
  }
  __device__ __forceinline__ static Frag global_row(const float* p, bool valid) {
    Frag f;
    if (!valid) {
#pragma unroll
      for (int s = 0; s < 8; ++s) f.v[s] = 0.f;
      return f;
    }
    f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
    f.v[0] = a[0]; f.v[1] = a[1]; f.v[2] = a[2]; f.v[3] = a[3];
    f.v[4] = b[0]; f.v[5] = b[1]; f.v[6] = b[2]; f.v[7] = b[3];
    return f;
  }
  __device__ __forceinline__ static Frag acc_to_frag(const f32x16& acc, int half) {
    Frag f;
#pragma unroll
    for (int s = 0; s < 8; ++s) f.v[s] = acc[8 * half + s];
    return f;
  }
  __device__ __forceinline__ static void store4(float* p, float a, float b, float c, float d) {
    *(f32x4*)p = f32x4{a, b, c, d};
  }
};

// Cooperative copy of `rows` rows of D elements (global row stride `gstride` elements)
// into a row-major LDS tile with byte pitch `pitch`. Rows at or past `valid_rows` are
// zero-filled. Done in two phases (load to registers, store to LDS) so the caller can
// overlap the global latency with compute.
template <typename T, int ROWS, int D, int NT>
struct TileLoader {
  static constexpr int kChunks = D * (int)sizeof(T) / 16;  // 16-byte chunks per row
  static constexpr int kTotal = ROWS * kChunks;
  static constexpr int kPer = (kTotal + NT - 1) / NT;
  static_assert(kTotal % NT == 0, "tile must split evenly over the threads");
  uint4 reg[kPer];
  __device__ __forceinline__ void load(const T* base, int gstride, int valid_rows, int tid) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = tid + i * NT;
      const int r = c / kChunks, k = c % kChunks;
      if (r < valid_rows)
        reg[i] = *(const uint4*)((const char*)(base + (size_t)r * gstride) + 16 * k);
      else
        reg[i] = uint4{0u, 0u, 0u, 0u};
    }
  }
  __device__ __forceinline__ void store(char* lds, int pitch, int tid) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = tid + i * NT;
      const int r = c / kChunks, k = c % kChunks;
      *(uint4*)(lds + r * pitch + 16 * k) = reg[i];
    }
  }
};

}  // namespace pg
