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

#include "pg_types.hpp"

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

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// wave-uniform value held in a scalar register
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// The value of lane l and of lane l ^ 32, through gfx950's v_permlane32_swap (a VALU
// exchange of the two half-waves; no LDS round trip, no wait on other LDS traffic).
// With both operands equal to v, one result holds v of this lane's half and the other
// v of the opposite half, on every lane.
__device__ __forceinline__ void swap_halves(float v, float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}
__device__ __forceinline__ float wave_swap32_max(float v) {
  float a, b;
  swap_halves(v, a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float wave_swap32_sum(float v) {
  float a, b;
  swap_halves(v, a, b);
  return a + b;
}

// ---------------------------------------------------------------- LDS tile addressing
// A tile is `rows` rows of D elements, row-major. bf16 rows are padded by 64 bytes
// (four 16-byte chunks) and the low two bits of each chunk index are XORed with
// (row >> 2) & 3. On the 64 x 4-byte LDS banks this keeps both access patterns of the
// kernels free of conflicts:
//  * row-fragment reads (ds_read_b128): 16 lanes read one chunk of 16 consecutive rows;
//    the pad spreads rows 4 apart by four bank groups and the XOR separates the rows
//    that wrap around;
//  * transposing reads (ds_read_b64_tr_b16): 32 lanes read 4 consecutive chunks (one
//    aligned group of 4) of 4 consecutive rows (starting at a multiple of 4).
// Because the XOR only touches the low two chunk bits and repeats every 16 rows, the
// offset of a fragment is a per-lane base plus compile-time multiples of 64 bytes and
// of 16 rows, which the LDS instructions take as immediates. fp32 tiles keep a 16-byte
// row pad instead.
template <typename T, int D>
struct LdsTile {
  static constexpr int kRowBytes = D * (int)sizeof(T);
  static constexpr int kChunks = kRowBytes / 16;
  static constexpr bool kSwizzle = sizeof(T) == 2;
  static constexpr int kPitch = kSwizzle ? kRowBytes + 64 : kRowBytes + 16;
  __device__ __forceinline__ static int swz(int row) { return kSwizzle ? ((row >> 2) & 3) : 0; }
  // byte offset of 16-byte chunk `chunk` of row `row`
  __device__ __forceinline__ static int chunk_off(int row, int chunk) {
    return row * kPitch + 16 * (chunk ^ swz(row));
  }
  // byte offset of element `col` of row `row` (any element inside a chunk)
  __device__ __forceinline__ static int elem_off(int row, int col) {
    const int b = col * (int)sizeof(T);
    return chunk_off(row, b >> 4) + (b & 15);
  }
  static constexpr int bytes(int rows) { return rows * kPitch; }
};

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
  // the 8 elements [8*half8, 8*half8+8) of row `row` (one 16-byte chunk)
  template <int D>
  __device__ __forceinline__ static Frag lds_row(const char* tile, int row, int chunk) {
    return *(const Frag*)(tile + LdsTile<bf16, D>::chunk_off(row, chunk));
  }
  // Transposed operand from a row-major tile: element s of the result is
  // tile[row(s)][col] with row(s) = base_row + 4h + (s & 3) + 8 (s >> 2) and
  // col = base_col + l%32. ds_read_b64_tr_b16 works on groups of 16 lanes: lane i of
  // a group receives element i%4 of the 8-byte rows addressed by lanes 4v + i/4,
  // v = 0..3, so lane j of the group addresses row base_row + 4h + j/4 at column
  // base_col + 16 g16 + 4 (j%4) and gets column base_col + 16 g16 + i of 4 rows.
  template <int D>
  __device__ __forceinline__ static Frag lds_tr(const char* tile, int base_row, int base_col, int lane) {
    using L = LdsTile<bf16, D>;
    const int g16 = (lane & 31) >> 4, j = lane & 15, h = lane >> 5;
    const int row = base_row + 4 * h + (j >> 2);
    const int col = base_col + 16 * g16 + 4 * (j & 3);
    const char* p0 = tile + L::elem_off(row, col);
    const char* p1 = tile + L::elem_off(row + 8, col);
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
  __device__ __forceinline__ static float frag_elem(const Frag& f, int e) { return (float)f[e]; }
  __device__ __forceinline__ static Frag to_frag(const float (&v)[8]) {
    Frag f;
#pragma unroll
    for (int s = 0; s < 8; ++s) f[s] = (bf16)v[s];
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
  template <int D>
  __device__ __forceinline__ static Frag lds_row(const char* tile, int row, int chunk) {
    // `chunk` counts 8-element groups (32 bytes for fp32)
    const char* p = tile + LdsTile<float, D>::elem_off(row, 8 * chunk);
    f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 16);
    Frag f;
    f.v[0] = a[0]; f.v[1] = a[1]; f.v[2] = a[2]; f.v[3] = a[3];
    f.v[4] = b[0]; f.v[5] = b[1]; f.v[6] = b[2]; f.v[7] = b[3];
    return f;
  }
  template <int D>
  __device__ __forceinline__ static Frag lds_tr(const char* tile, int base_row, int base_col, int lane) {
    const int h = lane >> 5;
    const int col = base_col + (lane & 31);
    Frag f;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int row = base_row + 4 * h + (s & 3) + 8 * (s >> 2);
      f.v[s] = *(const float*)(tile + LdsTile<float, D>::elem_off(row, col));
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
  __device__ __forceinline__ static float frag_elem(const Frag& f, int e) { return f.v[e]; }
  __device__ __forceinline__ static Frag to_frag(const float (&v)[8]) {
    Frag f;
#pragma unroll
    for (int s = 0; s < 8; ++s) f.v[s] = v[s];
    return f;
  }
  __device__ __forceinline__ static void store4(float* p, float a, float b, float c, float d) {
    *(f32x4*)p = f32x4{a, b, c, d};
  }
};

// Cooperative copy of ROWS rows of D elements (global row stride `gstride` elements)
// into an LDS tile laid out by LdsTile<T, D>, in two phases (load to registers, store
// to LDS) so the caller can overlap the global latency with compute. Loads go through
// a buffer resource whose range ends after the last valid row: rows past the end read
// as zeros with no per-row test. Thread tid owns 16-byte chunk tid % C of rows
// tid / C + i * (NT / C); its global and LDS offsets are affine in i (the swizzle
// repeats every 16 rows), so they are computed once.
// Byte range of a tile's buffer resource: only the rows the tile holds (at most `rows`)
// count, so the range stays far below 2^31 whatever the length of the sequence behind
// them; the host bounds h * head_dim so that rows * row_bytes does too. Reads past the
// range return zeros, which is how ragged tiles and padding lanes are filled. The value is
// uniform at every call site; readfirstlane keeps it in a scalar register (a per-lane value
// would make the compiler wrap each buffer load in a loop over distinct descriptors).
__device__ __forceinline__ int range_bytes(int valid_rows, int rows, int row_bytes) {
  const int r = valid_rows < rows ? (valid_rows > 0 ? valid_rows : 0) : rows;
  return __builtin_amdgcn_readfirstlane(r * row_bytes);
}

template <typename T, int ROWS, int D, int NT>
struct TileLoader {
  static constexpr int kChunks = D * (int)sizeof(T) / 16;  // 16-byte chunks per row
  static constexpr int kTotal = ROWS * kChunks;
  static constexpr bool kPartial = kTotal < NT;              // fewer chunks than threads
  static constexpr int kPer = kPartial ? 1 : kTotal / NT;
  static constexpr int kRowStep = kPartial ? ROWS : NT / kChunks;  // rows between a thread's chunks
  static_assert((kPartial || (kTotal % NT == 0 && NT % kChunks == 0)) &&
                    (!LdsTile<T, D>::kSwizzle || kPer == 1 || kRowStep % 16 == 0),
                "tile/threads mismatch");
  uint4 reg[kPer];
  int goff, loff, gstep;
  bool active;
  __device__ __forceinline__ void init(int gstride, int wave, int lane) {
    const int tid = 64 * wave + lane;
    const int r = tid / kChunks, k = tid % kChunks;
    active = !kPartial || tid < kTotal;
    gstep = kRowStep * gstride * (int)sizeof(T);
    goff = r * gstride * (int)sizeof(T) + 16 * k;
    loff = LdsTile<T, D>::chunk_off(r, k);
  }
  __device__ __forceinline__ void load(char* /*lds*/, const T* base, int gstride, int valid_rows) {
    const int bytes = range_bytes(valid_rows, ROWS, gstride * (int)sizeof(T));
    __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, bytes, 0x00020000);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      if (active) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(rs, goff + i * gstep, 0, 0);
        reg[i] = __builtin_bit_cast(uint4, v);
      }
    }
  }
  __device__ __forceinline__ void store(char* lds) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i)
      if (active) *(uint4*)(lds + loff + i * kRowStep * LdsTile<T, D>::kPitch) = reg[i];
  }
  __device__ __forceinline__ void wait() const {}
};

// bf16 tiles are copied global -> LDS directly (buffer_load ... lds, 16 bytes per lane): no
// registers are held and no LDS store is issued. One wave instruction fills 1 KiB of LDS
// starting at the address given for the whole wave, lane i writing bytes [16i, 16i+16), so
// each lane fetches the global chunk that belongs at its LDS position in the padded,
// swizzled layout; lanes that land on row padding (and rows past the end) fetch from beyond
// the buffer's range and store zeros. wait() must precede the barrier that publishes the tile.
// 16 bytes per lane from a buffer into LDS at `lds` + 16 * lane (lds is wave-uniform).
// The builtin only exists for the device; the host pass of this file sees an empty body
// (it would otherwise drop the host launch stubs of some kernels that use it).
__device__ __forceinline__ void lds_dma16(__amdgpu_buffer_rsrc_t rs, char* lds, int voff) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds, 16, voff, 0, 0, 0);
#endif
}

template <int ROWS, int D, int NWAVES>
struct DirectLoader {
  using L = LdsTile<bf16, D>;
  static constexpr int kBytes = ROWS * L::kPitch;
  static constexpr int kInstr = kBytes / 1024;                       // wave instructions per tile
  static constexpr int kPerWave = (kInstr + NWAVES - 1) / NWAVES;
  static_assert(kBytes % 1024 == 0, "tile must be a whole number of KiB");
  static constexpr int kOutOfRange = 0x7ffffff0;
  int voff[kPerWave];
  int wave_;
  __device__ __forceinline__ void init(int gstride, int wave, int lane) {
    wave_ = wave;
#pragma unroll
    for (int k = 0; k < kPerWave; ++k) {
      const int p = 1024 * (wave + k * NWAVES) + 16 * lane;  // LDS byte this lane fills
      const int row = p / L::kPitch, pc = (p % L::kPitch) / 16;
      voff[k] = (pc < L::kChunks && p < kBytes) ? row * gstride * 2 + 16 * (pc ^ L::swz(row)) : kOutOfRange;
    }
  }
  __device__ __forceinline__ void load(char* lds, const bf16* base, int gstride, int valid_rows) {
    const int bytes = range_bytes(valid_rows, ROWS, gstride * 2);
    __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, bytes, 0x00020000);
#pragma unroll
    for (int k = 0; k < kPerWave; ++k) {
      const int w = wave_ + k * NWAVES;
      if (w < kInstr) lds_dma16(rs, lds + 1024 * w, voff[k]);
    }
  }
  __device__ __forceinline__ void store(char* /*lds*/) const {}
  __device__ __forceinline__ void wait() const { __builtin_amdgcn_s_waitcnt(0); }
};

// Stager<T, ROWS, D, NT>: the tile copier a kernel with NT threads uses for element type T.
template <typename T, int ROWS, int D, int NT>
struct StagerSel {
  using type = TileLoader<T, ROWS, D, NT>;
};
template <int ROWS, int D, int NT>
struct StagerSel<bf16, ROWS, D, NT> {
  using type = DirectLoader<ROWS, D, NT / 64>;
};
template <typename T, int ROWS, int D, int NT>
using Stager = typename StagerSel<T, ROWS, D, NT>::type;

// Per-lane LDS offsets of the MFMA operand fragments, computed once per kernel.
//   row(tile, row_base, kk)  : row fragment of row row_base + lane%32 (row_base a multiple
//                              of 16), elements 16 kk + 8 (lane/32) .. +8;
//   tr(tile, t, db)          : transposed fragment (see Elt::lds_tr) for rows 16 t .., and
//                              columns 32 db + lane%32.
// bf16 tiles keep the offsets in registers (the swizzle repeats every 16 rows, so row
// and k-step offsets become immediates); fp32 tiles compute them on the fly.
template <typename T, int D>
struct FragOffsets;

template <int D>
struct FragOffsets<bf16, D> {
  using E = Elt<bf16>;
  using L = LdsTile<bf16, D>;
  int row_[2];  // row fragment, k steps with kk even / odd (kk >> 1 adds 64 bytes)
  int tr_[2];   // transposed fragment, first / second 4-row read (d block adds 64 bytes)
  __device__ __forceinline__ void init(int lane) {
    const int n = lane & 31, hh = lane >> 5;
    const int g16 = (lane & 31) >> 4, j = lane & 15;
    row_[0] = L::chunk_off(n, hh);
    row_[1] = L::chunk_off(n, 2 + hh);
    tr_[0] = L::elem_off(4 * hh + (j >> 2), 16 * g16 + 4 * (j & 3));
    tr_[1] = L::elem_off(4 * hh + (j >> 2) + 8, 16 * g16 + 4 * (j & 3));
  }
  __device__ __forceinline__ E::Frag row(const char* tile, int row_base, int kk) const {
    return *(const E::Frag*)(tile + row_[kk & 1] + 64 * (kk >> 1) + row_base * L::kPitch);
  }
  __device__ __forceinline__ E::Frag tr(const char* tile, int t, int db) const {
    // address arithmetic in the LDS address space, so the constant part becomes the
    // instruction's offset field
    typedef __attribute__((address_space(3))) const char lds_char;
    lds_char* base = (lds_char*)tile;
    lds_char* p0 = base + tr_[0] + (64 * db + 16 * t * L::kPitch);
    lds_char* p1 = base + tr_[1] + (64 * db + 16 * t * L::kPitch);
    i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p0));
    i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p1));
    i16x8 ab = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(E::Frag, ab);
  }
};

template <int D>
struct FragOffsets<float, D> {
  using E = Elt<float>;
  int lane_;
  __device__ __forceinline__ void init(int lane) { lane_ = lane; }
  __device__ __forceinline__ E::Frag row(const char* tile, int row_base, int kk) const {
    return E::template lds_row<D>(tile, row_base + (lane_ & 31), 2 * kk + (lane_ >> 5));
  }
  __device__ __forceinline__ E::Frag tr(const char* tile, int t, int db) const {
    return E::template lds_tr<D>(tile, 16 * t, 32 * db, lane_);
  }
};

}  // namespace pg
