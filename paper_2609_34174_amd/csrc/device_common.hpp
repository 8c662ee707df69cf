// Device building blocks for the gfx950 scan kernels: MFMA fragment types,
// LDS fragment loads, fp32 -> bf16 hi/lo splitting, and chunk-tile staging.
//
// Matrix-core convention used throughout
// --------------------------------------
// Every contraction is written as D[r][c] += sum_k P[r][k] * Q[c][k] on
// 16x16 output tiles, with P and Q both "k-contiguous" (row-major in k).
// One K step covers 32 logical k values split into two 16-wide sub-blocks.
// Lane l of a wave is (c = l % 16, q = l / 16) and supplies, for row c of P
// (and row c of Q), the 8 values at
//     slot e -> k = 16 * (e / 4) + 4 * q + (e % 4).
// P and Q use the same slot -> k map, so the hardware's own assignment of
// lane/slot to k is irrelevant: a dot product is invariant under a common
// permutation of k.  The 16x16 fp32 accumulator holds D[4q + r][c] in lane
// (c, q), slot r.  Hence an accumulator tile is itself a ready-made operand:
// tile D (rows k, cols x) supplies row x of an operand over one 16-k
// sub-block, i.e. a tile can be contracted over its row index without a trip
// through LDS.
//
// Two element types are supported:
//   bf16: one v_mfma_f32_16x16x32_bf16 per K step.  fp32 values that meet the
//         matrix core (fast-weight states, eta-scaled costates) are split
//         into hi + lo bf16 terms (two MFMAs), which keeps about 16 mantissa
//         bits; bf16 inputs are exact.
//   fp32: eight v_mfma_f32_16x16x4_f32 per K step (slot e is instruction e),
//         exact fp32 products.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gradlev {

typedef __bf16 bf16;
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

__device__ __forceinline__ f32x8 cat(f32x4 a, f32x4 b) {
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Logical k of slot e for the lane group q inside one 32-wide K step.
__device__ __forceinline__ int slot_k(int e, int q) { return 16 * (e >> 2) + 4 * q + (e & 3); }

// ---------------------------------------------------------------------------
// Operand policies
// ---------------------------------------------------------------------------
struct OpBF16 {
  typedef bf16 elem;
  typedef bf16x8 frag;
  static constexpr int kSplit = 2;

  __device__ static __forceinline__ f32x4 mma(f32x4 acc, frag a, frag b) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
  }
  // Fragment of row (row0 + c) of a k-contiguous LDS array, K step at k0.
  __device__ static __forceinline__ frag load(const elem* base, int ld, int row0, int k0, int lane) {
    const elem* p = base + (row0 + (lane & 15)) * ld + k0 + 4 * (lane >> 4);
    bf16x4 a = *reinterpret_cast<const bf16x4*>(p);
    bf16x4 b = *reinterpret_cast<const bf16x4*>(p + 16);
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  }
  __device__ static __forceinline__ f32x8 load_f32(const elem* base, int ld, int row0, int k0, int lane) {
    frag f = load(base, ld, row0, k0, lane);
    f32x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (float)f[e];
    return v;
  }
  __device__ static __forceinline__ frag round(f32x8 v) {
    frag f;
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = (bf16)v[e];
    return f;
  }
  // v ~= hi + lo, both bf16 (about 16 significant bits in total).
  __device__ static __forceinline__ void split(f32x8 v, frag& hi, frag& lo) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      bf16 h = (bf16)v[e];
      hi[e] = h;
      lo[e] = (bf16)(v[e] - (float)h);
    }
  }
  // Store 4 consecutive elements (8 bytes).
  __device__ static __forceinline__ void store4(elem* p, f32x4 v) {
    bf16x4 o;
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = (bf16)v[r];
    *reinterpret_cast<bf16x4*>(p) = o;
  }
  __device__ static __forceinline__ void store1(elem* p, float v) { *p = (bf16)v; }
};

struct OpF32 {
  typedef float elem;
  typedef f32x8 frag;
  static constexpr int kSplit = 1;

  __device__ static __forceinline__ f32x4 mma(f32x4 acc, frag a, frag b) {
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], acc, 0, 0, 0);
    return acc;
  }
  __device__ static __forceinline__ frag load(const elem* base, int ld, int row0, int k0, int lane) {
    const elem* p = base + (row0 + (lane & 15)) * ld + k0 + 4 * (lane >> 4);
    f32x4 a = *reinterpret_cast<const f32x4*>(p);
    f32x4 b = *reinterpret_cast<const f32x4*>(p + 16);
    return cat(a, b);
  }
  __device__ static __forceinline__ f32x8 load_f32(const elem* base, int ld, int row0, int k0, int lane) {
    return load(base, ld, row0, k0, lane);
  }
  __device__ static __forceinline__ frag round(f32x8 v) { return v; }
  __device__ static __forceinline__ void split(f32x8 v, frag& hi, frag& lo) {
    hi = v;
    lo = v;  // unused: kSplit == 1
  }
  __device__ static __forceinline__ void store4(elem* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
  __device__ static __forceinline__ void store1(elem* p, float v) { *p = v; }
};

// acc += P * Q where P is given as fp32 values (split when the op needs it).
template <class OP>
__device__ __forceinline__ f32x4 mma_split_a(f32x4 acc, const typename OP::frag& hi,
                                             const typename OP::frag& lo, const typename OP::frag& b) {
  acc = OP::mma(acc, hi, b);
  if constexpr (OP::kSplit == 2) acc = OP::mma(acc, lo, b);
  return acc;
}
template <class OP>
__device__ __forceinline__ f32x4 mma_split_b(f32x4 acc, const typename OP::frag& a,
                                             const typename OP::frag& hi, const typename OP::frag& lo) {
  acc = OP::mma(acc, a, hi);
  if constexpr (OP::kSplit == 2) acc = OP::mma(acc, a, lo);
  return acc;
}

// ---------------------------------------------------------------------------
// Chunk tile staging: a C x K tile of a row-major [T][K] global matrix, held
// in registers as 16-byte vectors while the previous chunk computes, then
// written to LDS row-major (k = column) and/or transposed (k = row).
// Rows at or beyond `rows` are zero-filled, which masks a partial chunk.
// ---------------------------------------------------------------------------
template <class OP, int C, int K, int NT>
struct TileRegs {
  typedef typename OP::elem elem;
  static constexpr int VE = 16 / (int)sizeof(elem);  // elements per vector
  static constexpr int NV = C * K / VE;               // vectors per tile
  static constexpr int PER = (NV + NT - 1) / NT;
  static_assert(K % VE == 0, "row width must hold whole vectors");
  uint4 v[PER];

  __device__ __forceinline__ void load(const elem* src, int rows, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = tid + i * NT;
      const int row = idx * VE / K;
      uint4 z = {0u, 0u, 0u, 0u};
      if (idx < NV && row < rows) z = *reinterpret_cast<const uint4*>(src + (int64_t)idx * VE);
      v[i] = z;
    }
  }
  __device__ __forceinline__ void clear() {
#pragma unroll
    for (int i = 0; i < PER; ++i) v[i] = uint4{0u, 0u, 0u, 0u};
  }
  // lds[row][col], row stride ld (elements; ld * sizeof(elem) multiple of 8).
  __device__ __forceinline__ void store_rows(elem* lds, int ld, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = tid + i * NT;
      if (idx >= NV) continue;
      const int row = idx * VE / K, col = idx * VE % K;
      elem* p = lds + row * ld + col;
      const uint2* s = reinterpret_cast<const uint2*>(&v[i]);
      reinterpret_cast<uint2*>(p)[0] = s[0];
      reinterpret_cast<uint2*>(p)[1] = s[1];
    }
  }
  // lds[col][row], row stride ld.
  __device__ __forceinline__ void store_cols(elem* lds, int ld, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = tid + i * NT;
      if (idx >= NV) continue;
      const int row = idx * VE / K, col = idx * VE % K;
      const elem* s = reinterpret_cast<const elem*>(&v[i]);
#pragma unroll
      for (int e = 0; e < VE; ++e) lds[(col + e) * ld + row] = s[e];
    }
  }
};

__device__ __forceinline__ int tri_row(int idx) {
  // Row tb of the idx-th lower-triangular tile (tb >= sb), row-major order.
  int tb = 0;
  while ((tb + 1) * (tb + 2) / 2 <= idx) ++tb;
  return tb;
}

constexpr int cmax(int a, int b) { return a > b ? a : b; }

}  // namespace gradlev
