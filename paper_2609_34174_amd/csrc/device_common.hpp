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
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 values as bf16 hi + lo pairs (v ~= hi + lo): hi rounds each value
// to bf16 (one packed conversion for the pair), its fp32 value is the packed
// word's upper or lower half moved into place, and lo rounds the exact
// remainder v - hi.  The same values as converting each element on its own,
// with one conversion per pair for each of hi and lo.
__device__ __forceinline__ void split2(float v0, float v1, bf16x2& hi, bf16x2& lo) {
  hi = __builtin_convertvector((f32x2){v0, v1}, bf16x2);
  const uint32_t hb = __builtin_bit_cast(uint32_t, hi);
  const float h0 = __builtin_bit_cast(float, hb << 16), h1 = __builtin_bit_cast(float, hb & 0xffff0000u);
  lo = __builtin_convertvector((f32x2){v0 - h0, v1 - h1}, bf16x2);
}
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef short i16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// A compile-time integer passed to a generic lambda (one instantiation per value).
template <int V>
struct IntC {
  static constexpr int value = V;
};

__device__ __forceinline__ f32x8 cat(f32x4 a, f32x4 b) {
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Logical k of slot e for the lane group q inside one 32-wide K step.
__device__ __forceinline__ int slot_k(int e, int q) { return 16 * (e >> 2) + 4 * q + (e & 3); }

// ---------------------------------------------------------------------------
// LDS tiles.  Every staged matrix lives in LDS row-major, unpadded, with its
// 4-element chunks XOR-swizzled by row:
//     element (r, k) of a [rows][K] tile is stored at
//     r*K + 4*((k/4) ^ swz(r)) + k%4,     swz(r) = 4*(r%4) + (r/4)%4.
// With 32 banks of 4 bytes, both fragment reads below touch 16 distinct
// 8-byte chunks per 16-lane group (no bank conflicts), and a 16-lane group
// writing one row's 16 chunks is conflict-free as well.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int swz(int r, int K) { return (((r & 3) << 2) | ((r >> 2) & 3)) & ((K >> 2) - 1); }
__device__ __forceinline__ int lds_off(int r, int k, int K) {
  return r * K + ((((k >> 2) ^ swz(r, K)) << 2) | (k & 3));
}

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// The lane-dependent part of the fragment addresses into a [rows][K] tile of
// ES-byte elements.  For a row block starting at a multiple of 16 the swizzle
// key of row row0 + (lane % 16) is the lane's own, and a 4-chunk step of the
// column changes the XORed chunk index by a constant: so every address of the
// fragment reads below is one of four per-lane byte offsets plus a
// compile-time constant.
//   n[j]: row lane%16, chunk (4j + q) ^ swz     (load_n halves, 4-element stores)
//   t[j]: row 4q + c/4, chunk (4j + c%4) ^ swz  (load_t halves)
// with q = lane / 16, c = lane % 16.  With PRE the offsets are computed once
// and pass through an empty asm statement, so the compiler can neither
// re-derive them per use from the lane nor hoist every derived address into
// a register of its own (8 registers per tile width); without PRE every
// address is formed from the lane where it is used.
template <int K, int ES, bool PRE>
struct LaneOff {
  static constexpr int NJ = K >= 64 ? 4 : K / 16;
  int n[PRE ? NJ : 1], t[PRE ? NJ : 1], lane;
  // Byte offset of element (row0 + c, k + 4q); row0 and k multiples of 16.
  __device__ __forceinline__ int nat(int row0, int k) const {
    if constexpr (!PRE) return lds_off(row0 + (lane & 15), k + 4 * (lane >> 4), K) * ES;
    const int kc = k >> 2;
    return (row0 * K + 4 * (kc & ~15)) * ES + sel(n, (kc >> 2) & 3);
  }
  // Byte offset of element (r0 + 4q + c/4, n0 + 4(c%4)); r0 and n0 multiples of 16.
  __device__ __forceinline__ int tat(int r0, int n0) const {
    if constexpr (!PRE) return lds_off(r0 + 4 * (lane >> 4) + ((lane & 15) >> 2), n0 + 4 * (lane & 3), K) * ES;
    const int kc = n0 >> 2;
    return (r0 * K + 4 * (kc & ~15)) * ES + sel(t, (kc >> 2) & 3);
  }
  // The same for a column known only at run time (wave-uniform): with PRE
  // the offset is formed once from the lane (no run-time index into the
  // arrays above, which would move them to scratch memory) and kept opaque.
  __device__ __forceinline__ int nat_rt(int row0, int k) const {
    if constexpr (!PRE) return nat(row0, k);
    const int kc = k >> 2, c = lane & 15, q = lane >> 4;
    int x = (row0 * K + 4 * (kc & ~15) + c * K + 4 * (((kc & 12) + q) ^ swz(c, K))) * ES;
    asm volatile("" : "+v"(x));
    return x;
  }
  __device__ __forceinline__ int tat_rt(int r0, int n0) const {
    if constexpr (!PRE) return tat(r0, n0);
    const int kc = n0 >> 2, c = lane & 15, q = lane >> 4;
    int x = (r0 * K + 4 * (kc & ~15) + (4 * q + (c >> 2)) * K + 4 * (((kc & 12) + (c & 3)) ^ swz(4 * q + (c >> 2), K))) * ES;
    asm volatile("" : "+v"(x));
    return x;
  }

 private:
  // v[j] by selects (j a compile-time constant wherever these are used).
  template <int N>
  __device__ static __forceinline__ int sel(const int (&v)[N], int j) {
    int x = v[0];
#pragma unroll
    for (int i = 1; i < N; ++i) x = j == i ? v[i] : x;
    return x;
  }
};
template <int K, int ES, bool PRE>
__device__ __forceinline__ LaneOff<K, ES, PRE> lane_off(int lane) {
  LaneOff<K, ES, PRE> o;
  o.lane = lane;
  if constexpr (PRE) {
    const int c = lane & 15, q = lane >> 4, sn = swz(c, K), st = swz(4 * q + (c >> 2), K);
#pragma unroll
    for (int j = 0; j < LaneOff<K, ES, PRE>::NJ; ++j) {
      o.n[j] = (c * K + 4 * ((4 * j + q) ^ sn)) * ES;
      o.t[j] = ((4 * q + (c >> 2)) * K + 4 * ((4 * j + (c & 3)) ^ st)) * ES;
      asm volatile("" : "+v"(o.n[j]), "+v"(o.t[j]));
    }
  }
  return o;
}
// The offsets of width K2 given those of width K1 (shared when equal).
template <int K2, int K1, int ES, bool PRE>
__device__ __forceinline__ LaneOff<K2, ES, PRE> lane_off_like(const LaneOff<K1, ES, PRE>& o) {
  if constexpr (K1 == K2) return o;
  else return lane_off<K2, ES, PRE>(o.lane);
}
template <class T>
__device__ __forceinline__ const T& at_byte(const void* base, int off) {
  return *reinterpret_cast<const T*>(static_cast<const char*>(base) + off);
}
template <class T>
__device__ __forceinline__ T* ptr_byte(void* base, int off) {
  return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}

// ---------------------------------------------------------------------------
// Operand policies.  load_n reads the fragment of row (row0 + c) of a tile
// with k along the tile's columns; load_t reads it with k along the tile's
// rows (the operand row index n0 + c is a tile column) - the hardware
// transposing read ds_read_b64_tr_b16 for bf16: inside each 16-lane group,
// lane 4a+b receives element b of the 8-byte rows addressed by lanes a, a+4,
// a+8, a+12, so lane i points at row k0 + 4q + i/4, columns n0 + 4(i%4).
// ---------------------------------------------------------------------------
struct OpBF16 {
  typedef bf16 elem;
  typedef bf16x8 frag;
  static constexpr int kSplit = 2;

  __device__ static __forceinline__ f32x4 mma(f32x4 acc, frag a, frag b) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
  }
  __device__ static __forceinline__ frag load_n(const elem* base, int K, int row0, int k0, int lane) {
    const int r = row0 + (lane & 15), k = k0 + 4 * (lane >> 4);
    const bf16x4 a = *reinterpret_cast<const bf16x4*>(base + lds_off(r, k, K));
    const bf16x4 b = *reinterpret_cast<const bf16x4*>(base + lds_off(r, k + 16, K));
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  }
  // load_n with reads the compiler keeps apart (volatile): it would otherwise
  // pair the first halves of two fragments into one two-address read and
  // then move each fragment's halves together.  Pays in the wide-map kernels
  // (LM-width MLP step -2.5 %); in the narrow scans the extra read
  // instructions and the fixed read order cost more than the moves saved.
  __device__ static __forceinline__ frag load_n_sep(const elem* base, int K, int row0, int k0, int lane) {
    const int r = row0 + (lane & 15), k = k0 + 4 * (lane >> 4);
    typedef const volatile __attribute__((address_space(3))) bf16x4 lds_v4;
    const bf16x4 a = *(lds_v4*)(base + lds_off(r, k, K));
    const bf16x4 b = *(lds_v4*)(base + lds_off(r, k + 16, K));
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  }
  __device__ static __forceinline__ frag load_t(const elem* base, int K, int k0, int n0, int lane) {
    const int c = lane & 15, r = k0 + 4 * (lane >> 4) + (c >> 2), n = n0 + 4 * (c & 3);
    const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + lds_off(r, n, K)));
    const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + lds_off(r + 16, n, K)));
    const i16x8 v = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(frag, v);
  }
  // The same reads from precomputed lane offsets (row0, k0, n0 multiples of
  // 16); tcol is the offset of a transposed read's column block chosen at
  // run time.
  template <int K, bool PRE>
  __device__ static __forceinline__ frag load_n(const elem* base, const LaneOff<K, 2, PRE>& L, int row0, int k0) {
    if constexpr (!PRE) return load_n(base, K, row0, k0, L.lane);
    const bf16x4 a = at_byte<bf16x4>(base, L.nat(row0, k0));
    const bf16x4 b = at_byte<bf16x4>(base, L.nat(row0, k0 + 16));
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  }
  __device__ static __forceinline__ frag tr_pair(const elem* base, int oa, int ob) {
    const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)((const char*)base + oa));
    const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)((const char*)base + ob));
    const i16x8 v = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(frag, v);
  }
  template <int K, bool PRE>
  __device__ static __forceinline__ frag load_t(const elem* base, const LaneOff<K, 2, PRE>& L, int k0, int n0) {
    if constexpr (!PRE) return load_t(base, K, k0, n0, L.lane);
    return tr_pair(base, L.tat(k0, n0), L.tat(k0 + 16, n0));
  }
  struct tcol {
    int off;
  };
  // (Without precomputed offsets tcol keeps the column and the address is
  // formed at the read.)
  template <int K, bool PRE>
  __device__ static __forceinline__ tcol make_tcol(const LaneOff<K, 2, PRE>& L, int n0) {
    if constexpr (PRE) return tcol{L.tat_rt(0, n0)};
    else return tcol{n0};
  }
  template <int K, bool PRE>
  __device__ static __forceinline__ frag load_t(const elem* base, const LaneOff<K, 2, PRE>& L, int k0, tcol col) {
    if constexpr (PRE) return tr_pair(base, k0 * K * 2 + col.off, (k0 + 16) * K * 2 + col.off);
    else return load_t(base, L, k0, col.off);
  }
  __device__ static __forceinline__ f32x8 to_f32(frag f) {
    f32x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (float)f[e];
    return v;
  }
  __device__ static __forceinline__ frag neg(frag f) {
    i16x8 v = __builtin_bit_cast(i16x8, f);
    v ^= (short)0x8000;
    return __builtin_bit_cast(frag, v);
  }
  // v ~= hi + lo, both bf16 (about 16 significant bits in total).
  __device__ static __forceinline__ void split(f32x8 v, frag& hi, frag& lo) {
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      bf16x2 h, l;
      split2(v[e], v[e + 1], h, l);
      hi[e] = h[0];
      hi[e + 1] = h[1];
      lo[e] = l[0];
      lo[e + 1] = l[1];
    }
  }
  // Store 4 consecutive elements (one chunk, 8 bytes).
  __device__ static __forceinline__ void store4(elem* p, f32x4 v) {
    bf16x4 o;
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = (bf16)v[r];
    *reinterpret_cast<bf16x4*>(p) = o;
  }
  __device__ static __forceinline__ void store4_split(elem* hi, elem* lo, f32x4 v) {
    bf16x4 h, l;
#pragma unroll
    for (int r = 0; r < 4; r += 2) {
      bf16x2 h2, l2;
      split2(v[r], v[r + 1], h2, l2);
      h[r] = h2[0];
      h[r + 1] = h2[1];
      l[r] = l2[0];
      l[r + 1] = l2[1];
    }
    *reinterpret_cast<bf16x4*>(hi) = h;
    *reinterpret_cast<bf16x4*>(lo) = l;
  }
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
  __device__ static __forceinline__ frag load_n(const elem* base, int K, int row0, int k0, int lane) {
    const int r = row0 + (lane & 15), k = k0 + 4 * (lane >> 4);
    const f32x4 a = *reinterpret_cast<const f32x4*>(base + lds_off(r, k, K));
    const f32x4 b = *reinterpret_cast<const f32x4*>(base + lds_off(r, k + 16, K));
    return cat(a, b);
  }
  __device__ static __forceinline__ frag load_n_sep(const elem* base, int K, int row0, int k0, int lane) {
    return load_n(base, K, row0, k0, lane);
  }
  __device__ static __forceinline__ frag load_t(const elem* base, int K, int k0, int n0, int lane) {
    const int c = lane & 15, q = lane >> 4;
    frag v;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = base[lds_off(k0 + slot_k(e, q), n0 + c, K)];
    return v;
  }
  template <int K, bool PRE>
  __device__ static __forceinline__ frag load_n(const elem* base, const LaneOff<K, 4, PRE>& L, int row0, int k0) {
    if constexpr (!PRE) return load_n(base, K, row0, k0, L.lane);
    return cat(at_byte<f32x4>(base, L.nat(row0, k0)), at_byte<f32x4>(base, L.nat(row0, k0 + 16)));
  }
  // fp32 transposed fragments are gathered element by element from the lane.
  template <int K, bool PRE>
  __device__ static __forceinline__ frag load_t(const elem* base, const LaneOff<K, 4, PRE>& L, int k0, int n0) {
    return load_t(base, K, k0, n0, L.lane);
  }
  struct tcol {
    int n0;
  };
  template <int K, bool PRE>
  __device__ static __forceinline__ tcol make_tcol(const LaneOff<K, 4, PRE>&, int n0) {
    return tcol{n0};
  }
  template <int K, bool PRE>
  __device__ static __forceinline__ frag load_t(const elem* base, const LaneOff<K, 4, PRE>& L, int k0, tcol col) {
    return load_t(base, K, k0, col.n0, L.lane);
  }
  __device__ static __forceinline__ f32x8 to_f32(frag f) { return f; }
  __device__ static __forceinline__ frag neg(frag f) { return -f; }
  __device__ static __forceinline__ void split(f32x8 v, frag& hi, frag& lo) {
    hi = v;
    lo = v;  // unused: kSplit == 1
  }
  __device__ static __forceinline__ void store4(elem* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
  __device__ static __forceinline__ void store4_split(elem* hi, elem* lo, f32x4 v) {
    (void)lo;
    *reinterpret_cast<f32x4*>(hi) = v;
  }
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

constexpr int cmax(int a, int b) { return a > b ? a : b; }

// ---------------------------------------------------------------------------
// Buffer addressing.  Streaming loads and stores of chunk data go through a
// raw buffer resource spanning one sequence's rows: an access at or past the
// resource's size reads zero / is dropped by the hardware, which masks the
// partial last chunk without a branch.  Branch-free memory operations keep
// the compiler's count of outstanding loads exact, so loads issued for later
// chunks stay in flight across the current chunk's barriers.
// ---------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
constexpr uint32_t kOOB = 0x80000000u;  // an offset past every resource (sizes are < 2^31)

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ bf16x4 buf_load4(rsrc_t r, uint32_t off, const bf16*) {
  return __builtin_bit_cast(bf16x4, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0));
}
__device__ __forceinline__ f32x4 buf_load4(rsrc_t r, uint32_t off, const float*) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}
__device__ __forceinline__ float buf_load1(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
}
// Cross-lane moves by DPP (a VALU operand modifier, no LDS round trip):
// lane i reads lane i - N (SHR) or i + N (SHL) of its 16-lane row, or of the
// whole wave (WAVE, N = 1), or lane (i + N) mod 16 of its row (ROR); lanes
// without a source get `fill`.
enum DppMove { kRowShr = 0x110, kRowShl = 0x100, kRowRor = 0x120, kWaveShr1 = 0x138, kWaveShl1 = 0x130 };
template <int CTRL>
__device__ __forceinline__ float dpp_move(float src, float fill) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, fill),
                                                               __builtin_bit_cast(int, src), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float lane_value(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
// Sum over each 16-lane row, in every lane of the row.
__device__ __forceinline__ float row_sum16(float x) {
  x += dpp_move<kRowRor + 8>(x, 0.f);
  x += dpp_move<kRowRor + 4>(x, 0.f);
  x += dpp_move<kRowRor + 2>(x, 0.f);
  x += dpp_move<kRowRor + 1>(x, 0.f);
  return x;
}
// Sum over the wave (the same value in every lane): the row sums added in
// row order.
__device__ __forceinline__ float wave_sum(float x) {
  x = row_sum16(x);
  return ((lane_value(x, 0) + lane_value(x, 16)) + lane_value(x, 32)) + lane_value(x, 48);
}

// Store cache policies.  Scan outputs are written once and read by later
// kernels only, so they are stored non-temporal at device scope (cache-policy
// bits SC1 | NT): the lines do not stay dirty in the XCD's L2, which otherwise
// has to be written back before the next kernel starts (about 15% of a scan
// step when measured).  A decode state small enough for the Infinity Cache
// keeps the default policy (the next step reads it back from there); larger
// ones are streamed too.
constexpr int kStoreStream = 16 | 2;
constexpr int kStoreDefault = 0;
template <int POLICY = kStoreStream>
__device__ __forceinline__ void buf_store4(rsrc_t r, uint32_t off, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, v), r, (int)off, 0, POLICY);
}
template <int POLICY = kStoreStream>
__device__ __forceinline__ void buf_store1(rsrc_t r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), r, (int)off, 0, POLICY);
}

// Whole-line output stores.  An accumulator tile stored as it lies writes 16
// rows x 64 bytes per instruction; streamed to HBM as half lines, such stores
// ran at about 70 % of the rate of stores that cover whole 128-byte lines.
// pair_rows takes two tiles over the same 16 rows and two adjacent 16-column
// blocks (lane (c, q): row c, columns 4q..4q+3 of each) and swaps halves
// between lanes c and c ^ 8 with a DPP row rotation by 8 (the bank mask picks
// the lanes that take the rotated value), so that lane (c, q) holds
//   a: row c & 7,       columns 16 (c >> 3) + 4q .. +3 of the 32-column pair,
//   b: row 8 + (c & 7), the same columns,
// and one store of a (or of b) covers 8 whole rows of 32 fp32.
template <int BANKS>  // 0x3: lanes c < 8 take the rotated value; 0xC: lanes c >= 8
__device__ __forceinline__ float dpp_ror8(float old, float src) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old),
                                                               __builtin_bit_cast(int, src), 0x128, 0xF, BANKS, false));
}
__device__ __forceinline__ void pair_rows(f32x4 t0, f32x4 t1, f32x4& a, f32x4& b) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    a[r] = dpp_ror8<0xC>(t0[r], t1[r]);  // lanes c >= 8 take tile 1's row c - 8
    b[r] = dpp_ror8<0x3>(t1[r], t0[r]);  // lanes c < 8 take tile 0's row c + 8
  }
}
// Byte offset, within a row-major fp32 matrix of `width` columns, of what
// pair_rows puts in `a` for the tiles at rows [row0, row0 + 16) and columns
// [col0, col0 + 32); `b` lies 8 rows further.
__device__ __forceinline__ uint32_t pair_off(int64_t row0, int col0, int width, int c, int q) {
  return (uint32_t)(((row0 + (c & 7)) * width + col0 + 16 * (c >> 3) + 4 * q) * 4);
}

}  // namespace gradlev
