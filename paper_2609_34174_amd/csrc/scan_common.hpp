// Pieces shared by the forward and backward scan kernels: kernel arguments,
// the block -> (sequence, segment) map, chunk-tile staging and the
// segment-aggregate kernel.
#pragma once

#include "../../include/gradlev.h"
#include "device_common.hpp"
#include "internal.hpp"

namespace gradlev {

struct KArgs {
  const float* W0;
  const void* X;
  const void* G;
  const void* dY;
  const float* eta;
  float eta_scalar;
  int64_t BH, H, T, seg_len, nseg;
  float* out0;   // fwd: Y
  float* aggA;   // [BH][nseg][m*d] write aggregates A_k (fwd: [m][d]; bwd: transposed [d][m])
  float* aggB;   // bwd: [BH][nseg][d][m] transposed dY x^T aggregates B_k (k >= 1)
  float* wend;   // fwd, or null: [BH][nsave][m][d] fast weights after each save_len-token block
  int64_t save_len, nsave;
  // Document resets (unit retention): reset [B][T] uint8, 1 where a document
  // starts.  cstate [BH][ceil(T/C)][d][m]: the forward stores the state at the
  // start of every chunk holding a reset there, transposed.  aggF
  // [BH][nseg][d][m]: the backward's full dY x^T per segment (for dW0; aggB
  // then holds the part before the segment's first reset).
  const uint8_t* reset;
  float* cstate;
  float* aggF;
  // With resets, or null: per work item (bh * nseg + seg) the aggregate pass
  // records the segment's last (forward) or first (backward) document start,
  // -1 for none, so that the main kernel need not search the flags again.
  int* segreset;
};

// ---------------------------------------------------------------------------
// Workgroups are dealt round-robin over the 8 XCDs of an MI355X by linear
// block id.  All segments of one sequence are mapped to the same XCD (block id
// congruent mod 8), so the segment aggregates a sequence exchanges stay in
// that XCD's L2.  Grid size: 8 * nseg * ceil(BH / 8); blocks past BH exit.
// ---------------------------------------------------------------------------
constexpr int kXCD = 8;

__host__ __device__ inline int64_t seg_grid(int64_t BH, int64_t nseg) {
  return kXCD * nseg * ((BH + kXCD - 1) / kXCD);
}

__device__ __forceinline__ bool map_block(int64_t BH, int64_t nseg, int64_t& bh, int64_t& seg) {
  const int64_t L = blockIdx.x;
  const int64_t r = L / kXCD;
  seg = r % nseg;
  bh = L % kXCD + kXCD * (r / nseg);
  return bh < BH;
}

// ---------------------------------------------------------------------------
// Chunk tile staging by 4x4 element blocks.  A C x K tile of a row-major
// [T][K] global matrix is held in registers (thread b owns rows 4*rb..4*rb+3
// and the 4-element chunk cb; consecutive threads take consecutive chunks of
// a row so the global loads coalesce) while earlier chunks compute, then
// written row by row into a swizzled LDS tile: a 16-lane group writes 16
// distinct chunks of one row.  The loads go through the sequence's buffer
// resource, so rows past the sequence end arrive as zero, which masks a
// partial chunk.  (Segments are whole chunks, so only the sequence end can
// cut a chunk.)
// ---------------------------------------------------------------------------
template <typename T>
struct Vec4;
template <>
struct Vec4<bf16> {
  typedef bf16x4 type;
};
template <>
struct Vec4<float> {
  typedef f32x4 type;
};

template <class OP, int C, int K, int NT>
struct Tile4 {
  typedef typename OP::elem elem;
  typedef typename Vec4<elem>::type vec4;
  static constexpr int NCB = K / 4, NB = (C / 4) * NCB, PER = (NB + NT - 1) / NT;
  vec4 v[PER][4];

  // Loads the chunk whose first row starts at byte `off` of `src`; with
  // off == kOOB the tile is zero and nothing is read.
  __device__ __forceinline__ void load(rsrc_t src, uint32_t off, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int b = tid + i * NT, rb = b / NCB, cb = b % NCB;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t o = (off == kOOB || b >= NB) ? kOOB : off + (uint32_t)(((4 * rb + k) * K + 4 * cb) * sizeof(elem));
        v[i][k] = buf_load4(src, o, (const elem*)nullptr);
      }
    }
  }
  __device__ __forceinline__ void store(elem* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int b = tid + i * NT, rb = b / NCB, cb = b % NCB;
      if (b >= NB) continue;
#pragma unroll
      for (int k = 0; k < 4; ++k) *reinterpret_cast<vec4*>(lds + lds_off(4 * rb + k, 4 * cb, K)) = v[i][k];
    }
  }
  // Store of s_row * value split into hi + lo tiles (one tile for fp32
  // operands), with per-row scale s_row = et[row].
  __device__ __forceinline__ void store_scaled(elem* hi, elem* lo, int tid, const float* et) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int b = tid + i * NT, rb = b / NCB, cb = b % NCB;
      if (b >= NB) continue;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float s = et[4 * rb + k];
        f32x4 f;
#pragma unroll
        for (int e = 0; e < 4; ++e) f[e] = (float)v[i][k][e] * s;
        const int o = lds_off(4 * rb + k, 4 * cb, K);
        OP::store4_split(hi + o, lo + o, f);
      }
    }
  }
};

// Chunk tile staging by 4-element row pieces: piece e = tid + i * NT holds
// row e / (K/4), columns 4 (e % (K/4)) .. +3.  Every thread of a wide
// workgroup takes a share of the tile (Tile4's 4x4 blocks occupy at most
// C K / 16 threads), so each holds fewer staging registers; consecutive
// threads still read consecutive global bytes.
template <class OP, int C, int K, int NT>
struct TileRow {
  typedef typename OP::elem elem;
  typedef typename Vec4<elem>::type vec4;
  static constexpr int NCB = K / 4, NE = C * NCB, PER = (NE + NT - 1) / NT;
  vec4 v[PER];

  __device__ __forceinline__ void load(rsrc_t src, uint32_t off, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = tid + i * NT, row = e / NCB, cb = e % NCB;
      const uint32_t o = (off == kOOB || e >= NE) ? kOOB : off + (uint32_t)((row * K + 4 * cb) * sizeof(elem));
      v[i] = buf_load4(src, o, (const elem*)nullptr);
    }
  }
  __device__ __forceinline__ void store(elem* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = tid + i * NT, row = e / NCB, cb = e % NCB;
      if (e >= NE) continue;
      *reinterpret_cast<vec4*>(lds + lds_off(row, 4 * cb, K)) = v[i];
    }
  }
  __device__ __forceinline__ void store_scaled(elem* hi, elem* lo, int tid, const float* et) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = tid + i * NT, row = e / NCB, cb = e % NCB;
      if (e >= NE) continue;
      const float s = et[row];
      f32x4 f;
#pragma unroll
      for (int j = 0; j < 4; ++j) f[j] = (float)v[i][j] * s;
      const int o = lds_off(row, 4 * cb, K);
      OP::store4_split(hi + o, lo + o, f);
    }
  }
};

// Step sizes of one chunk, loaded together with the chunk's tiles (thread
// tid < C holds row tid; per-token values only), then staged into LDS as
// sign * eta for the valid rows and 0 past them.
template <bool ETAV>
struct EtaReg {
  float v;
  __device__ __forceinline__ void load(rsrc_t r, uint32_t off_row0, int tid, int C) {
    v = 0.f;
    if constexpr (ETAV) v = buf_load1(r, (off_row0 == kOOB || tid >= C) ? kOOB : off_row0 + 4 * tid);
  }
  __device__ __forceinline__ void stage(float* et, int C, float eta_scalar, int nvalid, float sign, int tid) const {
    if (tid < C) et[tid] = tid < nvalid ? sign * (ETAV ? v : eta_scalar) : 0.f;
  }
};

__device__ __forceinline__ rsrc_t eta_rsrc(const float* eta, int64_t bh, int64_t T) {
  return make_rsrc(eta ? eta + bh * T : nullptr, eta ? (uint32_t)(T * 4) : 0u);
}

// ---------------------------------------------------------------------------
// Document resets at unit retention.  A reset at token t (t > 0) starts a new
// document: t's read sees W_0 plus the writes of its own document only
// (Section 3: Eq. 2 holds within each reset segment).  Within one chunk of
// C = 64 tokens this is a set of masks, all taken from the chunk's 64-bit
// flag mask m (bit p: a document starts at chunk position p):
//   same_doc(s, t)  no flag in (min, max] of the two positions
//   fr              first flagged position (C if none): rows p < fr read the
//                   carried state, rows p >= fr read W_0 (and their document)
//   lr              last flagged position (-1 if none): only writes at
//                   p >= lr reach the next chunk, which starts from W_0.
// Every wave loads the chunk's flags (lane p: position p, with the chunk's
// tiles; a buffer load, so past the sequence end it reads 0) and forms m with
// a ballot, so no wave waits for another.  A flag at t = 0 has no earlier
// write to drop and is ignored.
// ---------------------------------------------------------------------------
template <bool RST>
struct RstReg {
  int v;
  __device__ __forceinline__ void load(rsrc_t row, int64_t t0, bool ok, int tid, int C) {
    v = 0;
    if constexpr (RST) {
      const int lane = tid & 63;
      const int64_t t = t0 + lane;
      v = __builtin_amdgcn_raw_buffer_load_b8(row, (ok && lane < C && t > 0) ? (int)t : (int)kOOB, 0, 0);
    }
  }
  // The chunk's flag mask (wave-uniform).
  __device__ __forceinline__ uint64_t mask() const {
    if constexpr (RST) return __ballot(v != 0);
    return 0;
  }
};

__device__ __forceinline__ rsrc_t reset_rsrc(const uint8_t* reset, int64_t b, int64_t T) {
  return make_rsrc(reset ? reset + b * T : nullptr, reset ? (uint32_t)T : 0u);
}

// Positions s and t (0..63) of one chunk lie in the same document.
__device__ __forceinline__ bool same_doc(uint64_t m, int s, int t) {
  const int lo = s < t ? s : t, hi = s < t ? t : s;
  const uint64_t upto_hi = hi >= 63 ? ~0ull : ((2ull << hi) - 1);
  const uint64_t upto_lo = (2ull << lo) - 1;
  return (m & upto_hi & ~upto_lo) == 0;
}
__device__ __forceinline__ int first_flag(uint64_t m) { return m ? __builtin_ctzll(m) : 64; }
__device__ __forceinline__ int last_flag(uint64_t m) { return m ? 63 - __builtin_clzll(m) : -1; }

// A fragment with the elements whose k (k0 + slot_k(e, q)) lies outside
// [lo, hi) set to zero: for operands read with k along the tile rows.
template <class OP>
__device__ __forceinline__ typename OP::frag mask_k(typename OP::frag f, int k0, int q, int lo, int hi) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int k = k0 + slot_k(e, q);
    if (k < lo || k >= hi) f[e] = (typename OP::elem)0.f;
  }
  return f;
}
// A row fragment (row = row0 + lane % 16) kept or zeroed as a whole.
template <class OP>
__device__ __forceinline__ typename OP::frag keep_row(typename OP::frag f, bool keep) {
#pragma unroll
  for (int e = 0; e < 8; ++e)
    if (!keep) f[e] = (typename OP::elem)0.f;
  return f;
}

// Last document start in (lo, hi], or the first in [lo, hi) (-1 if none;
// t = 0 never counts), over one sequence's reset flags, by the whole
// workgroup: blocks of 16 NT tokens (16 independent byte loads per thread,
// each through the row's resource, so nothing past the row is read) from the
// end nearest the segment, stopping at the first block that holds a reset.
// Every thread returns the same value.
template <int NT>
__device__ __forceinline__ int64_t last_reset_in(rsrc_t row, int64_t lo, int64_t hi, int tid, int* red) {
  constexpr int SPAN = 16 * NT;
  for (int64_t top = hi; top > lo; top -= SPAN) {
    int best = -1;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int64_t t = top - (int64_t)u * NT - tid;
      const bool in = t > lo && t >= 1;
      const int f = __builtin_amdgcn_raw_buffer_load_b8(row, in ? (int)t : (int)kOOB, 0, 0);
      if (in && f && (int)t > best) best = (int)t;
    }
    __syncthreads();
    if (tid == 0) red[0] = -1;
    __syncthreads();
    if (best >= 0) atomicMax(red, best);
    __syncthreads();
    const int r = red[0];
    if (r >= 0) return r;
  }
  return -1;
}
template <int NT>
__device__ __forceinline__ int64_t first_reset_in(rsrc_t row, int64_t lo, int64_t hi, int tid, int* red) {
  constexpr int SPAN = 16 * NT;
  for (int64_t base = lo; base < hi; base += SPAN) {
    int best = 0x7fffffff;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int64_t t = base + (int64_t)u * NT + tid;
      const bool in = t < hi && t >= 1;
      const int f = __builtin_amdgcn_raw_buffer_load_b8(row, in ? (int)t : (int)kOOB, 0, 0);
      if (in && f && (int)t < best) best = (int)t;
    }
    __syncthreads();
    if (tid == 0) red[0] = 0x7fffffff;
    __syncthreads();
    if (best != 0x7fffffff) atomicMin(red, best);
    __syncthreads();
    const int r = red[0];
    if (r != 0x7fffffff) return r;
  }
  return -1;
}

// ---------------------------------------------------------------------------
// Segment aggregates: A_k = sum_{t in seg k} eta_t g_t x_t^T (fp32) and, for
// the backward (mode kAggBwdAB), B_k = sum_{t in seg k} dY_t x_t^T for k >= 1.
// Forward: A row-major [m][d].  Backward: A and B transposed [d][m] (its waves
// own column blocks of W and R).  Segments [0, nagg) of every sequence; wave
// w owns rows i in [16w, 16w+16).  With a scalar eta the products are exact
// bf16 products and eta scales the sum once; per-token eta is folded into a
// hi + lo split operand staged once per chunk.
// ---------------------------------------------------------------------------
// kAggBwdB: the dY x^T aggregates only (segments >= 1), for a backward that
// starts from the forward's saved segment-end weights and needs no A_k.
enum AggMode { kAggFwd = 0, kAggBwdA = 1, kAggBwdAB = 2, kAggBwdB = 3 };

// With document resets (RST, modes kAggFwd and kAggBwdB): the forward's A_k
// keeps only the writes at or after the segment's last reset (the ones that
// reach the next segment); the backward's B_k keeps the tokens before the
// segment's first reset (the ones a read in an earlier segment's document
// sees), and aggF takes the full sum of every segment for dW0.
template <class OP, int D, int M, int C, int MODE, bool ETAV, bool RST = false>
__global__ void __launch_bounds__(cmax(D, M) / 16 * 64)
agg_kernel(const KArgs a, int64_t nagg) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr bool BWD = MODE == kAggBwdAB || MODE == kAggBwdB;  // aggregate dY x^T
  constexpr bool WA = MODE != kAggBwdB;                          // aggregate the writes
  constexpr bool TRANS = MODE != kAggFwd;    // backward layout
  constexpr bool SPLITV = ETAV && OP::kSplit == 2;
  constexpr int NW = cmax(D, M) / 16, NT = NW * 64;
  constexpr int JB = D / 16, IB = M / 16;
  __shared__ E Xs[C * D];
  __shared__ E Gs[C * M];                 // G, or eta G hi when ETAV
  __shared__ E Gl[SPLITV ? C * M : 1];    // eta G lo
  __shared__ E Ds[BWD ? C * M : 1];
  __shared__ float et[C];
  __shared__ int red[1];

  int64_t bh, seg;
  if (!map_block(a.BH, a.nseg, bh, seg) || seg >= nagg) return;
  if (!WA && !RST && seg == 0) return;  // B_0 is never needed (with resets, its full sum is)
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, c = lane & 15, q = lane >> 4;
  const int64_t T = a.T;
  const int64_t t_begin = seg * a.seg_len;
  const int64_t t_end = t_begin + a.seg_len < T ? t_begin + a.seg_len : T;
  const bool with_b = BWD && (seg >= 1 || RST);

  const rsrc_t X = make_rsrc(static_cast<const E*>(a.X) + bh * T * D, (uint32_t)(T * D * sizeof(E)));
  const rsrc_t G = make_rsrc(WA ? static_cast<const E*>(a.G) + bh * T * M : nullptr, WA ? (uint32_t)(T * M * sizeof(E)) : 0u);
  const rsrc_t Dy = make_rsrc(BWD ? static_cast<const E*>(a.dY) + bh * T * M : nullptr, BWD ? (uint32_t)(T * M * sizeof(E)) : 0u);

  f32x4 accA[JB], accB[JB], accF[RST && BWD ? JB : 1];
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) accA[jb] = accB[jb] = zero4();
  if constexpr (RST && BWD)
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) accF[jb] = zero4();

  // The pass streams its inputs and does little arithmetic per byte; chunks
  // are staged DEPTH ahead.  Two measured best from HBM at B=8, H=16,
  // T=2048, d=m=64 (forward pass 16.4 -> 15.4 us, backward 18.5 -> 16.5 us
  // against four; one, three, six and eight were slower, and so were two
  // groups of waves per workgroup): more loads in flight per CU only add
  // concurrent streams.  Every group runs all DEPTH chunk steps (a step past
  // the segment end sees zero tiles and adds nothing), which keeps the memory
  // operations branch-free.
  constexpr int DEPTH = 2;
  Tile4<OP, C, D, NT> xr[DEPTH];
  Tile4<OP, C, M, NT> gr[DEPTH], dr[DEPTH];
  EtaReg<ETAV> er[DEPTH];
  const rsrc_t Et = eta_rsrc(a.eta, bh, T);
  auto fetch = [&](int k, int64_t t0) {
    const bool ok = t0 < t_end;
    if (WA) er[k].load(Et, ok ? (uint32_t)(t0 * 4) : kOOB, tid, C);
    xr[k].load(X, ok ? (uint32_t)(t0 * D * sizeof(E)) : kOOB, tid);
    if (WA) gr[k].load(G, ok ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
    if (with_b) dr[k].load(Dy, ok ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
  };
  // Issued in slot order (the scheduler would otherwise hoist the later
  // slots' loads above the first's, and the loop's first wait, which must
  // hold for both entries into the loop, would then drain every load).
#pragma unroll
  for (int k = 0; k < DEPTH; ++k) {
    fetch(k, t_begin + k * C);
    __builtin_amdgcn_sched_barrier(0);
  }
  // Segment-local reset bounds: writes kept from wlo on, dY x^T pre-reset part below bhi.
  int64_t wlo = t_begin, bhi = t_end;
  if constexpr (RST) {
    const rsrc_t rrow = reset_rsrc(a.reset, bh / a.H, T);
    if constexpr (WA) {
      const int64_t lr = last_reset_in<NT>(rrow, t_begin - 1, t_end - 1, threadIdx.x, red);
      if (lr >= 0) wlo = lr;
      if (a.segreset && threadIdx.x == 0) a.segreset[bh * a.nseg + seg] = (int)lr;
    } else {
      const int64_t fr = first_reset_in<NT>(rrow, t_begin, t_end, threadIdx.x, red);
      if (fr >= 0) bhi = fr;
      if (a.segreset && threadIdx.x == 0) a.segreset[bh * a.nseg + seg] = (int)fr;
    }
  }

  auto chunk = [&](int k, int64_t t0) {
    const int nvalid = (int)(t_end - t0 < C ? (t_end > t0 ? t_end - t0 : 0) : C);
    __syncthreads();
    if (WA && ETAV) er[k].stage(et, C, a.eta_scalar, nvalid, 1.f, tid);
    xr[k].store(Xs, tid);
    if (with_b) dr[k].store(Ds, tid);
    if (WA && !ETAV) gr[k].store(Gs, tid);
    if (WA && ETAV) {
      __syncthreads();
      gr[k].store_scaled(Gs, Gl, tid, et);
    }
    __syncthreads();
    fetch(k, t0 + DEPTH * C);
    if (w < IB) {
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
        // A^T[j][i] += sum_t X[t][j] (eta G)[t][i];  B^T[j][i] += sum_t X[t][j] dY[t][i]
        F gh{}, gl{}, dv{}, dp{};
        if constexpr (WA) {
          gh = OP::load_t(Gs, M, 32 * kb, 16 * w, lane);
          gl = gh;
          if constexpr (SPLITV) gl = OP::load_t(Gl, M, 32 * kb, 16 * w, lane);
          if constexpr (RST) {
            gh = mask_k<OP>(gh, 32 * kb, q, (int)(wlo - t0 > -1 ? (wlo - t0 < C ? wlo - t0 : C) : 0), C);
            gl = mask_k<OP>(gl, 32 * kb, q, (int)(wlo - t0 > -1 ? (wlo - t0 < C ? wlo - t0 : C) : 0), C);
          }
          dv = gh;
        }
        if (with_b) dv = OP::load_t(Ds, M, 32 * kb, 16 * w, lane);
        dp = dv;
        if constexpr (RST && BWD)
          dp = mask_k<OP>(dv, 32 * kb, q, 0, (int)(bhi - t0 < C ? (bhi - t0 > 0 ? bhi - t0 : 0) : C));
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) {
          const F xa = OP::load_t(Xs, D, 32 * kb, 16 * jb, lane);
          if constexpr (WA) {
            if constexpr (ETAV) accA[jb] = mma_split_b<OP>(accA[jb], xa, gh, gl);
            else accA[jb] = OP::mma(accA[jb], xa, gh);
          }
          if (with_b) accB[jb] = OP::mma(accB[jb], xa, dp);
          if constexpr (RST && BWD) accF[jb] = OP::mma(accF[jb], xa, dv);
        }
      }
    }
  };
  for (int64_t t0 = t_begin; t0 < t_end; t0 += DEPTH * C) {
#pragma unroll
    for (int k = 0; k < DEPTH; ++k) chunk(k, t0 + k * C);
  }
  if (w < IB) {
    // accA[jb] holds A^T[j = 16jb + 4q + r][i = 16w + c].
    const int64_t base = (bh * a.nseg + seg) * M * D;
    const float s = ETAV ? 1.f : a.eta_scalar;
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) {
      if constexpr (!WA) {
      } else if (TRANS) {
#pragma unroll
        for (int r = 0; r < 4; ++r) a.aggA[base + (int64_t)(16 * jb + 4 * q + r) * M + 16 * w + c] = s * accA[jb][r];
      } else {
        *reinterpret_cast<f32x4*>(a.aggA + base + (int64_t)(16 * w + c) * D + 16 * jb + 4 * q) = s * accA[jb];
      }
      if (with_b) {
#pragma unroll
        for (int r = 0; r < 4; ++r) a.aggB[base + (int64_t)(16 * jb + 4 * q + r) * M + 16 * w + c] = accB[jb][r];
      }
      if constexpr (RST && BWD) {
#pragma unroll
        for (int r = 0; r < 4; ++r) a.aggF[base + (int64_t)(16 * jb + 4 * q + r) * M + 16 * w + c] = accF[jb][r];
      }
    }
  }
}

}  // namespace gradlev
