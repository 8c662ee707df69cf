// Wide maps (d_in and d_out multiples of 128, at least one above 128): the
// parallel form of the gated scans, i.e. the chunked form of Appendix C
// (Eq. 16) with one chunk spanning the whole sequence.
//
// With the retention products F[t][s] = prod_{s<j<t} alpha_j (Section 3,
// Eq. 2 general form; a reset at token r acts as alpha_{r-1} = eta_{r-1} = 0)
// and the write coefficients c_s = -eta_s:
//
//   forward        y_t      = W_0 x_t     + sum_{s<t} F[t][s] c_s (x_s . x_t)  g_s
//   transpose read gtilde_t = W_0^T dY_t  + sum_{s<t} F[t][s] c_s (g_s . dY_t) x_s
//
// Both are one operation, OUT = Q P0 + S V with the causal score matrix
// S[t][s] = F[t][s] c_s (Q_t . K_s):
//
//   forward:   Q = X,  K = X, P0 = W_0^T, V = G, OUT = Y       [T x d_out]
//   read:      Q = dY, K = G, P0 = W_0,   V = X, OUT = gtilde  [T x d_in]
//
// At the widths of the paper's adapted MLP (1024 -> 4096 -> 1024) and its
// context of 1024 tokens this costs 2 m d + (T - 1)(d + m) flops per token,
// less than a chunked scan's 4 m d, and it is three dense MFMA contractions
// with no sequential dependency.  Kernels:
//
//   wide_gate_kernel   per sequence: c_t, and the zero count and log-sum
//                      prefixes of the retentions that give F exactly
//                      (wide_prep_kernel: the same beside the bf16 W_0 split);
//   wide_score_kernel  64 x 64 tiles of S (contraction over the query width),
//                      scaled by F and c, masked to s < t, stored as bf16
//                      hi + lo (fp32 for fp32 inputs);
//   wide_out_kernel    128 x 128 output tiles: the W_0 term (fp32 W_0 split
//                      into bf16 hi + lo while it is staged) followed by the
//                      causal S V term, both into one fp32 accumulator.
#include "scan_common.hpp"

namespace gradlev {

// ---------------------------------------------------------------------------
// Gates.  F[t][s] (s < t) is zero when a zero retention lies strictly
// between s and t, else +-exp(lc[t-1] - lc[s]) with lc the inclusive prefix
// sum of log|alpha| over the nonzero retentions.  zc packs the inclusive
// count of zero retentions (times two) with the parity of the negative ones:
// F != 0 iff zc[t-1] >> 1 == zc[s] >> 1, and F < 0 iff their low bits
// differ.  The log sums are kept in fp64 so that long sequences lose nothing
// when two of them are subtracted.  Padding tokens (t >= T) have c = 0 and
// alpha = 1.
// ---------------------------------------------------------------------------
struct WGateArgs {
  const float* eta;
  float eta_scalar, eta_mul;
  const float* alpha;
  float alpha_scalar;
  const uint8_t* reset;
  int64_t H, T, Tp;
  float* cw;   // [BH][Tp]
  int* zc;     // [BH][Tp]
  double* lc;  // [BH][Tp]
};

__device__ __forceinline__ void gate_at(const WGateArgs& g, int64_t bh, int64_t b, int64_t t, float& a, float& e) {
  if (t >= g.T) {
    a = 1.f;
    e = 0.f;
    return;
  }
  e = (g.eta ? g.eta[bh * g.T + t] : g.eta_scalar) * g.eta_mul;
  a = g.alpha ? g.alpha[bh * g.T + t] : g.alpha_scalar;
  if (g.reset && t + 1 < g.T && g.reset[b * g.T + t + 1]) {
    a = 0.f;
    e = 0.f;
  }
}

// Packed zero count and sign parity: a zero adds 2, a negative toggles bit 0.
__device__ __forceinline__ int zc_step(int z, float a) { return a == 0.f ? z + 2 : (a < 0.f ? z ^ 1 : z); }
__device__ __forceinline__ int zc_join(int l, int r) { return ((l & ~1) + (r & ~1)) | ((l ^ r) & 1); }

__device__ __forceinline__ void wide_gate_block(const WGateArgs& g, int64_t bh) {
  const int64_t b = bh / g.H;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t per = (g.Tp + 255) / 256;
  const int64_t t0 = tid * per, t1 = t0 + per < g.Tp ? t0 + per : g.Tp;
  __shared__ int sz[4];
  __shared__ double sl[4];
  // Thread totals over its span, then an exclusive scan over the block:
  // inclusive scan inside each wave (shuffles), wave totals through LDS.
  int z = 0;
  double l = 0.0;
  for (int64_t t = t0; t < t1; ++t) {
    float a, e;
    gate_at(g, bh, b, t, a, e);
    z = zc_step(z, a);
    if (a != 0.f && fabsf(a) != 1.f) l += log(fabs((double)a));  // log 1 = 0 exactly
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int zo = __shfl_up(z, o);
    const double lo = __shfl_up(l, o);
    if (lane >= o) {
      z = zc_join(zo, z);
      l = lo + l;
    }
  }
  if (lane == 63) {
    sz[w] = z;
    sl[w] = l;
  }
  // exclusive within the wave
  int ze = __shfl_up(z, 1);
  double le = __shfl_up(l, 1);
  if (lane == 0) {
    ze = 0;
    le = 0.0;
  }
  __syncthreads();
  int zp = 0;
  double lp = 0.0;
  for (int i = 0; i < w; ++i) {
    zp = zc_join(zp, sz[i]);
    lp += sl[i];
  }
  z = zc_join(zp, ze);
  l = lp + le;
  for (int64_t t = t0; t < t1; ++t) {
    float a, e;
    gate_at(g, bh, b, t, a, e);
    z = zc_step(z, a);
    if (a != 0.f && fabsf(a) != 1.f) l += log(fabs((double)a));
    g.zc[bh * g.Tp + t] = z;
    g.lc[bh * g.Tp + t] = l;
    g.cw[bh * g.Tp + t] = -e;
  }
}
static __global__ void __launch_bounds__(256) wide_gate_kernel(const WGateArgs g) { wide_gate_block(g, blockIdx.x); }

// ---------------------------------------------------------------------------
// Staging of a ROWS x COLS tile of a row-major global matrix into a swizzled
// LDS tile (layout of device_common.hpp) in 16-byte units: consecutive
// threads take consecutive units of a row, so the loads coalesce.  Loads go
// through a buffer resource; rows past its end read as zero.
// ---------------------------------------------------------------------------
template <typename E, int ROWS, int COLS, int NT>
struct GTile {
  static constexpr int EPU = 16 / (int)sizeof(E);  // elements per unit
  static constexpr int UPR = COLS / EPU, NU = ROWS * UPR, PER = NU / NT;
  static_assert(NU % NT == 0, "tile units must divide evenly over the threads");
  i32x4 v[PER];

  // Unit (row r, column unit cu) lives at byte row_off + r * stride + col0 + 16 cu.
  __device__ __forceinline__ void load(rsrc_t src, uint32_t row_off, uint32_t stride, uint32_t col0, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = tid + i * NT, r = u / UPR, cu = u % UPR;
      v[i] = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                            src, (int)(row_off + (uint32_t)r * stride + col0 + 16u * cu), 0, 0));
    }
  }
  // One 16-byte LDS store per unit.  A bf16 unit is the chunk pair
  // (2c, 2c + 1); the swizzle XORs chunk indices, so the pair stays an aligned
  // pair, in swapped order when the row's swizzle is odd.
  __device__ __forceinline__ void store(E* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = tid + i * NT, r = u / UPR, k = (u % UPR) * EPU;
      if constexpr (sizeof(E) == 2) {
        const int ch = (k >> 2) ^ swz(r, COLS);
        const i32x4 x = (ch & 1) ? i32x4{v[i][2], v[i][3], v[i][0], v[i][1]} : v[i];
        *reinterpret_cast<i32x4*>(lds + r * COLS + 4 * (ch & ~1)) = x;
      } else {
        *reinterpret_cast<i32x4*>(lds + lds_off(r, k, COLS)) = v[i];
      }
    }
  }
  // fp32 source split into hi (and lo) tiles of the operand type.
  template <class OP>
  __device__ __forceinline__ void store_split(typename OP::elem* hi, typename OP::elem* lo, int tid) const {
    static_assert(sizeof(E) == 4, "split staging reads fp32");
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = tid + i * NT, r = u / UPR, k = (u % UPR) * EPU;
      const int o = lds_off(r, k, COLS);
      OP::store4_split(hi + o, lo + o, __builtin_bit_cast(f32x4, v[i]));
    }
  }
};

// ---------------------------------------------------------------------------
// Score tiles.  Tile (tb, sb), sb <= tb, covers rows t in [128 tb, +128) and
// columns s in [128 sb, +128): the lower triangle of 128-token blocks, which
// is exactly what an output tile of rows [128 tb, +128) reads.  Workgroup of
// 4 waves; wave (wt, ws) owns rows t in [64 wt, +64), columns s in
// [64 ws, +64) as 4 x 4 accumulator blocks D[s][t] (lane: 4 consecutive s of
// one t, so the score rows are stored 8 bytes at a time).
//
// When the triangle has too few tiles to fill the chip, the contraction is
// split into KS ranges of the query width: each workgroup writes its fp32
// partial tile and wide_score_finish sums the partials in a fixed order, so
// results do not depend on scheduling.
// ---------------------------------------------------------------------------
struct WScoreArgs {
  const void* Q;
  const void* K;
  int64_t T, Tp, w, BH;
  int KS;
  const float* cw;
  const int* zc;
  const double* lc;
  void* Sh;
  void* Sl;
  float* part;  // [KS][BH][Tp][Tp] fp32 partial tiles (KS > 1)
};

// Tile index within one sequence's lower triangle of 128-token blocks.
__device__ __forceinline__ void tri_tile(int64_t L, int64_t& tb, int64_t& sb) {
  tb = (int64_t)((sqrt(8.0 * (double)L + 1.0) - 1.0) * 0.5);
  while ((tb + 1) * (tb + 2) / 2 <= L) ++tb;
  while (tb > 0 && tb * (tb + 1) / 2 > L) --tb;
  sb = L - tb * (tb + 1) / 2;
}

// Scales 4 consecutive scores (t; s .. s+3) by F[t][s] c_s, masks s >= t and
// padding rows, and stores them split (bf16 hi + lo) or as fp32.  F is
// rebased on the log sum at the end of the 64-column block holding s, so that
// the fp32 exponent argument stays small wherever F is not negligible.
template <class OP, int FMODE>
__device__ __forceinline__ void score_store(const WScoreArgs& a, int64_t bh, int64_t t, int64_t s, f32x4 acc) {
  typedef typename OP::elem E;
  const float* cw = a.cw + bh * a.Tp;
  const int* zc = a.zc + bh * a.Tp;
  const double* lc = a.lc + bh * a.Tp;
  const double ref = FMODE == 2 ? lc[s | 63] : 0.0;
  int zt = 0;
  float at = 0.f;
  if (FMODE >= 1 && t >= 1) zt = zc[t - 1];
  if (FMODE == 2 && t >= 1) at = (float)(lc[t - 1] - ref);
  const f32x4 cv = *reinterpret_cast<const f32x4*>(cw + s);
  f32x4 v;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float f = (s + r < t && t < a.T) ? cv[r] : 0.f;
    const int zs = FMODE >= 1 ? zc[s + r] : 0;
    if (FMODE >= 1 && (zs >> 1) != (zt >> 1)) f = 0.f;
    if (FMODE == 2 && f != 0.f) f *= ((zs ^ zt) & 1 ? -1.f : 1.f) * expf(at + (float)(ref - lc[s + r]));
    v[r] = acc[r] * f;
  }
  E* Sh = static_cast<E*>(a.Sh) + bh * a.Tp * a.Tp;
  E* Sl = static_cast<E*>(a.Sl) + bh * a.Tp * a.Tp;
  OP::store4_split(Sh + t * a.Tp + s, Sl + t * a.Tp + s, v);
}

template <class OP, int FMODE>
static __global__ void __launch_bounds__(256) wide_score_kernel(const WScoreArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int BT = 128, BK = 64, NT = 256;
  __shared__ __attribute__((aligned(16))) E Ps[BT * BK];  // K rows s
  __shared__ __attribute__((aligned(16))) E Qs[BT * BK];  // Q rows t

  const int64_t Kp = a.Tp / BT, per_seq = Kp * (Kp + 1) / 2;
  const int64_t ks = blockIdx.x % a.KS, tile = blockIdx.x / a.KS;
  const int64_t bh = tile / per_seq;
  int64_t tb, sb;
  tri_tile(tile % per_seq, tb, sb);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, wt = w >> 1, ws = w & 1;
  const int c = lane & 15, q = lane >> 4;
  // this range's 64-wide steps of the contraction (ranges differ by at most one step)
  const int64_t nsteps = a.w / 64, kb = nsteps * ks / a.KS, ke = nsteps * (ks + 1) / a.KS;
  const int64_t kbeg = 64 * kb;

  f32x4 acc[4][4];  // [s block][t block]: D[s][t] = K_s . Q_t
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = zero4();

  {
    const size_t es = sizeof(E);
    const rsrc_t Qr = make_rsrc(static_cast<const E*>(a.Q) + bh * a.T * a.w, (uint32_t)(a.T * a.w * es));
    const rsrc_t Kr = make_rsrc(static_cast<const E*>(a.K) + bh * a.T * a.w, (uint32_t)(a.T * a.w * es));
    const uint32_t stride = (uint32_t)(a.w * es);
    const uint32_t qoff = (uint32_t)(BT * tb * stride), koff = (uint32_t)(BT * sb * stride);
    // Two-deep register pipeline as in wide_out_kernel; an odd step count
    // ends with one step of zeros (its fetch lies past the range).
    struct Set {
      GTile<E, BT, BK, NT> qt, kt;
    } st[2];
    const int64_t nk = ke - kb;
    auto fetch = [&](Set& x, int64_t k) {
      const bool ok = k < nk;
      const uint32_t col = (uint32_t)((kbeg + k * BK) * es);
      x.qt.load(Qr, ok ? qoff : kOOB, stride, col, tid);
      x.kt.load(Kr, ok ? koff : kOOB, stride, col, tid);
    };
    auto step = [&](Set& x, int64_t k) {
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      x.qt.store(Qs, tid);
      x.kt.store(Ps, tid);
      __syncthreads();
      fetch(x, k + 2);
#pragma unroll
      for (int kk = 0; kk < BK; kk += 32) {
        F qf[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) qf[j] = OP::load_n_sep(Qs, BK, 64 * wt + 16 * j, kk, lane);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const F pf = OP::load_n_sep(Ps, BK, 64 * ws + 16 * i, kk, lane);
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = OP::mma(acc[i][j], pf, qf[j]);
        }
      }
    };
    fetch(st[0], 0);
    // Issue order is the loop's: the first wait of every step counts only
    // the other set's loads, on entry too.
    __builtin_amdgcn_sched_barrier(0);
    fetch(st[1], 1);
    for (int64_t k = 0; k < nk; k += 2) {
      step(st[0], k);
      step(st[1], k + 1);
    }
  }

  // Lane (c, q) of block (i, j) holds s = s0 + 16 i + 4 q + r, t = t0 + 16 j + c.
  const int64_t s0 = BT * sb + 64 * ws, t0 = BT * tb + 64 * wt;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t t = t0 + 16 * j + c;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t s = s0 + 16 * i + 4 * q;
      if (a.KS == 1) score_store<OP, FMODE>(a, bh, t, s, acc[i][j]);
      else *reinterpret_cast<f32x4*>(a.part + ((ks * a.BH + bh) * a.Tp + t) * a.Tp + s) = acc[i][j];
    }
  }
}

// Sum of the KS partial tiles in order, then the scaling and split of
// score_store.  Thread: 4 consecutive columns of one row; workgroup: 8 rows
// of one tile (16 workgroups per tile).
template <class OP, int FMODE>
static __global__ void __launch_bounds__(256) wide_score_finish(const WScoreArgs a) {
  const int64_t Kp = a.Tp / 128, per_seq = Kp * (Kp + 1) / 2;
  const int64_t tile = blockIdx.x / 16, part = blockIdx.x % 16;
  const int64_t bh = tile / per_seq;
  int64_t tb, sb;
  tri_tile(tile % per_seq, tb, sb);
  const int tid = threadIdx.x;
  const size_t plane = (size_t)a.BH * a.Tp * a.Tp;
  const int64_t t = 128 * tb + 8 * part + tid / 32, s = 128 * sb + 4 * (tid % 32);
  const float* p = a.part + (bh * a.Tp + t) * a.Tp + s;
  f32x4 v = *reinterpret_cast<const f32x4*>(p);
  for (int k = 1; k < a.KS; ++k) v += *reinterpret_cast<const f32x4*>(p + k * plane);
  score_store<OP, FMODE>(a, bh, t, s, v);
}

// ---------------------------------------------------------------------------
// Output tiles.  Workgroup of 8 waves, tile 128 (t) x BN (n), BN 128 or 64
// (64 when 128-wide tiles would leave compute units idle).  Wave
// (kh, wt, wn) owns rows [64 wt, +64) and columns [BN/2 wn, +BN/2) as
// accumulator blocks D[n][t] (a lane holds 4 consecutive n of one t:
// 16-byte stores) and contracts the k sub-step kh of every staged 64-wide
// slice; the two halves are added through LDS at the end.
// Phase 1 contracts Q with W_0 over the query width, phase 2 contracts S with
// V over s < 128 (tile + 1).  Tiles are issued heaviest (last rows) first.
// ---------------------------------------------------------------------------
// ---------------------------------------------------------------------------
// Gate gradient of the write strengths (Appendix E keeps gate derivatives):
//   deta_s = -sum_{t>s} F[t][s] (x_s . x_t) (g_s . dY_t).
// Each lower-triangle 128 x 128 tile contracts dY G^T (over m) and X X^T
// (over d) into two accumulators, multiplies them with F and the causal mask,
// and sums its columns over the rows t of each wave's 64-row half; the partial
// column sums [BH][2 Tp/128][Tp] are added in a fixed order by
// wide_deta_reduce, which zeroes the tokens a reset overrides.
// ---------------------------------------------------------------------------
struct WDetaArgs {
  const void* X;
  const void* G;
  const void* dY;
  int64_t T, Tp, d, m, BH, H;
  const int* zc;
  const double* lc;
  float* dpart;
  float* deta;
  const uint8_t* reset;
  const float* cw;  // c_s = -eta_s, for Km
  float* Km;        // [BH][Tp][Tp] or null: K[t][s] = c_s (dY_t . g_s)(x_t . x_s), s < t (lower tiles)
  float* Fm;        // [BH][Tp][Tp] or null: F[t][s], s < t (lower tiles)
};

template <class OP, int FMODE>
static __global__ void __launch_bounds__(256) wide_deta_kernel(const WDetaArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int BT = 128, BK = 64, NT = 256;
  __shared__ __attribute__((aligned(16))) E Ps[BT * BK];
  __shared__ __attribute__((aligned(16))) E Qs[BT * BK];
  __shared__ float csum[2][BT];

  const int64_t Kp = a.Tp / BT, per_seq = Kp * (Kp + 1) / 2;
  const int64_t bh = blockIdx.x / per_seq;
  int64_t tb, sb;
  tri_tile(blockIdx.x % per_seq, tb, sb);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, wt = w >> 1, ws = w & 1;
  const int c = lane & 15, q = lane >> 4;
  const size_t es = sizeof(E);

  f32x4 acc[2][4][4];  // [contraction][s block][t block]: 0: dY_t . g_s, 1: x_t . x_s
#pragma unroll
  for (int z = 0; z < 2; ++z)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[z][i][j] = zero4();

#pragma unroll
  for (int z = 0; z < 2; ++z) {
    const int64_t w_ = z == 0 ? a.m : a.d;
    const rsrc_t Qr = make_rsrc(static_cast<const E*>(z == 0 ? a.dY : a.X) + bh * a.T * w_, (uint32_t)(a.T * w_ * es));
    const rsrc_t Kr = make_rsrc(static_cast<const E*>(z == 0 ? a.G : a.X) + bh * a.T * w_, (uint32_t)(a.T * w_ * es));
    const uint32_t stride = (uint32_t)(w_ * es);
    const uint32_t qoff = (uint32_t)(BT * tb * stride), koff = (uint32_t)(BT * sb * stride);
    GTile<E, BT, BK, NT> qt, kt;
    qt.load(Qr, qoff, stride, 0, tid);
    kt.load(Kr, koff, stride, 0, tid);
    for (int64_t k0 = 0; k0 < w_; k0 += BK) {
      __syncthreads();
      qt.store(Qs, tid);
      kt.store(Ps, tid);
      __syncthreads();
      const bool more = k0 + BK < w_;
      qt.load(Qr, more ? qoff : kOOB, stride, (uint32_t)((k0 + BK) * es), tid);
      kt.load(Kr, more ? koff : kOOB, stride, (uint32_t)((k0 + BK) * es), tid);
#pragma unroll
      for (int kk = 0; kk < BK; kk += 32) {
        F qf[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) qf[j] = OP::load_n_sep(Qs, BK, 64 * wt + 16 * j, kk, lane);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const F pf = OP::load_n_sep(Ps, BK, 64 * ws + 16 * i, kk, lane);
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[z][i][j] = OP::mma(acc[z][i][j], pf, qf[j]);
        }
      }
    }
  }

  // Lane (c, q) of block (i, j): s = s0 + 16 i + 4 q + r, t = t0 + 16 j + c.
  const int64_t s0 = BT * sb + 64 * ws, t0 = BT * tb + 64 * wt;
  const int* zc = a.zc + bh * a.Tp;
  const double* lc = a.lc + bh * a.Tp;
  const double ref = FMODE == 2 ? lc[s0 + 63] : 0.0;
  float col[4][4];  // [i][r]: this lane's partial column sums
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) col[i][r] = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t t = t0 + 16 * j + c;
    int zt = 0;
    float at = 0.f;
    if (FMODE >= 1 && t >= 1) zt = zc[t - 1];
    if (FMODE == 2 && t >= 1) at = (float)(lc[t - 1] - ref);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t s = s0 + 16 * i + 4 * q;
      f32x4 kv, fv;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool live = s + r < t && t < a.T;
        float f = live ? 1.f : 0.f;
        const int zs = FMODE >= 1 ? zc[s + r] : 0;
        if (FMODE >= 1 && (zs >> 1) != (zt >> 1)) f = 0.f;
        if (FMODE == 2 && f != 0.f) f = ((zs ^ zt) & 1 ? -1.f : 1.f) * expf(at + (float)(ref - lc[s + r]));
        const float k = acc[0][i][j][r] * acc[1][i][j][r];
        col[i][r] += f * k;
        fv[r] = f;
        kv[r] = live ? a.cw[bh * a.Tp + s + r] * k : 0.f;
      }
      if (a.Km) {
        const int64_t o = (bh * a.Tp + t) * a.Tp + s;
        *reinterpret_cast<f32x4*>(a.Km + o) = kv;
        *reinterpret_cast<f32x4*>(a.Fm + o) = fv;
      }
    }
  }
  // Sum over the 16 rows t held by lanes c = 0..15, then write this wave's
  // 64-row partial for its 64 columns.
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = col[i][r];
#pragma unroll
      for (int o = 8; o >= 1; o >>= 1) v += __shfl_xor(v, o, 16);
      col[i][r] = v;
    }
  if (c == 0) {
    float* out = a.dpart + ((bh * 2 * (a.Tp / BT)) + 2 * tb + wt) * a.Tp;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<f32x4*>(out + s0 + 16 * i + 4 * q) = f32x4{col[i][0], col[i][1], col[i][2], col[i][3]};
  }
}

// out[bh][s] = sign * (sum of the partial column sums of the row halves at
// or below s's block, in order), 0 for a token whose gates a reset overrides
// (deta: sign -1; dalpha: sign +1).
static __global__ void __launch_bounds__(256) wide_colsum_reduce(const WDetaArgs a, float* out, float sign) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= a.BH * a.T) return;
  const int64_t bh = i / a.T, s = i % a.T, b = bh / a.H;
  const int64_t nh = 2 * (a.Tp / 128);
  const float* p = a.dpart + bh * nh * a.Tp + s;
  float v = 0.f;
  for (int64_t h = 2 * (s / 128); h < nh; ++h) v += p[h * a.Tp];
  const bool cut = a.reset && s + 1 < a.T && a.reset[b * a.T + s + 1];
  out[bh * a.T + s] = cut ? 0.f : sign * v;
}

// ---------------------------------------------------------------------------
// Retention gradient (Appendix E keeps gate derivatives):
//   dalpha_t = <Lambda_{t+1}, Delta_t>_F
//            = sum_{u>t} F[u][t] Z[u][t],   Z[u][t] = sum_{s<t} F[t][s] K[u][s],
// with K[u][s] = c_s (dY_u . g_s)(x_u . x_s) and F the retention products:
// a pair of reads u and write s straddling t contributes through both decays
// on either side of t (the product is never divided by alpha_t, so zero
// retentions and resets stay exact).  Z = K F^T is a dense fp32 contraction
// over s (MFMA 16x16x4 f32) of the K and F tiles that wide_deta_kernel
// stored; tile (u block tb, t block sb) contracts s over [0, 128 (sb + 1)),
// where F[t][.] is nonzero, and its masked column sums over u go to the same
// partial layout as deta's.
// ---------------------------------------------------------------------------
template <int FMODE>
static __global__ void __launch_bounds__(256) wide_dalpha_kernel(const WDetaArgs a) {
  typedef OpF32 OP;
  typedef OP::frag F;
  constexpr int BT = 128, BK = 64, NT = 256;
  __shared__ __attribute__((aligned(16))) float Ps[BT * BK];  // F rows t
  __shared__ __attribute__((aligned(16))) float Qs[BT * BK];  // K rows u

  const int64_t Kp = a.Tp / BT, per_seq = Kp * (Kp + 1) / 2;
  const int64_t bh = blockIdx.x / per_seq;
  int64_t tb, sb;
  tri_tile(blockIdx.x % per_seq, tb, sb);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, wt = w >> 1, ws = w & 1;
  const int c = lane & 15, q = lane >> 4;

  f32x4 acc[4][4];  // [t block][u block]: D[t][u] = F_t . K_u = Z[u][t]
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = zero4();
  {
    const size_t plane = (size_t)a.Tp * a.Tp;
    const rsrc_t Qr = make_rsrc(a.Km + bh * plane, (uint32_t)(plane * 4));
    const rsrc_t Kr = make_rsrc(a.Fm + bh * plane, (uint32_t)(plane * 4));
    const uint32_t stride = (uint32_t)(a.Tp * 4);
    const uint32_t qoff = (uint32_t)(BT * tb) * stride, koff = (uint32_t)(BT * sb) * stride;
    GTile<float, BT, BK, NT> qt, kt;
    const int64_t nk = 2 * (sb + 1);
    qt.load(Qr, qoff, stride, 0, tid);
    kt.load(Kr, koff, stride, 0, tid);
    for (int64_t k = 0; k < nk; ++k) {
      __syncthreads();
      qt.store(Qs, tid);
      kt.store(Ps, tid);
      __syncthreads();
      const bool more = k + 1 < nk;
      qt.load(Qr, more ? qoff : kOOB, stride, (uint32_t)((k + 1) * BK * 4), tid);
      kt.load(Kr, more ? koff : kOOB, stride, (uint32_t)((k + 1) * BK * 4), tid);
#pragma unroll
      for (int kk = 0; kk < BK; kk += 32) {
        F qf[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) qf[j] = OP::load_n_sep(Qs, BK, 64 * wt + 16 * j, kk, lane);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const F pf = OP::load_n_sep(Ps, BK, 64 * ws + 16 * i, kk, lane);
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = OP::mma(acc[i][j], pf, qf[j]);
        }
      }
    }
  }

  // Lane (c, q) of block (i, j): t = s0 + 16 i + 4 q + r (the gradient's
  // token), u = t0 + 16 j + c (the read).
  const int64_t s0 = BT * sb + 64 * ws, t0 = BT * tb + 64 * wt;
  const int* zc = a.zc + bh * a.Tp;
  const double* lc = a.lc + bh * a.Tp;
  const double ref = FMODE == 2 ? lc[s0 + 63] : 0.0;
  float col[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) col[i][r] = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t u = t0 + 16 * j + c;
    int zu = 0;
    float au = 0.f;
    if (FMODE >= 1 && u >= 1) zu = zc[u - 1];
    if (FMODE == 2 && u >= 1) au = (float)(lc[u - 1] - ref);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t t = s0 + 16 * i + 4 * q;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float f = (t + r < u && u < a.T) ? 1.f : 0.f;
        const int zt = FMODE >= 1 ? zc[t + r] : 0;
        if (FMODE >= 1 && (zt >> 1) != (zu >> 1)) f = 0.f;
        if (FMODE == 2 && f != 0.f) f = ((zt ^ zu) & 1 ? -1.f : 1.f) * expf(au + (float)(ref - lc[t + r]));
        col[i][r] += f * acc[i][j][r];
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = col[i][r];
#pragma unroll
      for (int o = 8; o >= 1; o >>= 1) v += __shfl_xor(v, o, 16);
      col[i][r] = v;
    }
  if (c == 0) {
    float* out = a.dpart + ((bh * 2 * (a.Tp / BT)) + 2 * tb + wt) * a.Tp;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<f32x4*>(out + s0 + 16 * i + 4 * q) = f32x4{col[i][0], col[i][1], col[i][2], col[i][3]};
  }
}

// ---------------------------------------------------------------------------
// dW0[h] = sum_b sum_t dY_t x_t^T (the decay is centered on W_0, so every read
// sees W_0 undiscounted).  Tile 128 (i over d_out) x 128 (j over d_in) per
// head; the contraction runs over the batch rows and tokens in a fixed order,
// 64 tokens per step, both operands read transposed from row-major token
// tiles.  Wave (wj, wi) owns a 64 x 64 block D[j][i] (a lane holds 4
// consecutive j of one i: 16-byte stores into the row-major dW0).
// ---------------------------------------------------------------------------
struct WDw0Args {
  const void* X;
  const void* dY;
  float* dW0;
  int64_t B, H, T, d, m;
};

template <class OP>
static __global__ void __launch_bounds__(256) wide_dw0_kernel(const WDw0Args a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int BT = 64, BN = 128, NT = 256;
  __shared__ __attribute__((aligned(16))) E Xs[BT * BN];  // [t][j]
  __shared__ __attribute__((aligned(16))) E Ds[BT * BN];  // [t][i]
  const int64_t nJ = a.d / BN, nI = a.m / BN;
  const int64_t h = blockIdx.x / (nI * nJ), rest = blockIdx.x % (nI * nJ);
  const int64_t i0 = BN * (rest / nJ), j0 = BN * (rest % nJ);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, wj = w >> 1, wi = w & 1;
  const int c = lane & 15, q = lane >> 4;
  const size_t es = sizeof(E);
  f32x4 acc[4][4];  // [j block][i block]
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = zero4();
  const int64_t nsteps = (a.T + BT - 1) / BT;
  GTile<E, BT, BN, NT> xt, dt;
  auto fetch = [&](int64_t k) {
    const bool ok = k < a.B * nsteps;
    const int64_t b = ok ? k / nsteps : 0, t0 = ok ? BT * (k % nsteps) : 0;
    const int64_t bh = b * a.H + h;
    const rsrc_t Xr = make_rsrc(static_cast<const E*>(a.X) + bh * a.T * a.d, (uint32_t)(a.T * a.d * es));
    const rsrc_t Dr = make_rsrc(static_cast<const E*>(a.dY) + bh * a.T * a.m, (uint32_t)(a.T * a.m * es));
    xt.load(Xr, ok ? (uint32_t)(t0 * a.d * es) : kOOB, (uint32_t)(a.d * es), (uint32_t)(j0 * es), tid);
    dt.load(Dr, ok ? (uint32_t)(t0 * a.m * es) : kOOB, (uint32_t)(a.m * es), (uint32_t)(i0 * es), tid);
  };
  fetch(0);
  for (int64_t k = 0; k < a.B * nsteps; ++k) {
    __syncthreads();
    xt.store(Xs, tid);
    dt.store(Ds, tid);
    __syncthreads();
    fetch(k + 1);
#pragma unroll
    for (int kk = 0; kk < BT; kk += 32) {
      F df[4];
#pragma unroll
      for (int y = 0; y < 4; ++y) df[y] = OP::load_t(Ds, BN, kk, 64 * wi + 16 * y, lane);
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const F xf = OP::load_t(Xs, BN, kk, 64 * wj + 16 * x, lane);
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = OP::mma(acc[x][y], xf, df[y]);
      }
    }
  }
  // Lane (c, q) of block (x, y): j = j0 + 64 wj + 16 x + 4 q + r, i = i0 + 64 wi + 16 y + c.
#pragma unroll
  for (int y = 0; y < 4; ++y) {
    const int64_t i = i0 + 64 * wi + 16 * y + c;
#pragma unroll
    for (int x = 0; x < 4; ++x)
      *reinterpret_cast<f32x4*>(a.dW0 + (h * a.m + i) * a.d + j0 + 64 * wj + 16 * x + 4 * q) = acc[x][y];
  }
}

// fp32 W_0 split once per call into bf16 hi and lo planes of the same
// layout (the output tiles then stage bf16 directly; the split costs one
// pass over W_0 instead of one per row tile).  The gate prefixes ride in
// the same launch: blocks [0, nbh) take one sequence each (a sequential
// span per thread, a few blocks only), the rest split W_0 beside them,
// instead of the prefixes running alone ahead of the scores.
static __global__ void __launch_bounds__(256) wide_prep_kernel(const WGateArgs g, int64_t nbh,
                                                               const float* __restrict__ W0, bf16* __restrict__ hi,
                                                               bf16* __restrict__ lo, int64_t n4) {
  if ((int64_t)blockIdx.x < nbh) {
    wide_gate_block(g, blockIdx.x);
    return;
  }
  const int64_t nb = (int64_t)gridDim.x - nbh;
  for (int64_t i = ((int64_t)blockIdx.x - nbh) * 256 + threadIdx.x; i < n4; i += nb * 256)
    OpBF16::store4_split(hi + 4 * i, lo + 4 * i, *reinterpret_cast<const f32x4*>(W0 + 4 * i));
}

struct WOutArgs {
  const void* Q;
  const bf16* Wh;  // bf16 operands: W_0 split into hi and lo planes [H][m][d]
  const bf16* Wl;
  const float* W0;
  const void* Sh;
  const void* Sl;
  const void* V;
  float* out;
  const float* addend;  // anti-causal mode: added before the store (may be out itself), or null
  int64_t wq, wout, BH, H, T, Tp;
};

// MODE 0 (causal): OUT[t] = Q_t P0 + sum_{s<t} S[t][s] V[s], the forward and
// the transpose read.  MODE 1 (anti-causal, no W_0 phase): OUT[t] =
// addend[t] + sum_{s>t} S[s][t] V[s], the write-side gradients: with the
// forward's scores and V = dY it is dG, with the read's scores and V = X the
// write side of dX (the transposed contraction of the same score matrix, read
// from its stored lower triangle with transposing LDS reads).
template <class OP, bool TRANS, int BN, int MODE>
static __global__ void __launch_bounds__(512) wide_out_kernel(const WOutArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int BM = 128, BK = 64, NT = 512, NB = BN / 32;  // NB: 16-column blocks per wave
  constexpr int TILE = BM * BK, PT = BN * BK;
  constexpr bool SPLIT = OP::kSplit == 2;
  constexpr int P1 = TILE + (SPLIT ? 2 : 1) * PT, P2 = (SPLIT ? 2 : 1) * TILE + PT;
  constexpr int PR = BM * BN * 4 / (int)sizeof(E);  // the kh = 1 waves' accumulators: a BM x BN fp32 partial
  static_assert(4 * NB * 4 * 64 * 16 == BM * BN * 4, "reduction layout covers the tile once");
  constexpr int PM = P1 > P2 ? P1 : P2;
  __shared__ __attribute__((aligned(16))) E lds[PM > PR ? PM : PR];
  // Phase 1: Qs | Ph | Pl.  Phase 2: Shs | Sls | Vs (fp32: Qs | Ph and Shs | Vs).
  E* const Qs = lds;
  E* const Ph = lds + TILE;
  E* const Pl = SPLIT ? lds + TILE + PT : Ph;
  E* const Shs = lds;
  E* const Sls = SPLIT ? lds + TILE : lds;
  E* const Vs = lds + (SPLIT ? 2 : 1) * TILE;

  const int64_t nTB = a.Tp / BM, nNB = a.wout / BN;
  const int64_t L = blockIdx.x, per_row = a.BH * nNB;
  const int64_t tb = MODE == 0 ? nTB - 1 - L / per_row : L / per_row;  // heaviest row tiles first
  const int64_t bh = (L % per_row) / nNB, nb = L % nNB;
  const int64_t h = bh % a.H;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, kh = w >> 2, wt = (w >> 1) & 1, wn = w & 1;
  const int c = lane & 15, q = lane >> 4;
  const int64_t t0 = BM * tb, n0 = BN * nb;
  const size_t es = sizeof(E);

  f32x4 acc[NB][4];  // [n block][t block]
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = zero4();

  // Both phases run a two-deep register pipeline: the tiles of step k + 2
  // are requested while step k computes, by two staging sets used in turn.
  // Step counts are even (widths are multiples of 128 and the causal range is
  // whole 128-token blocks), and a request past the last step reads from an
  // offset beyond the buffer (zeros, no branch), so the outstanding-load
  // counts stay exact across the barriers.
  // Phase 1: acc += W_0-term over k in [0, wq).
  if constexpr (MODE == 0) {
    const rsrc_t Qr = make_rsrc(static_cast<const E*>(a.Q) + bh * a.T * a.wq, (uint32_t)(a.T * a.wq * es));
    const int64_t md = a.wq * a.wout;
    const rsrc_t Wr = make_rsrc(a.W0 + h * md, (uint32_t)(md * 4));
    const uint32_t qstride = (uint32_t)(a.wq * es);
    // W_0 is [m][d]: forward rows n over k (row length wq), read rows k over n
    // (row length wout).  bf16 operands stage the hi and lo planes, fp32 W_0.
    const rsrc_t Whr = make_rsrc(SPLIT ? a.Wh + h * md : nullptr, SPLIT ? (uint32_t)(md * 2) : 0u);
    const rsrc_t Wlr = make_rsrc(SPLIT ? a.Wl + h * md : nullptr, SPLIT ? (uint32_t)(md * 2) : 0u);
    typedef GTile<E, TRANS ? BK : BN, TRANS ? BN : BK, NT> WT;
    struct Set {
      GTile<E, BM, BK, NT> qt;
      WT wh, wl;
    } st[2];
    const int64_t n1 = a.wq / BK;
    auto fetch = [&](Set& x, int64_t k) {
      const bool ok = k < n1;
      const int64_t k0 = k * BK;
      x.qt.load(Qr, ok ? (uint32_t)(t0 * qstride) : kOOB, qstride, (uint32_t)(k0 * es), tid);
      const rsrc_t r0 = SPLIT ? Whr : Wr;
      const uint32_t rows = TRANS ? (uint32_t)(k0 * a.wout * es) : (uint32_t)(n0 * a.wq * es);
      const uint32_t stride = TRANS ? (uint32_t)(a.wout * es) : (uint32_t)(a.wq * es);
      const uint32_t col = TRANS ? (uint32_t)(n0 * es) : (uint32_t)(k0 * es);
      x.wh.load(r0, ok ? rows : kOOB, stride, col, tid);
      if constexpr (SPLIT) x.wl.load(Wlr, ok ? rows : kOOB, stride, col, tid);
    };
    auto step = [&](Set& x, int64_t k) {
      // Keep each step's work inside the step: hoisting the other set's
      // stores would make the compiler wait for its loads here.
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      x.qt.store(Qs, tid);
      x.wh.store(Ph, tid);
      if constexpr (SPLIT) x.wl.store(Pl, tid);
      __syncthreads();
      fetch(x, k + 2);
      const int kk = 32 * kh;
      F qf[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) qf[j] = OP::load_n_sep(Qs, BK, 64 * wt + 16 * j, kk, lane);
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        F ph, pl;
        if constexpr (TRANS) {
          ph = OP::load_t(Ph, BN, kk, BN / 2 * wn + 16 * i, lane);
          pl = SPLIT ? OP::load_t(Pl, BN, kk, BN / 2 * wn + 16 * i, lane) : ph;
        } else {
          ph = OP::load_n_sep(Ph, BK, BN / 2 * wn + 16 * i, kk, lane);
          pl = SPLIT ? OP::load_n_sep(Pl, BK, BN / 2 * wn + 16 * i, kk, lane) : ph;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mma_split_a<OP>(acc[i][j], ph, pl, qf[j]);
      }
    };
    fetch(st[0], 0);
    // Issue order is the loop's: the first wait of every step counts only
    // the other set's loads, on entry too.
    __builtin_amdgcn_sched_barrier(0);
    fetch(st[1], 1);
    for (int64_t k = 0; k < n1; k += 2) {
      step(st[0], k);
      step(st[1], k + 1);
    }
  }

  // Phase 2: acc += S V over s in [0, 128 (tb + 1)) (causal), or
  // S^T V over s in [128 tb, Tp) (anti-causal: tiles of rows s, columns t).
  {
    const rsrc_t Shr = make_rsrc(static_cast<const E*>(a.Sh) + bh * a.Tp * a.Tp, (uint32_t)(a.Tp * a.Tp * es));
    const rsrc_t Slr = make_rsrc(SPLIT ? static_cast<const E*>(a.Sl) + bh * a.Tp * a.Tp : nullptr,
                                 SPLIT ? (uint32_t)(a.Tp * a.Tp * es) : 0u);
    const rsrc_t Vr = make_rsrc(static_cast<const E*>(a.V) + bh * a.T * a.wout, (uint32_t)(a.T * a.wout * es));
    const uint32_t sstride = (uint32_t)(a.Tp * es), vstride = (uint32_t)(a.wout * es);
    typedef GTile<E, MODE == 0 ? BM : BK, MODE == 0 ? BK : BM, NT> ST;
    struct Set {
      ST sh, sl;
      GTile<E, BK, BN, NT> vt;
    } st[2];
    const int64_t n2 = MODE == 0 ? 2 * (tb + 1) : 2 * (nTB - tb);
    const int64_t sbeg = MODE == 0 ? 0 : t0;
    auto fetch = [&](Set& x, int64_t k) {
      const bool ok = k < n2;
      const int64_t s0 = sbeg + k * BK;
      // causal: rows t [t0, +128), columns s; anti-causal: rows s [s0, +64), columns t
      const uint32_t rows = MODE == 0 ? (uint32_t)(t0 * sstride) : (uint32_t)(s0 * sstride);
      const uint32_t col = MODE == 0 ? (uint32_t)(s0 * es) : (uint32_t)(t0 * es);
      x.sh.load(Shr, ok ? rows : kOOB, sstride, col, tid);
      if constexpr (SPLIT) x.sl.load(Slr, ok ? rows : kOOB, sstride, col, tid);
      x.vt.load(Vr, ok ? (uint32_t)(s0 * vstride) : kOOB, vstride, (uint32_t)(n0 * es), tid);
    };
    auto step = [&](Set& x, int64_t k) {
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      x.sh.store(Shs, tid);
      if constexpr (SPLIT) x.sl.store(Sls, tid);
      x.vt.store(Vs, tid);
      __syncthreads();
      fetch(x, k + 2);
      const int kk = 32 * kh;
      F sfh[4], sfl[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if constexpr (MODE == 0) {
          sfh[j] = OP::load_n_sep(Shs, BK, 64 * wt + 16 * j, kk, lane);
          sfl[j] = SPLIT ? OP::load_n_sep(Sls, BK, 64 * wt + 16 * j, kk, lane) : sfh[j];
        } else {
          sfh[j] = OP::load_t(Shs, BM, kk, 64 * wt + 16 * j, lane);
          sfl[j] = SPLIT ? OP::load_t(Sls, BM, kk, 64 * wt + 16 * j, lane) : sfh[j];
        }
      }
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const F vf = OP::load_t(Vs, BN, kk, BN / 2 * wn + 16 * i, lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mma_split_b<OP>(acc[i][j], vf, sfh[j], sfl[j]);
      }
    };
    fetch(st[0], 0);
    // Issue order is the loop's: the first wait of every step counts only
    // the other set's loads, on entry too.
    __builtin_amdgcn_sched_barrier(0);
    fetch(st[1], 1);
    for (int64_t k = 0; k < n2; k += 2) {
      step(st[0], k);
      step(st[1], k + 1);
    }
  }

  // The kh = 1 waves hand their accumulators to the kh = 0 waves of the same
  // (wt, wn) through LDS (16 bytes per lane, one contiguous block per wave).
  f32x4* red = reinterpret_cast<f32x4*>(lds) + (w & 3) * NB * 4 * 64 + lane;
  __syncthreads();
  if (kh == 1) {
#pragma unroll
    for (int i = 0; i < NB; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) red[(i * 4 + j) * 64] = acc[i][j];
  }
  __syncthreads();
  if (kh == 1) return;
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] += red[(i * 4 + j) * 64];

  // Lane (c, q) of block (i, j): n = n0 + BN/2 wn + 16 i + 4 q + r, t = t0 + 64 wt + 16 j + c.
  const rsrc_t Or = make_rsrc(a.out + bh * a.T * a.wout, (uint32_t)(a.T * a.wout * 4));
  const rsrc_t Ar = make_rsrc(MODE == 1 && a.addend ? a.addend + bh * a.T * a.wout : nullptr,
                              MODE == 1 && a.addend ? (uint32_t)(a.T * a.wout * 4) : 0u);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t t = t0 + 64 * wt + 16 * j + c;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int64_t n = n0 + BN / 2 * wn + 16 * i + 4 * q;
      const uint32_t o = (uint32_t)((t * a.wout + n) * 4);
      if constexpr (MODE == 1) acc[i][j] += buf_load4(Ar, o, (const float*)nullptr);
      buf_store4(Or, o, acc[i][j]);
    }
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
// Splits of the score contraction: at most 4 ranges of at least four
// 64-wide steps each, no more than 512 workgroups (two per compute unit).
static int wide_score_splits(int64_t BH, int64_t Tp, int64_t w) {
  const int64_t tiles = BH * (Tp / 128) * (Tp / 128 + 1) / 2;
  int ks = 1;
  while (ks < 4 && tiles * (ks + 1) <= 2 * 256 && w / 64 / (ks + 1) >= 4) ++ks;
  return ks;
}

size_t wide_workspace_bytes(const WideProblem& p) {
  const size_t BH = (size_t)(p.B * p.H), Tp = (size_t)p.Tp;
  const size_t gates = BH * Tp * (4 + 4 + 8);
  const size_t S = BH * Tp * Tp * 4;  // bf16 hi + lo, or fp32; also the fp32 K tiles of dalpha
  const int kd = wide_score_splits((int64_t)BH, (int64_t)Tp, p.d), km = wide_score_splits((int64_t)BH, (int64_t)Tp, p.m);
  const int ks = kd > km ? kd : km;  // the forward contracts over d, the read over m
  const size_t part = ks > 1 ? (size_t)ks * BH * Tp * Tp * 4 : 0;
  const size_t planes = p.bf16 ? (size_t)p.H * p.m * p.d * 4 : 0;  // W_0 hi + lo
  const size_t dpart = BH * 2 * (Tp / 128) * Tp * 4;               // partial column sums (deta, dalpha)
  const size_t fm = BH * Tp * Tp * 4;                              // dalpha: fp32 F tiles
  return (gates + 255) / 256 * 256 + (S + 255) / 256 * 256 + (part + 255) / 256 * 256 + (planes + 255) / 256 * 256 +
         (dpart + 255) / 256 * 256 + fm;
}

namespace {

struct WideWs {
  float* cw;
  int* zc;
  double* lc;
  void* Sh;
  void* Sl;
  float* part;
  bf16* Wh;
  bf16* Wl;
  float* dpart;
  float* Km;  // the score region, reused once the scores are no longer needed
  float* Fm;
};

WideWs wide_ws(const WideProblem& p, void* ws) {
  const size_t BH = (size_t)(p.B * p.H), Tp = (size_t)p.Tp;
  char* w = static_cast<char*>(ws);
  WideWs o;
  o.lc = reinterpret_cast<double*>(w);
  o.cw = reinterpret_cast<float*>(w + BH * Tp * 8);
  o.zc = reinterpret_cast<int*>(w + BH * Tp * 12);
  char* s = w + (BH * Tp * 16 + 255) / 256 * 256;
  o.Sh = s;
  o.Sl = s + BH * Tp * Tp * 2;  // bf16 only
  o.Km = reinterpret_cast<float*>(s);
  char* pt = s + (BH * Tp * Tp * 4 + 255) / 256 * 256;
  o.part = reinterpret_cast<float*>(pt);
  const int kd = wide_score_splits((int64_t)BH, (int64_t)Tp, p.d), km = wide_score_splits((int64_t)BH, (int64_t)Tp, p.m);
  const int ks = kd > km ? kd : km;
  char* wp = pt + ((ks > 1 ? (size_t)ks * BH * Tp * Tp * 4 : 0) + 255) / 256 * 256;
  o.Wh = reinterpret_cast<bf16*>(wp);
  o.Wl = reinterpret_cast<bf16*>(wp + (size_t)p.H * p.m * p.d * 2);
  char* dp = wp + ((p.bf16 ? (size_t)p.H * p.m * p.d * 4 : 0) + 255) / 256 * 256;
  o.dpart = reinterpret_cast<float*>(dp);
  o.Fm = reinterpret_cast<float*>(dp + (BH * 2 * (Tp / 128) * Tp * 4 + 255) / 256 * 256);
  return o;
}

template <class OP>
void wide_gates(const WideProblem& p, const WidePtrs& f, const WideWs& ws, hipStream_t s) {
  WGateArgs g{f.eta, f.eta_scalar, f.eta_mul, f.alpha, f.alpha_scalar, f.reset, p.H, p.T, p.Tp, ws.cw, ws.zc, ws.lc};
  hipLaunchKernelGGL(wide_gate_kernel, dim3((unsigned)(p.B * p.H)), dim3(256), 0, s, g);
}

// Causal score matrix S[t][s] = F[t][s] c_s (Q_t . K_s) over width w into the
// score region (lower-triangle 128 x 128 tiles).
template <class OP>
void wide_scores(const WideProblem& p, const WideWs& ws, const void* Q, const void* K, int64_t w, hipStream_t s) {
  const int64_t BH = p.B * p.H;
  WScoreArgs sa{};
  sa.Q = Q;
  sa.K = K;
  sa.T = p.T;
  sa.Tp = p.Tp;
  sa.w = w;
  sa.BH = BH;
  sa.cw = ws.cw;
  sa.zc = ws.zc;
  sa.lc = ws.lc;
  sa.Sh = ws.Sh;
  sa.Sl = OP::kSplit == 2 ? ws.Sl : ws.Sh;
  sa.part = ws.part;
  sa.KS = wide_score_splits(BH, p.Tp, sa.w);
  const int64_t Kp = p.Tp / 128;
  const unsigned tiles = (unsigned)(BH * Kp * (Kp + 1) / 2), sgrid = tiles * sa.KS;
  if (p.fmode == 0) hipLaunchKernelGGL((wide_score_kernel<OP, 0>), dim3(sgrid), dim3(256), 0, s, sa);
  else if (p.fmode == 1) hipLaunchKernelGGL((wide_score_kernel<OP, 1>), dim3(sgrid), dim3(256), 0, s, sa);
  else hipLaunchKernelGGL((wide_score_kernel<OP, 2>), dim3(sgrid), dim3(256), 0, s, sa);
  if (sa.KS > 1) {
    if (p.fmode == 0) hipLaunchKernelGGL((wide_score_finish<OP, 0>), dim3(16 * tiles), dim3(256), 0, s, sa);
    else if (p.fmode == 1) hipLaunchKernelGGL((wide_score_finish<OP, 1>), dim3(16 * tiles), dim3(256), 0, s, sa);
    else hipLaunchKernelGGL((wide_score_finish<OP, 2>), dim3(16 * tiles), dim3(256), 0, s, sa);
  }
}

// Output tiles of MODE 0 (W_0 term read as W_0^T when !trans, W_0 when
// trans, plus the causal S V) or MODE 1 (anti-causal S^T V plus addend).
template <class OP>
void wide_out(const WideProblem& p, const WidePtrs& f, const WideWs& ws, int mode, bool trans, const void* Q,
              int64_t wq, const void* V, int64_t wout, float* out, const float* addend, hipStream_t s) {
  const int64_t BH = p.B * p.H;
  WOutArgs oa{};
  oa.Q = Q;
  oa.W0 = f.W0;
  oa.Wh = ws.Wh;
  oa.Wl = ws.Wl;
  oa.Sh = ws.Sh;
  oa.Sl = OP::kSplit == 2 ? ws.Sl : ws.Sh;
  oa.V = V;
  oa.out = out;
  oa.addend = addend;
  oa.wq = wq;
  oa.wout = wout;
  oa.BH = BH;
  oa.H = p.H;
  oa.T = p.T;
  oa.Tp = p.Tp;
  // 128-wide column tiles unless that leaves fewer than two tiles per compute unit.
  const int64_t t128 = BH * (p.Tp / 128) * (wout / 128);
  const bool narrow = t128 < 2 * 256;
  const unsigned g = (unsigned)(narrow ? 2 * t128 : t128);
  if (mode == 1) {
    if (narrow) hipLaunchKernelGGL((wide_out_kernel<OP, false, 64, 1>), dim3(g), dim3(512), 0, s, oa);
    else hipLaunchKernelGGL((wide_out_kernel<OP, false, 128, 1>), dim3(g), dim3(512), 0, s, oa);
  } else if (trans && narrow) hipLaunchKernelGGL((wide_out_kernel<OP, true, 64, 0>), dim3(g), dim3(512), 0, s, oa);
  else if (trans) hipLaunchKernelGGL((wide_out_kernel<OP, true, 128, 0>), dim3(g), dim3(512), 0, s, oa);
  else if (narrow) hipLaunchKernelGGL((wide_out_kernel<OP, false, 64, 0>), dim3(g), dim3(512), 0, s, oa);
  else hipLaunchKernelGGL((wide_out_kernel<OP, false, 128, 0>), dim3(g), dim3(512), 0, s, oa);
}

// The gate prefixes and, for bf16 operands, the W_0 split in one launch.
template <class OP>
void wide_prep(const WideProblem& p, const WidePtrs& f, const WideWs& ws, hipStream_t s) {
  if (OP::kSplit != 2) {
    wide_gates<OP>(p, f, ws, s);
    return;
  }
  WGateArgs g{f.eta, f.eta_scalar, f.eta_mul, f.alpha, f.alpha_scalar, f.reset, p.H, p.T, p.Tp, ws.cw, ws.zc, ws.lc};
  const int64_t n4 = p.H * (int64_t)p.m * p.d / 4, BH = p.B * p.H;
  const int64_t gs = n4 / 256 < 4096 ? (n4 + 255) / 256 : 4096;
  hipLaunchKernelGGL(wide_prep_kernel, dim3((unsigned)(BH + gs)), dim3(256), 0, s, g, BH, f.W0, ws.Wh, ws.Wl, n4);
}

// Forward (read = false: Q = K = X, V = G) or transpose read (read = true:
// Q = dY, K = G, V = X) into `out`.
template <class OP>
hipError_t wide_run(const WideProblem& p, const WidePtrs& f, bool read, float* out, hipStream_t s) {
  const WideWs ws = wide_ws(p, f.ws);
  timing_begin(GRADLEV_K_WIDE_SCORE, s);
  wide_prep<OP>(p, f, ws, s);
  wide_scores<OP>(p, ws, read ? f.dY : f.X, read ? f.G : f.X, read ? p.m : p.d, s);
  timing_end(GRADLEV_K_WIDE_SCORE, s);
  timing_begin(GRADLEV_K_WIDE_OUT, s);
  wide_out<OP>(p, f, ws, 0, read, read ? f.dY : f.X, read ? p.m : p.d, read ? f.X : f.G, read ? p.d : p.m, out,
               nullptr, s);
  timing_end(GRADLEV_K_WIDE_OUT, s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_wide_fwd(const WideProblem& p, const WidePtrs& f, hipStream_t s) {
  return p.bf16 ? wide_run<OpBF16>(p, f, false, f.Y, s) : wide_run<OpF32>(p, f, false, f.Y, s);
}

// The backward of a wide map, each output when requested:
//   gtilde = dY W_0 + S_read X        (causal; S_read = F c (dY G^T))
//   dX     = gtilde + S_read^T X      (anti-causal, write side)
//   dG     = S_fwd^T dY               (anti-causal; S_fwd = F c (X X^T))
//   deta, dalpha: masked column sums of the pair terms (wide_deta_kernel,
//   wide_dalpha_kernel); dW0 = sum_b dY^T X.
template <class OP>
static hipError_t wide_bwd(const WideProblem& p, const WidePtrs& f, hipStream_t s) {
  const int64_t BH = p.B * p.H;
  const WideWs ws = wide_ws(p, f.ws);
  const bool need_gates = f.gtilde || f.dX || f.dG || f.deta || f.dalpha;
  if (f.gtilde || f.dX) {
    // The read lands in gtilde, or directly in dX when only dX is requested.
    float* g = f.gtilde ? f.gtilde : f.dX;
    const hipError_t e = wide_run<OP>(p, f, true, g, s);
    if (e != hipSuccess) return e;
    if (f.dX) {
      timing_begin(GRADLEV_K_WIDE_OUT, s);
      wide_out<OP>(p, f, ws, 1, false, nullptr, 0, f.X, p.d, f.dX, g, s);
      timing_end(GRADLEV_K_WIDE_OUT, s);
    }
  } else if (need_gates) {
    wide_gates<OP>(p, f, ws, s);
  }
  if (f.dG) {
    timing_begin(GRADLEV_K_WIDE_SCORE, s);
    wide_scores<OP>(p, ws, f.X, f.X, p.d, s);
    timing_end(GRADLEV_K_WIDE_SCORE, s);
    timing_begin(GRADLEV_K_WIDE_OUT, s);
    wide_out<OP>(p, f, ws, 1, false, nullptr, 0, f.dY, p.m, f.dG, nullptr, s);
    timing_end(GRADLEV_K_WIDE_OUT, s);
  }
  if (f.deta || f.dalpha) {
    // The K and F tiles of dalpha take the score region, free from here on.
    WDetaArgs da{f.X, f.G, f.dY, p.T, p.Tp, p.d, p.m, BH, p.H, ws.zc, ws.lc, ws.dpart, f.deta, f.reset,
                 ws.cw, f.dalpha ? ws.Km : nullptr, f.dalpha ? ws.Fm : nullptr};
    const int64_t Kp = p.Tp / 128;
    const unsigned grid = (unsigned)(BH * Kp * (Kp + 1) / 2);
    const unsigned rgrid = (unsigned)((BH * p.T + 255) / 256);
    timing_begin(GRADLEV_K_WIDE_SCORE, s);
    if (p.fmode == 0) hipLaunchKernelGGL((wide_deta_kernel<OP, 0>), dim3(grid), dim3(256), 0, s, da);
    else if (p.fmode == 1) hipLaunchKernelGGL((wide_deta_kernel<OP, 1>), dim3(grid), dim3(256), 0, s, da);
    else hipLaunchKernelGGL((wide_deta_kernel<OP, 2>), dim3(grid), dim3(256), 0, s, da);
    if (f.deta) hipLaunchKernelGGL(wide_colsum_reduce, dim3(rgrid), dim3(256), 0, s, da, f.deta, -1.f);
    if (f.dalpha) {
      if (p.fmode == 0) hipLaunchKernelGGL((wide_dalpha_kernel<0>), dim3(grid), dim3(256), 0, s, da);
      else if (p.fmode == 1) hipLaunchKernelGGL((wide_dalpha_kernel<1>), dim3(grid), dim3(256), 0, s, da);
      else hipLaunchKernelGGL((wide_dalpha_kernel<2>), dim3(grid), dim3(256), 0, s, da);
      hipLaunchKernelGGL(wide_colsum_reduce, dim3(rgrid), dim3(256), 0, s, da, f.dalpha, 1.f);
    }
    timing_end(GRADLEV_K_WIDE_SCORE, s);
  }
  if (f.dW0) {
    WDw0Args wa{f.X, f.dY, f.dW0, p.B, p.H, p.T, p.d, p.m};
    timing_begin(GRADLEV_K_WIDE_OUT, s);
    hipLaunchKernelGGL((wide_dw0_kernel<OP>), dim3((unsigned)(p.H * (p.m / 128) * (p.d / 128))), dim3(256), 0, s, wa);
    timing_end(GRADLEV_K_WIDE_OUT, s);
  }
  return hipGetLastError();
}

hipError_t launch_wide_read(const WideProblem& p, const WidePtrs& f, hipStream_t s) {
  return p.bf16 ? wide_bwd<OpBF16>(p, f, s) : wide_bwd<OpF32>(p, f, s);
}

}  // namespace gradlev
