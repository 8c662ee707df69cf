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
//                      prefixes of the retentions that give F exactly;
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

static __global__ void __launch_bounds__(256) wide_gate_kernel(const WGateArgs g) {
  const int64_t bh = blockIdx.x, b = bh / g.H;
  const int tid = threadIdx.x;
  const int64_t per = (g.Tp + 255) / 256;
  const int64_t t0 = tid * per, t1 = t0 + per < g.Tp ? t0 + per : g.Tp;
  __shared__ int sz[256];
  __shared__ double sl[256];
  int z = 0;
  double l = 0.0;
  for (int64_t t = t0; t < t1; ++t) {
    float a, e;
    gate_at(g, bh, b, t, a, e);
    z = zc_step(z, a);
    if (a != 0.f) l += log(fabs((double)a));
  }
  sz[tid] = z;
  sl[tid] = l;
  __syncthreads();
  if (tid == 0) {
    int zz = 0;
    double ll = 0.0;
    for (int i = 0; i < 256; ++i) {
      const int tz = sz[i];
      const double tl = sl[i];
      sz[i] = zz;
      sl[i] = ll;
      zz = zc_join(zz, tz);
      ll += tl;
    }
  }
  __syncthreads();
  z = sz[tid];
  l = sl[tid];
  for (int64_t t = t0; t < t1; ++t) {
    float a, e;
    gate_at(g, bh, b, t, a, e);
    z = zc_step(z, a);
    if (a != 0.f) l += log(fabs((double)a));
    g.zc[bh * g.Tp + t] = z;
    g.lc[bh * g.Tp + t] = l;
    g.cw[bh * g.Tp + t] = -e;
  }
}

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
  __device__ __forceinline__ void store(E* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = tid + i * NT, r = u / UPR, k = (u % UPR) * EPU;
#pragma unroll
      for (int h = 0; h < EPU / 4; ++h) {
        typedef typename Vec4<E>::type vec4;
        vec4 x;
        if constexpr (sizeof(E) == 2) {
          const i32x2 p = {v[i][2 * h], v[i][2 * h + 1]};
          x = __builtin_bit_cast(vec4, p);
        } else {
          x = __builtin_bit_cast(vec4, v[i]);
        }
        *reinterpret_cast<vec4*>(lds + lds_off(r, k + 4 * h, COLS)) = x;
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
// Score tiles.  Tile (tb, sb) covers rows t in [64 tb, 64 tb + 64) and
// columns s in [64 sb, 64 sb + 64).  The output kernel reads, for its
// 128-row tile p, the columns [0, 128 (p + 1)), so every tile with
// sb <= (tb | 1) is written: those above the diagonal as zeros.  Per
// sequence that is 2 K (K + 1) tiles, K = Tp / 128.
// ---------------------------------------------------------------------------
struct WScoreArgs {
  const void* Q;
  const void* K;
  int64_t T, Tp, w, BH;
  const float* cw;
  const int* zc;
  const double* lc;
  void* Sh;
  void* Sl;
};

template <class OP, int FMODE>
static __global__ void __launch_bounds__(64) wide_score_kernel(const WScoreArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int BK = 64;
  __shared__ E Ps[64 * BK];  // K rows s
  __shared__ E Qs[64 * BK];  // Q rows t

  const int64_t Kp = a.Tp / 128, per_seq = 2 * Kp * (Kp + 1);
  const int64_t bh = blockIdx.x / per_seq;
  int64_t L = blockIdx.x % per_seq;
  // Pair row p holds tile rows 2p and 2p + 1 with 2p + 2 tiles each; the
  // rows before it hold 2 p (p + 1) tiles.
  int64_t p = (int64_t)((sqrt(1.0 + 2.0 * (double)L) - 1.0) * 0.5);
  while (2 * (p + 1) * (p + 2) <= L) ++p;
  while (p > 0 && 2 * p * (p + 1) > L) --p;
  L -= 2 * p * (p + 1);
  const int64_t tb = 2 * p + L / (2 * p + 2), sb = L % (2 * p + 2);
  const int lane = threadIdx.x, c = lane & 15, q = lane >> 4;
  const int64_t t0 = 64 * tb, s0 = 64 * sb;
  E* Sh = static_cast<E*>(a.Sh) + bh * a.Tp * a.Tp;
  E* Sl = static_cast<E*>(a.Sl) + bh * a.Tp * a.Tp;

  f32x4 acc[4][4];  // [s block][t block]: D[s][t] = K_s . Q_t
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = zero4();

  if (sb <= tb) {
    const size_t es = sizeof(E);
    const rsrc_t Qr = make_rsrc(static_cast<const E*>(a.Q) + bh * a.T * a.w, (uint32_t)(a.T * a.w * es));
    const rsrc_t Kr = make_rsrc(static_cast<const E*>(a.K) + bh * a.T * a.w, (uint32_t)(a.T * a.w * es));
    const uint32_t stride = (uint32_t)(a.w * es);
    GTile<E, 64, BK, 64> qt, kt;
    qt.load(Qr, (uint32_t)(t0 * stride), stride, 0, lane);
    kt.load(Kr, (uint32_t)(s0 * stride), stride, 0, lane);
    for (int64_t k0 = 0; k0 < a.w; k0 += BK) {
      __syncthreads();
      qt.store(Qs, lane);
      kt.store(Ps, lane);
      __syncthreads();
      if (k0 + BK < a.w) {
        qt.load(Qr, (uint32_t)(t0 * stride), stride, (uint32_t)((k0 + BK) * es), lane);
        kt.load(Kr, (uint32_t)(s0 * stride), stride, (uint32_t)((k0 + BK) * es), lane);
      }
#pragma unroll
      for (int kk = 0; kk < BK; kk += 32) {
        F qf[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) qf[j] = OP::load_n(Qs, BK, 16 * j, kk, lane);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const F pf = OP::load_n(Ps, BK, 16 * i, kk, lane);
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = OP::mma(acc[i][j], pf, qf[j]);
        }
      }
    }
  }

  // Epilogue: lane (c, q) of block (i, j) holds s = s0 + 16 i + 4 q + r and
  // t = t0 + 16 j + c.
  const float* cw = a.cw + bh * a.Tp;
  const int* zc = a.zc + bh * a.Tp;
  const double* lc = a.lc + bh * a.Tp;
  const double ref = FMODE == 2 ? lc[s0 + 63] : 0.0;
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
      const f32x4 cv = *reinterpret_cast<const f32x4*>(cw + s);
      f32x4 v;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float f = (s + r < t && t < a.T) ? cv[r] : 0.f;
        const int zs = FMODE >= 1 ? zc[s + r] : 0;
        if (FMODE >= 1 && (zs >> 1) != (zt >> 1)) f = 0.f;
        if (FMODE == 2 && f != 0.f) f *= ((zs ^ zt) & 1 ? -1.f : 1.f) * expf(at + (float)(ref - lc[s + r]));
        v[r] = acc[i][j][r] * f;
      }
      OP::store4_split(Sh + t * a.Tp + s, Sl + t * a.Tp + s, v);
    }
  }
}

// ---------------------------------------------------------------------------
// Output tiles.  Workgroup of 4 waves, tile 128 (t) x 128 (n); wave (wt, wn)
// owns rows [64 wt, +64) and columns [64 wn, +64) as 4 x 4 accumulator
// blocks D[n][t] (a lane holds 4 consecutive n of one t: 16-byte stores).
// Phase 1 contracts Q with W_0 over the query width, phase 2 contracts S with
// V over s < 128 (tile + 1).  Tiles are issued heaviest (last rows) first.
// ---------------------------------------------------------------------------
struct WOutArgs {
  const void* Q;
  const float* W0;
  const void* Sh;
  const void* Sl;
  const void* V;
  float* out;
  int64_t wq, wout, BH, H, T, Tp;
};

template <class OP, bool TRANS>
static __global__ void __launch_bounds__(256) wide_out_kernel(const WOutArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int BM = 128, BN = 128, BK = 64, NT = 256;
  constexpr int TILE = BM * BK;  // elements of one staged tile (all are 128 x 64 or 64 x 128)
  constexpr bool SPLIT = OP::kSplit == 2;
  __shared__ E lds[(SPLIT ? 3 : 2) * TILE];
  // Phase 1: Qs | Ph | Pl.  Phase 2: Shs | Sls | Vs (fp32: Qs | Ph and Shs | Vs).
  E* const Qs = lds;
  E* const Ph = lds + TILE;
  E* const Pl = SPLIT ? lds + 2 * TILE : Ph;
  E* const Shs = lds;
  E* const Sls = SPLIT ? lds + TILE : lds;
  E* const Vs = lds + (SPLIT ? 2 : 1) * TILE;

  const int64_t nTB = a.Tp / BM, nNB = a.wout / BN;
  const int64_t L = blockIdx.x, per_row = a.BH * nNB;
  const int64_t tb = nTB - 1 - L / per_row;
  const int64_t bh = (L % per_row) / nNB, nb = L % nNB;
  const int64_t h = bh % a.H;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, wt = w >> 1, wn = w & 1;
  const int c = lane & 15, q = lane >> 4;
  const int64_t t0 = BM * tb, n0 = BN * nb;
  const size_t es = sizeof(E);

  f32x4 acc[4][4];  // [n block][t block]
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = zero4();

  // Phase 1: acc += W_0-term over k in [0, wq).
  {
    const rsrc_t Qr = make_rsrc(static_cast<const E*>(a.Q) + bh * a.T * a.wq, (uint32_t)(a.T * a.wq * es));
    const int64_t md = a.wq * a.wout;
    const rsrc_t Wr = make_rsrc(a.W0 + h * md, (uint32_t)(md * 4));
    const uint32_t qstride = (uint32_t)(a.wq * es);
    GTile<E, BM, BK, NT> qt;
    // W_0 is [m][d]: forward rows n over k (row length wq), read rows k over n (row length wout).
    typedef GTile<float, TRANS ? BK : BN, TRANS ? BN : BK, NT> WT;
    WT wtile;
    auto wload = [&](int64_t k0) {
      if constexpr (TRANS) wtile.load(Wr, (uint32_t)(k0 * a.wout * 4), (uint32_t)(a.wout * 4), (uint32_t)(n0 * 4), tid);
      else wtile.load(Wr, (uint32_t)(n0 * a.wq * 4), (uint32_t)(a.wq * 4), (uint32_t)(k0 * 4), tid);
    };
    qt.load(Qr, (uint32_t)(t0 * qstride), qstride, 0, tid);
    wload(0);
    for (int64_t k0 = 0; k0 < a.wq; k0 += BK) {
      __syncthreads();
      qt.store(Qs, tid);
      if constexpr (SPLIT) wtile.template store_split<OP>(Ph, Pl, tid);
      else wtile.store(reinterpret_cast<float*>(Ph), tid);
      __syncthreads();
      if (k0 + BK < a.wq) {
        qt.load(Qr, (uint32_t)(t0 * qstride), qstride, (uint32_t)((k0 + BK) * es), tid);
        wload(k0 + BK);
      }
#pragma unroll
      for (int kk = 0; kk < BK; kk += 32) {
        F qf[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) qf[j] = OP::load_n(Qs, BK, 64 * wt + 16 * j, kk, lane);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          F ph, pl;
          if constexpr (TRANS) {
            ph = OP::load_t(Ph, BN, kk, 64 * wn + 16 * i, lane);
            pl = SPLIT ? OP::load_t(Pl, BN, kk, 64 * wn + 16 * i, lane) : ph;
          } else {
            ph = OP::load_n(Ph, BK, 64 * wn + 16 * i, kk, lane);
            pl = SPLIT ? OP::load_n(Pl, BK, 64 * wn + 16 * i, kk, lane) : ph;
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = mma_split_a<OP>(acc[i][j], ph, pl, qf[j]);
        }
      }
    }
  }

  // Phase 2: acc += S V over s in [0, 128 (tb + 1)).
  {
    const int64_t send = BM * (tb + 1);
    const rsrc_t Shr = make_rsrc(static_cast<const E*>(a.Sh) + bh * a.Tp * a.Tp, (uint32_t)(a.Tp * a.Tp * es));
    const rsrc_t Slr = make_rsrc(SPLIT ? static_cast<const E*>(a.Sl) + bh * a.Tp * a.Tp : nullptr,
                                 SPLIT ? (uint32_t)(a.Tp * a.Tp * es) : 0u);
    const rsrc_t Vr = make_rsrc(static_cast<const E*>(a.V) + bh * a.T * a.wout, (uint32_t)(a.T * a.wout * es));
    const uint32_t sstride = (uint32_t)(a.Tp * es), vstride = (uint32_t)(a.wout * es);
    GTile<E, BM, BK, NT> sh, sl;
    GTile<E, BK, BN, NT> vt;
    auto load = [&](int64_t s0) {
      sh.load(Shr, (uint32_t)(t0 * sstride), sstride, (uint32_t)(s0 * es), tid);
      if constexpr (SPLIT) sl.load(Slr, (uint32_t)(t0 * sstride), sstride, (uint32_t)(s0 * es), tid);
      vt.load(Vr, (uint32_t)(s0 * vstride), vstride, (uint32_t)(n0 * es), tid);
    };
    load(0);
    for (int64_t s0 = 0; s0 < send; s0 += BK) {
      __syncthreads();
      sh.store(Shs, tid);
      if constexpr (SPLIT) sl.store(Sls, tid);
      vt.store(Vs, tid);
      __syncthreads();
      if (s0 + BK < send) load(s0 + BK);
#pragma unroll
      for (int kk = 0; kk < BK; kk += 32) {
        F sfh[4], sfl[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          sfh[j] = OP::load_n(Shs, BK, 64 * wt + 16 * j, kk, lane);
          sfl[j] = SPLIT ? OP::load_n(Sls, BK, 64 * wt + 16 * j, kk, lane) : sfh[j];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const F vf = OP::load_t(Vs, BN, kk, 64 * wn + 16 * i, lane);
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = mma_split_b<OP>(acc[i][j], vf, sfh[j], sfl[j]);
        }
      }
    }
  }

  // Lane (c, q) of block (i, j): n = n0 + 64 wn + 16 i + 4 q + r, t = t0 + 64 wt + 16 j + c.
  const rsrc_t Or = make_rsrc(a.out + bh * a.T * a.wout, (uint32_t)(a.T * a.wout * 4));
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t t = t0 + 64 * wt + 16 * j + c;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t n = n0 + 64 * wn + 16 * i + 4 * q;
      buf_store4(Or, (uint32_t)((t * a.wout + n) * 4), acc[i][j]);
    }
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
size_t wide_workspace_bytes(const WideProblem& p) {
  const size_t BH = (size_t)(p.B * p.H), Tp = (size_t)p.Tp;
  const size_t gates = BH * Tp * (4 + 4 + 8);
  const size_t S = BH * Tp * Tp * (p.bf16 ? 4 : 4);  // bf16 hi + lo, or fp32
  return (gates + 255) / 256 * 256 + (S + 255) / 256 * 256;
}

namespace {

struct WideWs {
  float* cw;
  int* zc;
  double* lc;
  void* Sh;
  void* Sl;
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
  return o;
}

template <class OP>
hipError_t wide_run(const WideProblem& p, const WidePtrs& f, bool read, hipStream_t s) {
  const int64_t BH = p.B * p.H;
  const WideWs ws = wide_ws(p, f.ws);
  WGateArgs g{f.eta, f.eta_scalar, f.eta_mul, f.alpha, f.alpha_scalar, f.reset, p.H, p.T, p.Tp, ws.cw, ws.zc, ws.lc};
  timing_begin(GRADLEV_K_WIDE_SCORE, s);
  hipLaunchKernelGGL(wide_gate_kernel, dim3((unsigned)BH), dim3(256), 0, s, g);

  // forward: Q = K = X over d; read: Q = dY over m, K = G.
  WScoreArgs sa{};
  sa.Q = read ? f.dY : f.X;
  sa.K = read ? f.G : f.X;
  sa.T = p.T;
  sa.Tp = p.Tp;
  sa.w = read ? p.m : p.d;
  sa.BH = BH;
  sa.cw = ws.cw;
  sa.zc = ws.zc;
  sa.lc = ws.lc;
  sa.Sh = ws.Sh;
  sa.Sl = OP::kSplit == 2 ? ws.Sl : ws.Sh;
  const int64_t Kp = p.Tp / 128;
  const unsigned sgrid = (unsigned)(BH * 2 * Kp * (Kp + 1));
  if (p.fmode == 0) hipLaunchKernelGGL((wide_score_kernel<OP, 0>), dim3(sgrid), dim3(64), 0, s, sa);
  else if (p.fmode == 1) hipLaunchKernelGGL((wide_score_kernel<OP, 1>), dim3(sgrid), dim3(64), 0, s, sa);
  else hipLaunchKernelGGL((wide_score_kernel<OP, 2>), dim3(sgrid), dim3(64), 0, s, sa);
  timing_end(GRADLEV_K_WIDE_SCORE, s);

  WOutArgs oa{};
  oa.Q = sa.Q;
  oa.W0 = f.W0;
  oa.Sh = ws.Sh;
  oa.Sl = sa.Sl;
  oa.V = read ? f.X : f.G;
  oa.out = read ? f.gtilde : f.Y;
  oa.wq = sa.w;
  oa.wout = read ? p.d : p.m;
  oa.BH = BH;
  oa.H = p.H;
  oa.T = p.T;
  oa.Tp = p.Tp;
  const unsigned ogrid = (unsigned)(BH * (p.Tp / 128) * (oa.wout / 128));
  timing_begin(GRADLEV_K_WIDE_OUT, s);
  if (read) hipLaunchKernelGGL((wide_out_kernel<OP, true>), dim3(ogrid), dim3(256), 0, s, oa);
  else hipLaunchKernelGGL((wide_out_kernel<OP, false>), dim3(ogrid), dim3(256), 0, s, oa);
  timing_end(GRADLEV_K_WIDE_OUT, s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_wide_fwd(const WideProblem& p, const WidePtrs& f, hipStream_t s) {
  return p.bf16 ? wide_run<OpBF16>(p, f, false, s) : wide_run<OpF32>(p, f, false, s);
}

hipError_t launch_wide_read(const WideProblem& p, const WidePtrs& f, hipStream_t s) {
  return p.bf16 ? wide_run<OpBF16>(p, f, true, s) : wide_run<OpF32>(p, f, true, s);
}

}  // namespace gradlev
