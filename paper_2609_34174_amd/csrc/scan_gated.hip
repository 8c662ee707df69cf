// Gated scans of GradLev on gfx950: retention and document resets (Section 3,
// Eq. 2 general form; Eq. 3 with alpha).  For one sequence,
//
//   Delta_{t+1} = alpha_t Delta_t - eta_t g_t x_t^T,      y_t = (W_0 + Delta_t) x_t,
//
// and a reset at token t (Eq. 2 holds within each reset segment) is applied
// as alpha_{t-1} = eta_{t-1} = 0.
//
// Chunk form (C tokens starting at state Delta_n; indices inside the chunk):
//   F[t][s] = prod_{s<j<t} alpha_j              (pair decay, s < t)
//   pre_t   = prod_{j<t} alpha_j,  suf_s = prod_{s<j<C} alpha_j,  tot = prod_j alpha_j
//   y_t        = W_0 x_t + pre_t Delta_n x_t - sum_{s<t} F[t][s] eta_s (x_s . x_t) g_s
//   Delta_{n+1} = tot Delta_n - sum_s eta_s suf_s g_s x_s^T
// All decays are formed as plain products of retentions (no logarithms, no
// divisions), so zero retentions and resets are exact: within a 16-token
// block F is a running product, across blocks it factors as
//   F[t][s] = pin_t * (prod of the whole blocks between) * sin_s
// with pin/sin the products inside t's and s's blocks.
//
// Backward (reverse time, Lambda_e = dL/dDelta at the chunk end):
//   Lambda_{t+1} = suf_t Lambda_e + sum_{u>t} F[u][t] dY_u x_u^T
//   gtilde_t = W_0^T dY_t + pre_t Delta_n^T dY_t - sum_{s<t} F[t][s] eta_s (g_s . dY_t) x_s
//   u_t      = -Lambda_{t+1} x_t,  dG_t = eta_t u_t,  deta_t = <g_t, u_t>
//   dX_t     = gtilde_t - eta_t Lambda_{t+1}^T g_t
//   dalpha_t = <Lambda_{t+1}, Delta_t>_F, which splits by where the two
//              ends of each (write s, read u) pair lie:
//     pre_t suf_t <Lambda_e, Delta_n>          (s before the chunk, u after it)
//   + pre_t sum_{u>t} F[u][t] c3_u             (s before, u inside; c3_u = dY_u . Delta_n x_u)
//   + suf_t sum_{s<t} F[t][s] c2_s             (s inside, u after;  c2_s = -eta_s g_s . Lambda_e x_s)
//   + sum_{s<t<u} F[u][t] F[t][s] K[u][s]      (both inside; K[u][s] = -eta_s (g_s . dY_u)(x_s . x_u))
//     the last term is Z = K F^T on the matrix cores, then a masked column sum.
//   Lambda_n = tot Lambda_e + sum_u pre_u dY_u x_u^T
// The backward needs Delta_n at every chunk start; with retention the writes
// cannot be taken back stably (that would divide by the decays), so a state
// pass stores them first.
#include "scan_common.hpp"

namespace gradlev {

struct GArgs {
  const float* W0;
  const void* X;
  const void* G;
  const void* dY;
  const float* eta;
  float eta_scalar, eta_mul;
  const float* alpha;
  float alpha_scalar;
  const uint8_t* reset;
  int64_t BH, H, T, seg_len, nseg, nchunks;
  float* Y;
  float* gtilde;
  float* dX;
  float* dG;
  float* deta;
  float* dalpha;
  float* aggA;
  float* aggB;
  float* aggBu;
  float* aggD;
  float* states;
};

// ---------------------------------------------------------------------------
// Per-token gates of one chunk.  Thread tid < C loads token t0 + tid's
// retention, step size and the reset flag of the token after it; staging
// applies the reset (alpha = eta = 0 before a reset) and the sequence end
// (alpha = 1, eta = 0 past it, so a partial chunk neither decays nor writes).
// ---------------------------------------------------------------------------
struct GateSrc {
  rsrc_t al, et, rs;
  float a_s, e_s, e_mul;
  bool has_a, has_e, has_r;
};

__device__ __forceinline__ GateSrc gate_src(const GArgs& a, int64_t bh) {
  GateSrc g;
  const int64_t T = a.T;
  g.has_a = a.alpha != nullptr;
  g.has_e = a.eta != nullptr;
  g.has_r = a.reset != nullptr;
  g.al = make_rsrc(g.has_a ? a.alpha + bh * T : nullptr, g.has_a ? (uint32_t)(T * 4) : 0u);
  g.et = make_rsrc(g.has_e ? a.eta + bh * T : nullptr, g.has_e ? (uint32_t)(T * 4) : 0u);
  g.rs = make_rsrc(g.has_r ? a.reset + (bh / a.H) * T : nullptr, g.has_r ? (uint32_t)T : 0u);
  g.a_s = a.alpha_scalar;
  g.e_s = a.eta_scalar;
  g.e_mul = a.eta_mul;
  return g;
}

struct GateReg {
  float a, e;
  uint32_t r;
  __device__ __forceinline__ void load(const GateSrc& g, int64_t t0, bool ok, int tid, int C) {
    const bool mine = ok && tid < C;
    const uint32_t o = mine ? (uint32_t)(t0 + tid) : kOOB;
    a = g.has_a ? buf_load1(g.al, o == kOOB ? kOOB : 4 * o) : g.a_s;
    e = g.e_mul * (g.has_e ? buf_load1(g.et, o == kOOB ? kOOB : 4 * o) : g.e_s);
    // Reset flag of the next token (past the sequence end the load reads 0).
    r = g.has_r ? (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(g.rs, o == kOOB ? kOOB : (int)(o + 1), 0, 0) : 0u;
  }
  // al[t] = retention, et[t] = step size, gm[t] = 1 where the token's gates act.
  __device__ __forceinline__ void stage(float* al, float* et, float* gm, int nvalid, int tid, int C) const {
    if (tid < C) {
      const bool valid = tid < nvalid, cut = r != 0;
      al[tid] = valid ? (cut ? 0.f : a) : 1.f;
      et[tid] = valid && !cut ? e : 0.f;
      if (gm) gm[tid] = valid && !cut ? 1.f : 0.f;
    }
  }
};

// Inclusive product scans inside each 16-lane row: upward (lane i: product
// of lanes <= i of its row) or downward (lanes >= i).
template <bool DOWN>
__device__ __forceinline__ float row_scan_mul(float x) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) {
    float t;
    if (o == 1) t = dpp_move<(DOWN ? kRowShl : kRowShr) + 1>(x, 1.f);
    else if (o == 2) t = dpp_move<(DOWN ? kRowShl : kRowShr) + 2>(x, 1.f);
    else if (o == 4) t = dpp_move<(DOWN ? kRowShl : kRowShr) + 4>(x, 1.f);
    else t = dpp_move<(DOWN ? kRowShl : kRowShr) + 8>(x, 1.f);
    x *= t;
  }
  return x;
}
// The same over the whole wave: rows first, then each row times the totals
// of the rows before it (after it, downward), read back from lanes 15, 31,
// 47 (0, 16, 32, 48 downward) and multiplied in row order.
template <bool DOWN>
__device__ __forceinline__ float wave_scan_mul(float x, int lane) {
  x = row_scan_mul<DOWN>(x);
  const int row = lane >> 4;
  if constexpr (!DOWN) {
    const float r0 = lane_value(x, 15), r1 = lane_value(x, 31), r2 = lane_value(x, 47);
    const float m1 = r0, m2 = r0 * r1, m3 = m2 * r2;
    return x * (row == 0 ? 1.f : row == 1 ? m1 : row == 2 ? m2 : m3);
  } else {
    const float r1 = lane_value(x, 16), r2 = lane_value(x, 32), r3 = lane_value(x, 48);
    const float m2 = r3, m1 = r2 * r3, m0 = r1 * m1;
    return x * (row == 3 ? 1.f : row == 2 ? m2 : row == 1 ? m1 : m0);
  }
}

// Inclusive scan of affine maps z -> A z + B over the wave: lane i ends with
// its own map after those of the lanes below it (upward) or above it
// (downward).  Rows by DPP, then each row after the composed maps of the
// rows before it, read back from their end lanes.
template <int O, bool DOWN>
__device__ __forceinline__ void affine_step(float& A, float& B) {
  const float pa = dpp_move<(DOWN ? kRowShl : kRowShr) + O>(A, 1.f);
  const float pb = dpp_move<(DOWN ? kRowShl : kRowShr) + O>(B, 0.f);
  B = A * pb + B;
  A = A * pa;
}
template <bool DOWN>
__device__ __forceinline__ void affine_scan(float& A, float& B, int lane) {
  affine_step<1, DOWN>(A, B);
  affine_step<2, DOWN>(A, B);
  affine_step<4, DOWN>(A, B);
  affine_step<8, DOWN>(A, B);
  const int row = lane >> 4;
  float ca, cb;  // composed map of the rows before (after) this one
  if constexpr (!DOWN) {
    const float a0 = lane_value(A, 15), b0 = lane_value(B, 15), a1 = lane_value(A, 31), b1 = lane_value(B, 31),
                a2 = lane_value(A, 47), b2 = lane_value(B, 47);
    const float c1a = a1 * a0, c1b = a1 * b0 + b1;
    const float c2a = a2 * c1a, c2b = a2 * c1b + b2;
    ca = row == 1 ? a0 : row == 2 ? c1a : c2a;
    cb = row == 1 ? b0 : row == 2 ? c1b : c2b;
    if (row == 0) return;
  } else {
    const float a3 = lane_value(A, 48), b3 = lane_value(B, 48), a2 = lane_value(A, 32), b2 = lane_value(B, 32),
                a1 = lane_value(A, 16), b1 = lane_value(B, 16);
    const float d2a = a2 * a3, d2b = a2 * b3 + b2;
    const float d1a = a1 * d2a, d1b = a1 * d2b + b1;
    ca = row == 2 ? a3 : row == 1 ? d2a : d1a;
    cb = row == 2 ? b3 : row == 1 ? d2b : d1b;
    if (row == 3) return;
  }
  B = A * cb + B;
  A = A * ca;
}

// Decay products of a chunk (C <= 64), computed by one wave: lane t holds
// alpha_t (1 for lanes >= C).  Product scans, whole chunk and within 16-lane
// blocks.  Also vw[t] = vsign * eta_t * suf_t when vw != null.
template <int C>
__device__ __forceinline__ void gate_scan(const float* al, const float* et, float* pre, float* suf,
                                          float* pin, float* sinv, float* mid, float* tot,
                                          float* vw, float vsign, int lane) {
  constexpr int TB = C / 16;
  const float a = lane < C ? al[lane] : 1.f;
  const float pb = row_scan_mul<false>(a), sb = row_scan_mul<true>(a);
  const float p = wave_scan_mul<false>(a, lane), s = wave_scan_mul<true>(a, lane);
  const float pex = dpp_move<kWaveShr1>(p, 1.f);
  const float sex = dpp_move<kWaveShl1>(s, 1.f);
  const float pbx = dpp_move<kRowShr + 1>(pb, 1.f);
  const float sbx = dpp_move<kRowShl + 1>(sb, 1.f);
  float blk[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) blk[k] = lane_value(pb, 16 * k + 15);
  const float all = lane_value(p, 63);
  if (lane < C) {
    pre[lane] = pex;
    suf[lane] = sex;
    pin[lane] = pbx;
    sinv[lane] = sbx;
    if (vw) vw[lane] = vsign * et[lane] * sex;
  }
  if (lane < TB * TB) {
    const int s0 = lane / TB, t0 = lane % TB;
    float m = 1.f;
#pragma unroll
    for (int k = 0; k < TB; ++k)
      if (k > s0 && k < t0) m *= blk[k];
    mid[lane] = m;
  }
  if (lane == 0) *tot = all;
}

// F[t][s] for the four (s = 16sb + 4q + r, t = 16tb + c) pairs a lane holds in
// a score tile; zero where s >= t.
template <int TB>
__device__ __forceinline__ f32x4 decay4(const float* al, const float* pin, const float* sinv,
                                        const float* mid, int sb, int tb, int q, int c) {
  f32x4 f = zero4();
  if (sb < tb) {
    const float pt = pin[16 * tb + c] * mid[sb * TB + tb];
    const f32x4 ss = *reinterpret_cast<const f32x4*>(sinv + 16 * sb + 4 * q);
    f = pt * ss;
  } else if (sb == tb) {
    // Running product inside the block: prod_{4q+4 <= j < c}, then one more
    // factor alpha_{s+1} per step down to s = 4q, taken only while s+1 < c.
    const float* ab = al + 16 * sb;
    float pr = 1.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) pr *= (j >= 4 * q + 4 && j < c) ? ab[j] : 1.f;
    f[3] = pr;
    f[2] = f[3] * (4 * q + 3 < c ? ab[4 * q + 3] : 1.f);
    f[1] = f[2] * (4 * q + 2 < c ? ab[4 * q + 2] : 1.f);
    f[0] = f[1] * (4 * q + 1 < c ? ab[4 * q + 1] : 1.f);
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (4 * q + r >= c) f[r] = 0.f;
  }
  return f;
}

__device__ __forceinline__ float sum_q(float v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}

// ---------------------------------------------------------------------------
// Segment aggregates with decay.  Wave w < m/16 owns rows i of A, B, Bu.
// Walking the segment's chunks forward:
//   A  <- tot A + sum_s eta_s suf_s g_s x_s^T
//   B  <- B + P sum_u pre_u dY_u x_u^T,   P <- P tot      (P = decay since the segment start)
//   Bu <- Bu + sum_u dY_u x_u^T
// All stored row-major [m][d]; D_k = P at the end.  Modes: kGAggFwd (A, D),
// kGAggBwd (A, B, Bu, D) and kGAggBwdSaved (B, Bu, D: a backward whose
// chunk-start states the forward saved needs no A, and so no G).
// ---------------------------------------------------------------------------
enum GAggMode { kGAggFwd = 0, kGAggBwd = 1, kGAggBwdSaved = 2 };

template <class OP, int D, int M, int C, int MODE>
__global__ void __launch_bounds__(cmax(D, M) / 16 * 64)
agg_gated_kernel(const GArgs a, int64_t nagg) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr bool BWD = MODE != kGAggFwd;  // B, Bu
  constexpr bool WA = MODE != kGAggBwdSaved;  // A
  constexpr int NW = cmax(D, M) / 16, NT = NW * 64;
  constexpr int JB = D / 16, IB = M / 16;
  constexpr bool SPL = OP::kSplit == 2;
  __shared__ E Xs[C * D];
  __shared__ E Vh[WA ? C * M : 1];
  __shared__ E Vl[WA && SPL ? C * M : 1];
  __shared__ E Ds[BWD ? C * M : 1];
  __shared__ E Bh[BWD ? C * M : 1];
  __shared__ E Bl[BWD && SPL ? C * M : 1];
  __shared__ __attribute__((aligned(16))) float al[C], et[C], pre[C], suf[C], pin[C], sinv[C], vw[C], pw[C];
  __shared__ float mid[16], tot;

  int64_t bh, seg;
  if (!map_block(a.BH, a.nseg, bh, seg) || seg >= nagg) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, c = lane & 15, q = lane >> 4;
  const int64_t T = a.T;
  const int64_t t_begin = seg * a.seg_len;
  const int64_t t_end = t_begin + a.seg_len < T ? t_begin + a.seg_len : T;
  const rsrc_t X = make_rsrc(static_cast<const E*>(a.X) + bh * T * D, (uint32_t)(T * D * sizeof(E)));
  const rsrc_t G = make_rsrc(WA ? static_cast<const E*>(a.G) + bh * T * M : nullptr, WA ? (uint32_t)(T * M * sizeof(E)) : 0u);
  const rsrc_t Dy = make_rsrc(BWD ? static_cast<const E*>(a.dY) + bh * T * M : nullptr, BWD ? (uint32_t)(T * M * sizeof(E)) : 0u);
  const GateSrc gs = gate_src(a, bh);

  f32x4 accA[JB], accB[JB], accU[JB];
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) accA[jb] = accB[jb] = accU[jb] = zero4();
  float P = 1.f;

  // Chunks staged two ahead in two register slots; every pass runs both
  // slots' steps (a step past the segment end sees zero tiles, unit decay
  // and zero step sizes, so it changes nothing), which keeps the memory
  // operations branch-free.
  Tile4<OP, C, D, NT> xr[2];
  Tile4<OP, C, M, NT> gr[2], dr[2];
  GateReg ar[2];
  auto fetch = [&](int k, int64_t t0) {
    const bool ok = t0 < t_end;
    ar[k].load(gs, t0, ok, tid, C);
    xr[k].load(X, ok ? (uint32_t)(t0 * D * sizeof(E)) : kOOB, tid);
    if (WA) gr[k].load(G, ok ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
    if (BWD) dr[k].load(Dy, ok ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
  };
  fetch(0, t_begin);
  __builtin_amdgcn_sched_barrier(0);  // slot order (the loop's first wait holds on entry too)
  fetch(1, t_begin + C);
  auto chunk = [&](int k, int64_t t0) {
    const int nvalid = t0 < t_end ? (int)(t_end - t0 < C ? t_end - t0 : C) : 0;
    __syncthreads();
    ar[k].stage(al, et, nullptr, nvalid, tid, C);
    xr[k].store(Xs, tid);
    if (BWD) dr[k].store(Ds, tid);
    __syncthreads();
    if (w == 0) gate_scan<C>(al, et, pre, suf, pin, sinv, mid, &tot, WA ? vw : nullptr, 1.f, lane);
    __syncthreads();
    if (BWD && tid < C) pw[tid] = P * pre[tid];
    if (WA) gr[k].store_scaled(Vh, Vl, tid, vw);
    __syncthreads();
    if (BWD) dr[k].store_scaled(Bh, Bl, tid, pw);
    const float tt = tot;
    fetch(k, t0 + 2 * C);
    __syncthreads();
    if (w < IB) {
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) accA[jb] *= tt;
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
        F vh{}, vl{};
        if constexpr (WA) {
          vh = OP::load_t(Vh, M, 32 * kb, 16 * w, lane);
          vl = vh;
          if constexpr (SPL) vl = OP::load_t(Vl, M, 32 * kb, 16 * w, lane);
        }
        F bh2 = vh, bl2 = vh, dv = vh;
        if constexpr (BWD) {
          bh2 = OP::load_t(Bh, M, 32 * kb, 16 * w, lane);
          if constexpr (SPL) bl2 = OP::load_t(Bl, M, 32 * kb, 16 * w, lane);
          dv = OP::load_t(Ds, M, 32 * kb, 16 * w, lane);
        }
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) {
          const F xa = OP::load_t(Xs, D, 32 * kb, 16 * jb, lane);
          if constexpr (WA) accA[jb] = mma_split_b<OP>(accA[jb], xa, vh, vl);
          if constexpr (BWD) {
            accB[jb] = mma_split_b<OP>(accB[jb], xa, bh2, bl2);
            accU[jb] = OP::mma(accU[jb], xa, dv);
          }
        }
      }
    }
    P *= tt;
  };
  for (int64_t t0 = t_begin; t0 < t_end; t0 += 2 * C) {
    chunk(0, t0);
    chunk(1, t0 + C);
  }
  if (w < IB) {
    // acc[jb] holds A^T[j = 16jb + 4q + r][i = 16w + c]; stored as A[i][j].
    const int64_t base = (bh * a.nseg + seg) * M * D + (int64_t)(16 * w + c) * D + 4 * q;
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) {
      if (WA) *reinterpret_cast<f32x4*>(a.aggA + base + 16 * jb) = accA[jb];
      if (BWD) {
        *reinterpret_cast<f32x4*>(a.aggB + base + 16 * jb) = accB[jb];
        *reinterpret_cast<f32x4*>(a.aggBu + base + 16 * jb) = accU[jb];
      }
    }
  }
  if (tid == 0) a.aggD[bh * a.nseg + seg] = P;
}

// Start state of a segment from the aggregates of the segments before it:
// S = sum_{j<seg} (prod_{j<i<seg} D_i) A_j, summed in segment order.  Element
// (i, j) of the [m][d] aggregates; the caller returns -S.
__device__ __forceinline__ float seg_prefix(const GArgs& a, int64_t bh, int64_t seg, int64_t e, int64_t md) {
  float s = 0.f;
  const float* A = a.aggA + bh * a.nseg * md + e;
  for (int64_t j = 0; j < seg; ++j) s = a.aggD[bh * a.nseg + j] * s + A[j * md];
  return s;
}

// ---------------------------------------------------------------------------
// Gated forward.  Wave w < m/16 owns rows i in [16w, 16w+16) of the state,
// held as Delta^T tiles (rows j, cols i), and the matching columns of Y.
// ---------------------------------------------------------------------------
template <class OP, int D, int M, int C>
__global__ void __launch_bounds__(cmax(D, M) / 16 * 64)
fwd_gated_kernel(const GArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int NW = cmax(D, M) / 16, NT = NW * 64;
  constexpr int TB = C / 16, JB = D / 16, IB = M / 16;
  constexpr bool SPL = OP::kSplit == 2;
  __shared__ E Xs[C * D];
  __shared__ E Gs[C * M];
  __shared__ E Vh[C * M];
  __shared__ E Vl[SPL ? C * M : 1];
  __shared__ __attribute__((aligned(16))) float al[C], et[C], pre[C], suf[C], pin[C], sinv[C], vw[C];
  __shared__ float mid[16], tot;
  // Y staged through LDS for whole-row stores (16-row x 64-byte tile stores
  // stream to HBM at a fraction of the full-line rate); fp32 [C][M + 4], the
  // pad staggering the owners' tile writes over the banks.
  constexpr int YP = M + 4;
  constexpr bool YSTG = OP::kSplit == 2 && D == 64 && M == 64 && C == 64 && NT == C * M / 16;
  __shared__ __attribute__((aligned(16))) float Ys[YSTG ? C * YP : 4];

  int64_t bh, seg;
  if (!map_block(a.BH, a.nseg, bh, seg)) return;
  const int tid = threadIdx.x, lane = tid & 63, c = lane & 15, q = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: block indices stay scalar
  const int64_t h = bh % a.H;
  const int64_t T = a.T;
  const int64_t md = (int64_t)M * D;
  const int64_t t_begin = seg * a.seg_len;
  const int64_t t_end = t_begin + a.seg_len < T ? t_begin + a.seg_len : T;
  const rsrc_t X = make_rsrc(static_cast<const E*>(a.X) + bh * T * D, (uint32_t)(T * D * sizeof(E)));
  const rsrc_t G = make_rsrc(static_cast<const E*>(a.G) + bh * T * M, (uint32_t)(T * M * sizeof(E)));
  const rsrc_t Y = make_rsrc(a.Y + bh * T * M, (uint32_t)(T * M * 4));
  const GateSrc gs = gate_src(a, bh);

  // State Delta^T[j = 16jb + 4q + r][i = 16w + c] and the slow weights in the
  // same layout, split once for the W_0 read.
  f32x4 Dt[JB];
  F w0h[D / 32], w0l[D / 32];
  if (w < IB) {
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        Dt[jb][r] = seg > 0 ? -seg_prefix(a, bh, seg, (int64_t)(16 * w + c) * D + 16 * jb + 4 * q + r, md) : 0.f;
    }
    const float* w0 = a.W0 + h * md + (int64_t)(16 * w + c) * D + 4 * q;
#pragma unroll
    for (int kb = 0; kb < D / 32; ++kb) {
      const f32x4 lo4 = *reinterpret_cast<const f32x4*>(w0 + 32 * kb);
      const f32x4 hi4 = *reinterpret_cast<const f32x4*>(w0 + 32 * kb + 16);
      OP::split(cat(lo4, hi4), w0h[kb], w0l[kb]);
    }
  }

  Tile4<OP, C, D, NT> xr;
  Tile4<OP, C, M, NT> gr;
  GateReg ar;
  auto fetch = [&](int64_t t0) {
    const bool ok = t0 < t_end;
    ar.load(gs, t0, ok, tid, C);
    xr.load(X, ok ? (uint32_t)(t0 * D * sizeof(E)) : kOOB, tid);
    gr.load(G, ok ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
  };
  fetch(t_begin);
  for (int64_t t0 = t_begin; t0 < t_end; t0 += C) {
    const int nvalid = (int)(t_end - t0 < C ? t_end - t0 : C);
    __syncthreads();
    ar.stage(al, et, nullptr, nvalid, tid, C);
    xr.store(Xs, tid);
    gr.store(Gs, tid);
    __syncthreads();
    if (w == 0) gate_scan<C>(al, et, pre, suf, pin, sinv, mid, &tot, vw, -1.f, lane);
    __syncthreads();
    if (a.states && w < IB) {
      // Saved for a backward with the same chunk: Delta at this chunk's
      // start, in the order the backward's lanes load it (tiles of rows
      // 16ib + 4q' + r', columns 16w' + c', one f32x4 per (w', ib, lane')).
      // Issued here, before the longest stretch without a barrier, so that
      // the stores retire under the output computation.
      float* st = a.states + (bh * a.nchunks + t0 / C) * md + 256 * w + 4 * (16 * (c >> 2)) + (c & 3);
#pragma unroll
      for (int jb = 0; jb < JB; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) st[jb * IB * 256 + 4 * (4 * q + r)] = Dt[jb][r];
    }
    gr.store_scaled(Vh, Vl, tid, vw);  // -eta_s suf_s g_s, read by the carry after a barrier
    fetch(t0 + C);
    if (w < IB) {
      f32x4 acc[TB];
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) acc[tb] = zero4();
      // pre_t Delta_n x_t
#pragma unroll
      for (int kb = 0; kb < D / 32; ++kb) {
        F dh, dl;
        OP::split(cat(Dt[2 * kb], Dt[2 * kb + 1]), dh, dl);
#pragma unroll
        for (int tb = 0; tb < TB; ++tb)
          acc[tb] = mma_split_a<OP>(acc[tb], dh, dl, OP::load_n(Xs, D, 16 * tb, 32 * kb, lane));
      }
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) acc[tb] *= pre[16 * tb + c];
      // + W_0 x_t
#pragma unroll
      for (int kb = 0; kb < D / 32; ++kb) {
#pragma unroll
        for (int tb = 0; tb < TB; ++tb)
          acc[tb] = mma_split_a<OP>(acc[tb], w0h[kb], w0l[kb], OP::load_n(Xs, D, 16 * tb, 32 * kb, lane));
      }
      // - sum_{s<t} F[t][s] eta_s (x_s . x_t) g_s: score tiles built per wave.
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
        const F gq = OP::load_t(Gs, M, 32 * kb, 16 * w, lane);
#pragma unroll
        for (int tb = 2 * kb; tb < TB; ++tb) {
          f32x8 sv;
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int sb = 2 * kb + hh;
            f32x4 st = zero4();
            if (sb <= tb) {
#pragma unroll
              for (int kj = 0; kj < D / 32; ++kj)
                st = OP::mma(st, OP::load_n(Xs, D, 16 * sb, 32 * kj, lane), OP::load_n(Xs, D, 16 * tb, 32 * kj, lane));
              const f32x4 f = decay4<TB>(al, pin, sinv, mid, sb, tb, q, c);
              const f32x4 es = *reinterpret_cast<const f32x4*>(et + 16 * sb + 4 * q);
              st = st * f * (-es);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) sv[4 * hh + r] = st[r];
          }
          F sq, lo;
          OP::split(sv, sq, lo);
          acc[tb] = OP::mma(acc[tb], gq, sq);
        }
      }
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        const int t = 16 * tb + c;
        if constexpr (YSTG) *reinterpret_cast<f32x4*>(Ys + t * YP + 16 * w + 4 * q) = acc[tb];
        else buf_store4(Y, (uint32_t)(((t0 + t) * M + 16 * w + 4 * q) * 4), acc[tb]);
      }
    }
    __syncthreads();
    if constexpr (YSTG) {
      // Whole rows: thread tid stores 16 bytes of row tid / (M/4), so each
      // wave writes four 256-byte rows (rows past T are dropped).  Ys is
      // rewritten only after the next chunk's third barrier.
#pragma unroll
      for (int i = 0; i < C * M / 4 / NT; ++i) {
        const int e = tid + i * NT, r = e / (M / 4), c4 = 4 * (e % (M / 4));
        buf_store4(Y, (uint32_t)(((t0 + r) * M + c4) * 4), *reinterpret_cast<const f32x4*>(Ys + r * YP + c4));
      }
    }
    if (w < IB) {
      // Carry: Delta^T <- tot Delta^T + X^T V.
      const float tt = tot;
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) Dt[jb] *= tt;
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
        const F vh = OP::load_t(Vh, M, 32 * kb, 16 * w, lane);
        F vl = vh;
        if constexpr (SPL) vl = OP::load_t(Vl, M, 32 * kb, 16 * w, lane);
#pragma unroll
        for (int jb = 0; jb < JB; ++jb)
          Dt[jb] = mma_split_b<OP>(Dt[jb], OP::load_t(Xs, D, 32 * kb, 16 * jb, lane), vh, vl);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Chunk-start states for the backward.  Wave w < d/16 owns columns j in
// [16w, 16w+16) and holds Delta tiles (rows i = 16ib + 4q + r, cols j =
// 16w + c); chunk n's state is stored as f32x4 per (w, ib, lane) at
// states[bh][n], which is the order the backward loads it in.
// ---------------------------------------------------------------------------
template <class OP, int D, int M, int C>
__global__ void __launch_bounds__(cmax(D, M) / 16 * 64)
states_gated_kernel(const GArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int NW = cmax(D, M) / 16, NT = NW * 64;
  constexpr int JB = D / 16, IB = M / 16;
  constexpr bool SPL = OP::kSplit == 2;
  __shared__ E Xs[C * D];
  __shared__ E Vh[C * M];
  __shared__ E Vl[SPL ? C * M : 1];
  __shared__ __attribute__((aligned(16))) float al[C], et[C], pre[C], suf[C], pin[C], sinv[C], vw[C];
  __shared__ float mid[16], tot;

  int64_t bh, seg;
  if (!map_block(a.BH, a.nseg, bh, seg)) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, c = lane & 15, q = lane >> 4;
  const int64_t T = a.T;
  const int64_t md = (int64_t)M * D;
  const int64_t t_begin = seg * a.seg_len;
  const int64_t t_end = t_begin + a.seg_len < T ? t_begin + a.seg_len : T;
  const rsrc_t X = make_rsrc(static_cast<const E*>(a.X) + bh * T * D, (uint32_t)(T * D * sizeof(E)));
  const rsrc_t G = make_rsrc(static_cast<const E*>(a.G) + bh * T * M, (uint32_t)(T * M * sizeof(E)));
  const GateSrc gs = gate_src(a, bh);

  f32x4 St[IB];
  if (w < JB) {
#pragma unroll
    for (int ib = 0; ib < IB; ++ib) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        St[ib][r] = seg > 0 ? -seg_prefix(a, bh, seg, (int64_t)(16 * ib + 4 * q + r) * D + 16 * w + c, md) : 0.f;
    }
  }
  Tile4<OP, C, D, NT> xr;
  Tile4<OP, C, M, NT> gr;
  GateReg ar;
  auto fetch = [&](int64_t t0) {
    const bool ok = t0 < t_end;
    ar.load(gs, t0, ok, tid, C);
    xr.load(X, ok ? (uint32_t)(t0 * D * sizeof(E)) : kOOB, tid);
    gr.load(G, ok ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
  };
  fetch(t_begin);
  for (int64_t t0 = t_begin; t0 < t_end; t0 += C) {
    const int nvalid = (int)(t_end - t0 < C ? t_end - t0 : C);
    if (w < JB) {
      float* dst = a.states + (bh * a.nchunks + t0 / C) * md + (int64_t)w * IB * 256 + 4 * lane;
#pragma unroll
      for (int ib = 0; ib < IB; ++ib) *reinterpret_cast<f32x4*>(dst + 256 * ib) = St[ib];
    }
    if (t0 + C >= t_end) break;  // the last chunk's carry is not needed
    __syncthreads();
    ar.stage(al, et, nullptr, nvalid, tid, C);
    xr.store(Xs, tid);
    __syncthreads();
    if (w == 0) gate_scan<C>(al, et, pre, suf, pin, sinv, mid, &tot, vw, -1.f, lane);
    __syncthreads();
    gr.store_scaled(Vh, Vl, tid, vw);
    fetch(t0 + C);
    __syncthreads();
    if (w < JB) {
      const float tt = tot;
#pragma unroll
      for (int ib = 0; ib < IB; ++ib) St[ib] *= tt;
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
        const F xq = OP::load_t(Xs, D, 32 * kb, 16 * w, lane);
#pragma unroll
        for (int ib = 0; ib < IB; ++ib) {
          const F vh = OP::load_t(Vh, M, 32 * kb, 16 * ib, lane);
          F vl = vh;
          if constexpr (SPL) vl = OP::load_t(Vl, M, 32 * kb, 16 * ib, lane);
          St[ib] = mma_split_a<OP>(St[ib], vh, vl, xq);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Gated backward.  Wave w < d/16 owns columns j in [16w, 16w+16) of Lambda
// (tiles rows i, cols j), of gtilde and of dX.  The rows i in [16r, 16r+16)
// of u and dG belong to wave r as well (SPLITW false: max(d, m)/16 waves), or
// to a wave of their own, w = d/16 + r (SPLITW true: d/16 + m/16 waves, twice
// as many per CU to hide each other's latency).  Chunks run from the
// segment's last to its first.
// ---------------------------------------------------------------------------
template <class OP, int D, int M, int C, bool SPLITW>
__global__ void __launch_bounds__((SPLITW ? D / 16 + M / 16 : cmax(D, M) / 16) * 64)
bwd_gated_kernel(const GArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int NW = SPLITW ? D / 16 + M / 16 : cmax(D, M) / 16, NT = NW * 64;
  constexpr int TB = C / 16, JB = D / 16, IB = M / 16;
  constexpr bool SPL = OP::kSplit == 2;
  constexpr int LO = SPL ? 1 : 0;
  __shared__ E Xs[C * D];
  __shared__ E Gs[C * M];
  __shared__ E Ds[C * M];
  __shared__ E Dph[C * M];              // pre_u dY_u
  __shared__ E Dpl[LO ? C * M : 1];
  // Chunk matrices [row][col], row = the later token.
  __shared__ E Plh[C * C], Pll[LO ? C * C : 1];   // F
  __shared__ E Peh[C * C], Pel[LO ? C * C : 1];   // F (dY_t . g_s)
  __shared__ E E1h[C * C], E1l[LO ? C * C : 1];   // -eta_s F (dY_t . g_s)
  __shared__ E Pgh[C * C], Pgl[LO ? C * C : 1];   // F (x_t . x_s)
  __shared__ E Kh[C * C], Kl[LO ? C * C : 1];     // -eta_s (dY_t . g_s)(x_t . x_s), s < t
  __shared__ E LTh[D * M], LTl[LO ? D * M : 1];   // Lambda_e^T [j][i]
  __shared__ __attribute__((aligned(16))) float al[C], et[C], gm[C], pre[C], suf[C], pin[C], sinv[C];
  __shared__ float c3p[NW][C], c2p[NW][C], dep[NW][C], dap[NW][C];
  __shared__ float t1p[NW], mid[16], tot;

  int64_t bh, seg;
  if (!map_block(a.BH, a.nseg, bh, seg)) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, c = lane & 15, q = lane >> 4;
  const int64_t h = bh % a.H;
  const int64_t T = a.T;
  const int64_t md = (int64_t)M * D;
  const int64_t t_begin = seg * a.seg_len;
  const int64_t t_end = t_begin + a.seg_len < T ? t_begin + a.seg_len : T;
  const int64_t n_first = t_begin / C, n_last = (t_end - 1) / C;
  const rsrc_t X = make_rsrc(static_cast<const E*>(a.X) + bh * T * D, (uint32_t)(T * D * sizeof(E)));
  const rsrc_t G = make_rsrc(static_cast<const E*>(a.G) + bh * T * M, (uint32_t)(T * M * sizeof(E)));
  const rsrc_t Dy = make_rsrc(static_cast<const E*>(a.dY) + bh * T * M, (uint32_t)(T * M * sizeof(E)));
  const rsrc_t Og = make_rsrc(a.gtilde ? a.gtilde + bh * T * D : nullptr, a.gtilde ? (uint32_t)(T * D * 4) : 0u);
  const rsrc_t Ox = make_rsrc(a.dX ? a.dX + bh * T * D : nullptr, a.dX ? (uint32_t)(T * D * 4) : 0u);
  const rsrc_t Od = make_rsrc(a.dG ? a.dG + bh * T * M : nullptr, a.dG ? (uint32_t)(T * M * 4) : 0u);
  const rsrc_t Oe = make_rsrc(a.deta ? a.deta + bh * T : nullptr, a.deta ? (uint32_t)(T * 4) : 0u);
  const rsrc_t Oa = make_rsrc(a.dalpha ? a.dalpha + bh * T : nullptr, a.dalpha ? (uint32_t)(T * 4) : 0u);
  const rsrc_t Sn = make_rsrc(a.states + bh * a.nchunks * md, (uint32_t)(a.nchunks * md * 4));
  const GateSrc gs = gate_src(a, bh);

  // Lambda at the segment end: sum_{j>seg} (prod_{seg<i<j} D_i) B_j, summed
  // from the last segment down.  Tiles rows i = 16ib + 4q + r, cols j = 16w + c.
  f32x4 Lam[IB];
  F w0h[M / 32], w0l[M / 32];
  if (w < JB) {
#pragma unroll
    for (int ib = 0; ib < IB; ++ib) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t e = (int64_t)(16 * ib + 4 * q + r) * D + 16 * w + c;
        float s = 0.f;
        for (int64_t j = a.nseg - 1; j > seg; --j) s = a.aggD[bh * a.nseg + j] * s + a.aggB[(bh * a.nseg + j) * md + e];
        Lam[ib][r] = s;
      }
    }
    // W_0 tiles in the same layout, split for the read side (operand rows j, k = i).
#pragma unroll
    for (int kb = 0; kb < M / 32; ++kb) {
      f32x8 v;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = a.W0[h * md + (int64_t)(32 * kb + 16 * (e >> 2) + 4 * q + (e & 3)) * D + 16 * w + c];
      OP::split(v, w0h[kb], w0l[kb]);
    }
  }

  // Tiles above the diagonal are never written: zero once (the first chunk's
  // barriers order this before any read).
  for (int i = tid; i < C * C; i += NT) {
    Plh[i] = Peh[i] = E1h[i] = Pgh[i] = Kh[i] = (E)0.f;
    if constexpr (SPL) Pll[i] = Pel[i] = E1l[i] = Pgl[i] = Kl[i] = (E)0.f;
  }

  Tile4<OP, C, D, NT> xr;
  Tile4<OP, C, M, NT> gr, dr;
  GateReg ar;
  f32x4 dnx[IB];
  auto fetch = [&](int64_t n) {
    const bool ok = n >= n_first;
    const int64_t t0 = n * C;
    ar.load(gs, t0, ok, tid, C);
    xr.load(X, ok ? (uint32_t)(t0 * D * sizeof(E)) : kOOB, tid);
    gr.load(G, ok ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
    dr.load(Dy, ok ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
#pragma unroll
    for (int ib = 0; ib < IB; ++ib)
      dnx[ib] = buf_load4(Sn, ok && w < JB ? (uint32_t)((n * md + (int64_t)w * IB * 256 + 256 * ib + 4 * lane) * 4) : kOOB,
                          (const float*)nullptr);
  };
  fetch(n_last);
  for (int64_t n = n_last; n >= n_first; --n) {
    // Lane and thread indices as the loop sees them: opaque to the compiler,
    // so that LDS addresses are formed per use instead of being hoisted out
    // of the loop into hundreds of live registers.
    int ln = lane, td = tid;
    asm volatile("" : "+v"(ln), "+v"(td));
    const int c = ln & 15, q = ln >> 4;
    // Fragment address offsets of this lane (precomputed at 64 x 64),
    // those of the wave's own column blocks, and the lane part of the
    // transposed element reads of the F tile (rows 4q + r, column c).
    constexpr bool PRE = D == 64 && M == 64;
    const LaneOff<D, sizeof(E), PRE> lD = lane_off<D, sizeof(E), PRE>(ln);
    const LaneOff<M, sizeof(E), PRE> lM = lane_off_like<M>(lD);
    const LaneOff<C, sizeof(E), PRE> lC = lane_off_like<C>(lM);
    const int rw = SPLITW ? w - JB : w;  // row block of u and dG
    const typename OP::tcol tDw = OP::make_tcol(lD, 16 * w), tMr = OP::make_tcol(lM, 16 * rw);
    const int nDw = PRE ? lD.nat_rt(0, 16 * w) : 0, nMr = PRE ? lM.nat_rt(0, 16 * rw) : 0;
    // Element r of the 4-element chunk (row 16tb + c, column 16wb + 4q) of
    // X or G, and element (16ub + 4q + r, 16tb + c) of the F tile.
    auto x_el = [&](int tb, int r) -> float {
      if constexpr (PRE) return (float)at_byte<E>(Xs, 16 * tb * D * (int)sizeof(E) + nDw + r * (int)sizeof(E));
      else return (float)Xs[lds_off(16 * tb + c, 16 * w + 4 * q + r, D)];
    };
    auto g_el = [&](int tb, int r) -> float {
      if constexpr (PRE) return (float)at_byte<E>(Gs, 16 * tb * M * (int)sizeof(E) + nMr + r * (int)sizeof(E));
      else return (float)Gs[lds_off(16 * tb + c, 16 * rw + 4 * q + r, M)];
    };
    int fcol = 4 * q * C + 4 * ((c >> 2) ^ q) + (c & 3);
    if constexpr (PRE) asm volatile("" : "+v"(fcol));
    auto f_off = [&](int ub, int tb, int r) {
      if constexpr (PRE) return (16 * ub + r) * C + 4 * ((4 * tb) ^ ((4 * r) & (C / 4 - 1))) + fcol;
      else return lds_off(16 * ub + 4 * q + r, 16 * tb + c, C);
    };
    const int64_t t0 = n * C;
    const int nvalid = (int)(t_end - t0 < C ? t_end - t0 : C);
    f32x4 dn[IB];
#pragma unroll
    for (int ib = 0; ib < IB; ++ib) dn[ib] = dnx[ib];
    __syncthreads();
    ar.stage(al, et, gm, nvalid, td, C);
    xr.store(Xs, td);
    gr.store(Gs, td);
    dr.store(Ds, td);
    for (int i = td; i < NW * C; i += NT) (&dap[0][0])[i] = 0.f;
    // Publish Lambda_e^T [j][i] (split) and the partial <Lambda_e, Delta_n>.
    if (w < JB) {
      float t1 = 0.f;
#pragma unroll
      for (int ib = 0; ib < IB; ++ib) {
        const int o = lM.nat(16 * w, 16 * ib);
        OP::store4_split(ptr_byte<E>(LTh, o), ptr_byte<E>(LTl, o), Lam[ib]);
#pragma unroll
        for (int r = 0; r < 4; ++r) t1 += Lam[ib][r] * dn[ib][r];
      }
      t1 = wave_sum(t1);
      if (ln == 0) t1p[w] = t1;
    }
    __syncthreads();
    if (w == 0) gate_scan<C>(al, et, pre, suf, pin, sinv, mid, &tot, nullptr, 0.f, ln);
    __syncthreads();
    dr.store_scaled(Dph, Dpl, td, pre);
    // Chunk matrices, lower tiles (tb >= sb) spread over the waves.
#pragma unroll
    for (int idx = 0; idx < TB * (TB + 1) / 2; ++idx) {
      if (idx % NW != w) continue;
      int tb = 0;
      while ((tb + 1) * (tb + 2) / 2 <= idx) ++tb;
      const int sb = idx - tb * (tb + 1) / 2;
      // gx[r] = x_s . x_t, ed[r] = g_s . dY_t with s = 16sb + 4q + r, t = 16tb + c.
      f32x4 gx = zero4(), ed = zero4();
#pragma unroll
      for (int kb = 0; kb < D / 32; ++kb)
        gx = OP::mma(gx, OP::load_n(Xs, lD, 16 * sb, 32 * kb), OP::load_n(Xs, lD, 16 * tb, 32 * kb));
#pragma unroll
      for (int kb = 0; kb < M / 32; ++kb)
        ed = OP::mma(ed, OP::load_n(Gs, lM, 16 * sb, 32 * kb), OP::load_n(Ds, lM, 16 * tb, 32 * kb));
      const f32x4 f = decay4<TB>(al, pin, sinv, mid, sb, tb, q, c);
      const f32x4 es = *reinterpret_cast<const f32x4*>(et + 16 * sb + 4 * q);
      const int t = 16 * tb + c;
      f32x4 kk;
#pragma unroll
      for (int r = 0; r < 4; ++r) kk[r] = (16 * sb + 4 * q + r < t) ? -es[r] * ed[r] * gx[r] : 0.f;
      const int o = lC.nat(16 * tb, 16 * sb);
      OP::store4_split(ptr_byte<E>(Plh, o), ptr_byte<E>(Pll, o), f);
      OP::store4_split(ptr_byte<E>(Peh, o), ptr_byte<E>(Pel, o), f * ed);
      OP::store4_split(ptr_byte<E>(E1h, o), ptr_byte<E>(E1l, o), -es * f * ed);
      OP::store4_split(ptr_byte<E>(Pgh, o), ptr_byte<E>(Pgl, o), f * gx);
      OP::store4_split(ptr_byte<E>(Kh, o), ptr_byte<E>(Kl, o), kk);
    }
    const float tt = tot;
    fetch(n - 1);
    __syncthreads();

    F xt[C / 32];
    if (w < JB) {
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) xt[kb] = OP::load_t(Xs, lD, 32 * kb, tDw);
      // Read side: gtilde = W_0^T dY + pre Delta_n^T dY - (E1 X); write side of dX.
      // The chunk's state and Lambda_e are split once for all token blocks
      // at 64 x 64 (elsewhere per block: the held halves would spill).
      constexpr bool HOIST = D == 64 && M == 64;
      F dnh[HOIST ? M / 32 : 1], dnl[HOIST ? M / 32 : 1], lmh[HOIST ? M / 32 : 1], lml[HOIST ? M / 32 : 1];
      if constexpr (HOIST) {
#pragma unroll
        for (int kb = 0; kb < M / 32; ++kb) {
          OP::split(cat(dn[2 * kb], dn[2 * kb + 1]), dnh[kb], dnl[kb]);
          OP::split(cat(Lam[2 * kb], Lam[2 * kb + 1]), lmh[kb], lml[kb]);
        }
      }
      auto dn_split = [&](int kb, F& h, F& l) {
        if constexpr (HOIST) {
          h = dnh[kb];
          l = dnl[kb];
        } else {
          OP::split(cat(dn[2 * kb], dn[2 * kb + 1]), h, l);
        }
      };
      auto lam_split = [&](int kb, F& h, F& l) {
        if constexpr (HOIST) {
          h = lmh[kb];
          l = lml[kb];
        } else {
          OP::split(cat(Lam[2 * kb], Lam[2 * kb + 1]), h, l);
        }
      };
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        const int t = 16 * tb + c;
        f32x4 ad = zero4();
#pragma unroll
        for (int kb = 0; kb < M / 32; ++kb) {
          F dh, dl;
          dn_split(kb, dh, dl);
          ad = mma_split_a<OP>(ad, dh, dl, OP::load_n(Ds, lM, 16 * tb, 32 * kb));
        }
        // c3_t partial: x_t . (Delta_n^T dY_t) over this wave's j.
        float c3 = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) c3 += x_el(tb, r) * ad[r];
        c3 = sum_q(c3);
        if (q == 0) c3p[w][t] = c3;
        f32x4 ag = ad * pre[t];
#pragma unroll
        for (int kb = 0; kb < M / 32; ++kb)
          ag = mma_split_a<OP>(ag, w0h[kb], w0l[kb], OP::load_n(Ds, lM, 16 * tb, 32 * kb));
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
          const F eh = OP::load_n(E1h, lC, 16 * tb, 32 * kb);
          F el = eh;
          if constexpr (SPL) el = OP::load_n(E1l, lC, 16 * tb, 32 * kb);
          ag = mma_split_b<OP>(ag, xt[kb], eh, el);
        }
        const uint32_t off = (uint32_t)(((t0 + t) * D + 16 * w + 4 * q) * 4);
        if (a.gtilde) buf_store4(Og, off, ag);
        if (a.dX) {
          // Lambda_e^T g_t (scaled by suf_t) and sum_{u>t} F[u][t] (dY_u . g_t) x_u.
          f32x4 qs = zero4(), qi = zero4();
#pragma unroll
          for (int kb = 0; kb < M / 32; ++kb) {
            F lh, ll;
            lam_split(kb, lh, ll);
            qs = mma_split_a<OP>(qs, lh, ll, OP::load_n(Gs, lM, 16 * tb, 32 * kb));
          }
#pragma unroll
          for (int kb = 0; kb < C / 32; ++kb) {
            const F ph = OP::load_t(Peh, lC, 32 * kb, 16 * tb);
            F pl = ph;
            if constexpr (SPL) pl = OP::load_t(Pel, lC, 32 * kb, 16 * tb);
            qi = mma_split_b<OP>(qi, xt[kb], ph, pl);
          }
          const f32x4 dx = ag - et[t] * (suf[t] * qs + qi);
          buf_store4(Ox, off, dx);
        }
      }
    }
    if (SPLITW ? (w >= JB && w < JB + IB) : w < IB) {
      // u_t = -(suf_t Lambda_e x_t + sum_{u>t} F[u][t] (x_u . x_t) dY_u).
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        const int t = 16 * tb + c;
        f32x4 us = zero4(), ui = zero4();
#pragma unroll
        for (int kb = 0; kb < D / 32; ++kb) {
          const F lh = OP::load_t(LTh, lM, 32 * kb, tMr);
          F ll = lh;
          if constexpr (SPL) ll = OP::load_t(LTl, lM, 32 * kb, tMr);
          us = mma_split_a<OP>(us, lh, ll, OP::load_n(Xs, lD, 16 * tb, 32 * kb));
        }
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
          const F ph = OP::load_t(Pgh, lC, 32 * kb, 16 * tb);
          F pl = ph;
          if constexpr (SPL) pl = OP::load_t(Pgl, lC, 32 * kb, 16 * tb);
          ui = mma_split_b<OP>(ui, OP::load_t(Ds, lM, 32 * kb, tMr), ph, pl);
        }
        const f32x4 u = -(suf[t] * us + ui);
        float c2 = 0.f, de = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float gv = g_el(tb, r);
          c2 += gv * us[r];
          de += gv * u[r];
        }
        c2 = sum_q(c2);
        de = sum_q(de);
        if (q == 0) {
          c2p[rw][t] = c2;
          dep[rw][t] = de;
        }
        if (a.dG) buf_store4(Od, (uint32_t)(((t0 + t) * M + 16 * rw + 4 * q) * 4), et[t] * u);
      }
    }
    if (a.dalpha) {
      // Z[u][t] = sum_s K[u][s] F[t][s]; column sums of F[u][t] Z[u][t] over u > t.
      // With split roles the tiles are dealt from the u/dG waves first: the
      // gtilde/dX waves have the longer phase before this one.
#pragma unroll
      for (int idx = 0; idx < TB * (TB + 1) / 2; ++idx) {
        if ((SPLITW ? (idx + JB) % NW : idx % NW) != w) continue;
        int ub = 0;
        while ((ub + 1) * (ub + 2) / 2 <= idx) ++ub;
        const int tb = idx - ub * (ub + 1) / 2;
        f32x4 z = zero4();
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
          if (32 * kb > 16 * tb + 15) break;
          const F kh = OP::load_n(Kh, lC, 16 * ub, 32 * kb);
          const F fh = OP::load_n(Plh, lC, 16 * tb, 32 * kb);
          z = OP::mma(z, kh, fh);
          if constexpr (SPL) {
            z = OP::mma(z, OP::load_n(Kl, lC, 16 * ub, 32 * kb), fh);
            z = OP::mma(z, kh, OP::load_n(Pll, lC, 16 * tb, 32 * kb));
          }
        }
        // z[r] = Z[u = 16ub + 4q + r][t = 16tb + c]
        const int t = 16 * tb + c;
        float s = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int o = f_off(ub, tb, r);
          float fv = (float)Plh[o];
          if constexpr (SPL) fv += (float)Pll[o];
          s += fv * z[r];
        }
        s = sum_q(s);
        if (q == 0) dap[w][t] += s;
      }
    }
    __syncthreads();
    if (w == NW - 1) {
      // Per-token gate gradients.  Lane t < C.
      const int t = ln;
      const bool in = t < C;
      const int tc = in ? t : C - 1;
      float c3 = 0.f, c2 = 0.f, de = 0.f, da = 0.f, t1 = 0.f;
#pragma unroll
      for (int v = 0; v < NW; ++v) {
        if (v < JB) c3 += c3p[v][tc];
        if (v < IB) {
          c2 += c2p[v][tc];
          de += dep[v][tc];
        }
        da += dap[v][tc];
        if (v < JB) t1 += t1p[v];
      }
      c2 *= -et[tc];
      if (!in) c3 = c2 = 0.f;
      const float at = in ? al[tc] : 1.f;
      // z_t = alpha_{t-1} z_{t-1} + c2_{t-1}:  affine scan (A, B) upward.
      float A = dpp_move<kWaveShr1>(at, 0.f), B = dpp_move<kWaveShr1>(c2, 0.f);
      // w_t = alpha_{t+1} w_{t+1} + c3_{t+1}: affine scan downward.
      float A2 = dpp_move<kWaveShl1>(at, 0.f), B2 = dpp_move<kWaveShl1>(c3, 0.f);
      affine_scan<false>(A, B, ln);
      affine_scan<true>(A2, B2, ln);
      if (in) {
        const float pt = pre[tc], st = suf[tc];
        const float dal = (pt * st * t1 + pt * B2 + st * B + da) * gm[tc];
        const uint32_t o = (uint32_t)((t0 + t) * 4);
        if (a.dalpha) buf_store1(Oa, o, dal);
        if (a.deta) buf_store1(Oe, o, de * gm[tc]);
      }
    }
    if (w < JB) {
      // Lambda_n = tot Lambda_e + sum_u pre_u dY_u x_u^T.
#pragma unroll
      for (int ib = 0; ib < IB; ++ib) Lam[ib] *= tt;
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
#pragma unroll
        for (int ib = 0; ib < IB; ++ib) {
          const F ph = OP::load_t(Dph, lM, 32 * kb, 16 * ib);
          F pl = ph;
          if constexpr (SPL) pl = OP::load_t(Dpl, lM, 32 * kb, 16 * ib);
          Lam[ib] = mma_split_a<OP>(Lam[ib], ph, pl, xt[kb]);
        }
      }
    }
  }
}

// dW0[h] = sum_b sum_seg Bu[b, h, seg], fixed order.
__global__ void __launch_bounds__(256)
reduce_gated_dw0_kernel(const float* __restrict__ Bu, float* __restrict__ dW0, int64_t B, int64_t H,
                        int64_t nseg, int64_t md) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= H * md) return;
  const int64_t h = e / md, k = e % md;
  float s = 0.f;
  for (int64_t b = 0; b < B; ++b)
    for (int64_t j = 0; j < nseg; ++j) s += Bu[((b * H + h) * nseg + j) * md + k];
  dW0[e] = s;
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
int gated_fwd_chunk(int, int, int) { return 64; }
// The backward's LDS holds five C x C split tiles besides the chunk inputs and
// the published Lambda: 64-token tiles fit for bf16 64 x 64 maps only.
int gated_bwd_chunk(int bf16, int d, int m) { return (bf16 && d == 64 && m == 64) ? 64 : 32; }

static constexpr int lds_gated_bwd(int es, int lo, int d, int m, int C) {
  return es * (C * d + 3 * C * m + lo * C * m + (1 + lo) * 5 * C * C + (1 + lo) * d * m) +
         4 * (7 * C + 4 * (cmax(d, m) / 16) * C + 40);
}

int gated_wgs_per_cu(int fwd, int bf16, int d, int m) {
  const int waves = cmax(d, m) / 16;
  int n;
  if (fwd) {
    const int es = bf16 ? 2 : 4;
    n = 160 * 1024 / (es * 64 * (d + 2 * m + (bf16 ? m : 0)) + 1024);
  } else {
    n = 160 * 1024 / lds_gated_bwd(bf16 ? 2 : 4, bf16 ? 1 : 0, d, m, gated_bwd_chunk(bf16, d, m));
  }
  if (n * waves > 8) n = 8 / waves;
  return n < 1 ? 1 : n;
}

static GArgs gargs(const ScanProblem& p, const GatedPtrs& f) {
  GArgs k{};
  k.W0 = f.W0;
  k.X = f.X;
  k.G = f.G;
  k.dY = f.dY;
  k.eta = f.eta;
  k.eta_scalar = f.eta_scalar;
  k.eta_mul = f.eta_mul;
  k.alpha = f.alpha;
  k.alpha_scalar = f.alpha_scalar;
  k.reset = f.reset;
  k.BH = p.B * p.H;
  k.H = p.H;
  k.T = p.T;
  k.seg_len = p.seg_len;
  k.nseg = p.nseg;
  k.nchunks = (p.T + p.chunk - 1) / p.chunk;
  k.Y = f.Y;
  k.gtilde = f.gtilde;
  k.dX = f.dX;
  k.dG = f.dG;
  k.deta = f.deta;
  k.dalpha = f.dalpha;
  k.aggA = f.aggA;
  k.aggB = f.aggB;
  k.aggBu = f.aggBu;
  k.aggD = f.aggD;
  k.states = f.states;
  return k;
}

template <class OP, int D, int M, int C>
static hipError_t fwd_gated_dims_c(const ScanProblem& p, const GArgs& k, hipStream_t s) {
  constexpr int NT = cmax(D, M) / 16 * 64;
  const unsigned grid = (unsigned)seg_grid(k.BH, p.nseg);
  if (p.nseg > 1) {
    timing_begin(GRADLEV_K_GATED_AGG, s);
    hipLaunchKernelGGL((agg_gated_kernel<OP, D, M, C, kGAggFwd>), dim3(grid), dim3(NT), 0, s, k, p.nseg - 1);
    timing_end(GRADLEV_K_GATED_AGG, s);
  }
  timing_begin(GRADLEV_K_GATED_FWD, s);
  hipLaunchKernelGGL((fwd_gated_kernel<OP, D, M, C>), dim3(grid), dim3(NT), 0, s, k);
  timing_end(GRADLEV_K_GATED_FWD, s);
  return hipGetLastError();
}

// 64-token tiles; a forward that saves chunk-start states for a backward with
// 32-token tiles runs 32-token tiles itself.
template <class OP, int D, int M>
static hipError_t fwd_gated_dims(const ScanProblem& p, const GArgs& k, hipStream_t s) {
  if (p.chunk == 32) return fwd_gated_dims_c<OP, D, M, 32>(p, k, s);
  return fwd_gated_dims_c<OP, D, M, 64>(p, k, s);
}

template <class OP, int D, int M, int C>
static hipError_t bwd_gated_dims_c(const ScanProblem& p, const GArgs& k, float* dW0, bool saved,
                                   hipStream_t s) {
  constexpr int NT = cmax(D, M) / 16 * 64;
  const unsigned grid = (unsigned)seg_grid(k.BH, p.nseg);
  timing_begin(GRADLEV_K_GATED_AGG, s);
  if (saved)
    hipLaunchKernelGGL((agg_gated_kernel<OP, D, M, C, kGAggBwdSaved>), dim3(grid), dim3(NT), 0, s, k, p.nseg);
  else
    hipLaunchKernelGGL((agg_gated_kernel<OP, D, M, C, kGAggBwd>), dim3(grid), dim3(NT), 0, s, k, p.nseg);
  timing_end(GRADLEV_K_GATED_AGG, s);
  if (!saved) {  // the chunk-start states, unless the forward saved them
    timing_begin(GRADLEV_K_GATED_STATES, s);
    hipLaunchKernelGGL((states_gated_kernel<OP, D, M, C>), dim3(grid), dim3(NT), 0, s, k);
    timing_end(GRADLEV_K_GATED_STATES, s);
  }
  timing_begin(GRADLEV_K_GATED_BWD, s);
  // Separate waves for the row blocks of u where the wider workgroup keeps
  // its registers (measured on the 64 x 64 bf16 map).
  constexpr bool SPLITW = OP::kSplit == 2 && D == 64 && M == 64;
  constexpr int NTB = (SPLITW ? D / 16 + M / 16 : cmax(D, M) / 16) * 64;
  hipLaunchKernelGGL((bwd_gated_kernel<OP, D, M, C, SPLITW>), dim3(grid), dim3(NTB), 0, s, k);
  timing_end(GRADLEV_K_GATED_BWD, s);
  if (dW0) {
    const int64_t md = (int64_t)M * D;
    timing_begin(GRADLEV_K_BWD_DW0, s);
    hipLaunchKernelGGL(reduce_gated_dw0_kernel, dim3((unsigned)((p.H * md + 255) / 256)), dim3(256), 0, s,
                       (const float*)k.aggBu, dW0, p.B, p.H, p.nseg, md);
    timing_end(GRADLEV_K_BWD_DW0, s);
  }
  return hipGetLastError();
}

template <class OP, int D, int M>
static hipError_t bwd_gated_dims(const ScanProblem& p, const GArgs& k, float* dW0, bool saved, hipStream_t s) {
  if constexpr (OP::kSplit == 2 && D == 64 && M == 64) {
    if (p.chunk == 64) return bwd_gated_dims_c<OP, D, M, 64>(p, k, dW0, saved, s);
  }
  return bwd_gated_dims_c<OP, D, M, 32>(p, k, dW0, saved, s);
}

hipError_t launch_scan_fwd_gated(const ScanProblem& p, const GatedPtrs& f, hipStream_t s) {
  const GArgs k = gargs(p, f);
#define GL_DIMS(OPT)                                                            \
  if (p.d == 64 && p.m == 64) return fwd_gated_dims<OPT, 64, 64>(p, k, s);     \
  if (p.d == 64 && p.m == 128) return fwd_gated_dims<OPT, 64, 128>(p, k, s);   \
  if (p.d == 128 && p.m == 64) return fwd_gated_dims<OPT, 128, 64>(p, k, s);   \
  if (p.d == 128 && p.m == 128) return fwd_gated_dims<OPT, 128, 128>(p, k, s);
  if (p.bf16) {
    GL_DIMS(OpBF16)
  } else {
    GL_DIMS(OpF32)
  }
#undef GL_DIMS
  return hipErrorInvalidValue;
}

hipError_t launch_scan_bwd_gated(const ScanProblem& p, const GatedPtrs& f, hipStream_t s) {
  const GArgs k = gargs(p, f);
#define GL_DIMS(OPT)                                                                   \
  if (p.d == 64 && p.m == 64) return bwd_gated_dims<OPT, 64, 64>(p, k, f.dW0, f.saved_states, s);     \
  if (p.d == 64 && p.m == 128) return bwd_gated_dims<OPT, 64, 128>(p, k, f.dW0, f.saved_states, s);   \
  if (p.d == 128 && p.m == 64) return bwd_gated_dims<OPT, 128, 64>(p, k, f.dW0, f.saved_states, s);   \
  if (p.d == 128 && p.m == 128) return bwd_gated_dims<OPT, 128, 128>(p, k, f.dW0, f.saved_states, s);
  if (p.bf16) {
    GL_DIMS(OpBF16)
  } else {
    GL_DIMS(OpF32)
  }
#undef GL_DIMS
  return hipErrorInvalidValue;
}

}  // namespace gradlev
