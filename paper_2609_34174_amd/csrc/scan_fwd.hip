// Forward scan of GradLev's adapted map on gfx950 (Section 3 step 2, Eq. 3;
// Appendix C, Eq. 16 first line, with unit retention):
//
//   y_t = (W_0 + Delta_t) x_t,  Delta_t = - sum_{s<t} eta_s g_s x_s^T  (s<=t inclusive)
//
// Work decomposition for one sequence (b, h):
//   * the T tokens are cut into segments of `seg_len` tokens, one workgroup
//     each, so that short batches still fill 256 CUs;
//   * a segment walks its chunks of C tokens in order, keeping the fp32 state
//     W_n = W_0 + Delta_{nC} in the accumulator registers of its waves;
//   * per chunk, on the matrix cores:
//       S   = X X^T                        (C x C, causal mask, scaled by -eta)
//       Y   = X W_n^T + S G                (state read + intra-chunk reads)
//       W  <- W_n - (eta G)^T X            (carry to the next chunk)
//   * segments are joined by their aggregated writes A_k = sum eta g x^T,
//     computed by agg_kernel and turned into exclusive prefixes by
//     carry_kernel, so each segment starts from W_0 - sum_{j<k} A_j.
#include "../../include/gradlev.h"
#include "scan_common.hpp"

namespace gradlev {

// ---------------------------------------------------------------------------
// Carry across segments, per sequence and element (fixed summation order).
//   mode 0 (forward):  A[k] <- sum_{j<k} A[j]        (A[nseg-1] is not read)
//   mode 1 (backward): A[k] <- sum_{j<=k} A[j];  B[k] <- sum_{j>k} B[j]
//                      (B[0] is not read)
//   mode 2 (backward, no suffix): A[k] <- sum_{j<=k} A[j]
// ---------------------------------------------------------------------------
static __global__ void __launch_bounds__(256)
carry_kernel(float* A, float* B, int64_t BH, int64_t nseg, int64_t md4, int mode) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= BH * md4) return;
  const int64_t bh = gid / md4, e = gid % md4;
  f32x4* pa = reinterpret_cast<f32x4*>(A) + bh * nseg * md4 + e;
  f32x4 run = zero4();
  if (mode == 0) {
    for (int64_t k = 0; k < nseg; ++k) {
      const f32x4 v = k + 1 < nseg ? pa[k * md4] : zero4();
      pa[k * md4] = run;
      run += v;
    }
    return;
  }
  for (int64_t k = 0; k < nseg; ++k) {
    run += pa[k * md4];
    pa[k * md4] = run;
  }
  if (mode != 1) return;
  f32x4* pb = reinterpret_cast<f32x4*>(B) + bh * nseg * md4 + e;
  run = zero4();
  for (int64_t k = nseg - 1; k >= 1; --k) {
    const f32x4 v = pb[k * md4];
    pb[k * md4] = run;
    run += v;
  }
  pb[0] = run;
}

hipError_t launch_carry(float* A, float* B, int64_t BH, int64_t nseg, int64_t md, int mode,
                        hipStream_t s) {
  const int64_t md4 = md / 4, n = BH * md4;
  hipLaunchKernelGGL(carry_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, A, B, BH, nseg, md4, mode);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Main forward kernel.  Grid (nseg, B*H); NW = max(d, m)/16 waves.
// Wave w < m/16 owns output rows i in [16w, 16w+16): it holds that slice of
// the state as accumulator tiles of W^T (rows j, cols i) and produces the
// matching columns of Y for every token of the chunk.
// ---------------------------------------------------------------------------
template <class OP, int D, int M, int C, bool INCL>
__global__ void __launch_bounds__(cmax(D, M) / 16 * 64)
fwd_main_kernel(const KArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int NW = cmax(D, M) / 16, NT = NW * 64;
  constexpr int TB = C / 16, JB = D / 16, IB = M / 16;
  constexpr int LDR = D + 4, LDC = C + 4;
  __shared__ E Xr[C * LDR];   // X[t][j]
  __shared__ E Xt[D * LDC];   // X^T[j][t]
  __shared__ E Gt[M * LDC];   // G^T[i][t]
  __shared__ E Pl[C * LDC];   // -eta_s (x_t . x_s) masked, [t][s]
  __shared__ float et[C];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, c = lane & 15, q = lane >> 4;
  const int64_t seg = blockIdx.x, bh = blockIdx.y, h = bh % a.H;
  const int64_t T = a.T;
  const int64_t t_begin = seg * a.seg_len;
  const int64_t t_end = t_begin + a.seg_len < T ? t_begin + a.seg_len : T;
  const E* X = static_cast<const E*>(a.X) + bh * T * D;
  const E* G = static_cast<const E*>(a.G) + bh * T * M;
  float* Y = a.out0 + bh * T * M;

  for (int i = tid; i < C * LDC; i += NT) Pl[i] = (E)0.f;

  // State tiles: Ws[jb] holds W[i = 16w + c][j = 16jb + 4q + r].
  f32x4 Ws[JB];
  if (w < IB) {
    const float* w0 = a.W0 + h * M * D + (int64_t)(16 * w + c) * D;
    const float* pf = a.aggA ? a.aggA + (bh * a.nseg + seg) * M * D + (int64_t)(16 * w + c) * D : nullptr;
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) {
      f32x4 v = *reinterpret_cast<const f32x4*>(w0 + 16 * jb + 4 * q);
      if (pf) v -= *reinterpret_cast<const f32x4*>(pf + 16 * jb + 4 * q);
      Ws[jb] = v;
    }
  }

  TileRegs<OP, C, D, NT> xr;
  TileRegs<OP, C, M, NT> gr;
  {
    const int rows = (int)(t_end - t_begin < C ? t_end - t_begin : C);
    xr.load(X + t_begin * D, rows, tid);
    gr.load(G + t_begin * M, rows, tid);
  }
  for (int64_t t0 = t_begin; t0 < t_end; t0 += C) {
    const int nvalid = (int)(t_end - t0 < C ? t_end - t0 : C);
    __syncthreads();
    xr.store_rows(Xr, LDR, tid);
    xr.store_cols(Xt, LDC, tid);
    gr.store_cols(Gt, LDC, tid);
    if (tid < C) et[tid] = tid < nvalid ? (a.eta ? a.eta[bh * T + t0 + tid] : a.eta_scalar) : 0.f;
    __syncthreads();
    if (t0 + C < t_end) {
      const int rows = (int)(t_end - t0 - C < C ? t_end - t0 - C : C);
      xr.load(X + (t0 + C) * D, rows, tid);
      gr.load(G + (t0 + C) * M, rows, tid);
    }

    // Intra-chunk scores, lower-triangular tiles (tb >= sb) shared by all waves.
    for (int idx = w; idx < TB * (TB + 1) / 2; idx += NW) {
      const int tb = tri_row(idx), sb = idx - tb * (tb + 1) / 2;
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < D / 32; ++kb)
        acc = OP::mma(acc, OP::load(Xr, LDR, 16 * sb, 32 * kb, lane), OP::load(Xr, LDR, 16 * tb, 32 * kb, lane));
      // acc[r] = x_s . x_t with s = 16sb + 4q + r, t = 16tb + c.
      const int t = 16 * tb + c;
      f32x4 v;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int s = 16 * sb + 4 * q + r;
        const bool keep = INCL ? (s <= t) : (s < t);
        v[r] = keep ? -acc[r] * et[s] : 0.f;
      }
      OP::store4(Pl + t * LDC + 16 * sb + 4 * q, v);
    }
    __syncthreads();

    if (w < IB) {
      F Wh[D / 32], Wl[D / 32];
#pragma unroll
      for (int kb = 0; kb < D / 32; ++kb) OP::split(cat(Ws[2 * kb], Ws[2 * kb + 1]), Wh[kb], Wl[kb]);
      for (int tb = 0; tb < TB; ++tb) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < D / 32; ++kb)
          acc = mma_split_a<OP>(acc, Wh[kb], Wl[kb], OP::load(Xr, LDR, 16 * tb, 32 * kb, lane));
        for (int kb = 0; kb <= tb / 2; ++kb)
          acc = OP::mma(acc, OP::load(Gt, LDC, 16 * w, 32 * kb, lane), OP::load(Pl, LDC, 16 * tb, 32 * kb, lane));
        // acc[r] = y_t[i] with i = 16w + 4q + r, t = 16tb + c.
        const int t = 16 * tb + c;
        if (t < nvalid) *reinterpret_cast<f32x4*>(Y + (t0 + t) * M + 16 * w + 4 * q) = acc;
      }
      if (t0 + C < t_end) {
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
          f32x8 gv = OP::load_f32(Gt, LDC, 16 * w, 32 * kb, lane);
#pragma unroll
          for (int e = 0; e < 8; ++e) gv[e] *= -et[32 * kb + slot_k(e, q)];
          F vh, vl;
          OP::split(gv, vh, vl);
#pragma unroll
          for (int jb = 0; jb < JB; ++jb)
            Ws[jb] = mma_split_b<OP>(Ws[jb], OP::load(Xt, LDC, 16 * jb, 32 * kb, lane), vh, vl);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
static int lds_bytes_fwd(int bf16, int d, int m, int C) {
  const int es = bf16 ? 2 : 4;
  return es * (C * (d + 4) + d * (C + 4) + m * (C + 4) + C * (C + 4)) + 4 * C;
}

int fwd_chunk_for(int bf16, int d, int m, int requested) {
  int C = (bf16 && requested == 128) ? 128 : 64;
  if (C == 128 && lds_bytes_fwd(bf16, d, m, 128) > 160 * 1024) C = 64;
  return C;
}

int fwd_wgs_per_cu(int bf16, int d, int m, int C) {
  int n = 160 * 1024 / lds_bytes_fwd(bf16, d, m, C);
  const int waves = cmax(d, m) / 16;
  if (n * waves > 32) n = 32 / waves;
  return n < 1 ? 1 : n;
}

template <class OP, int D, int M, int C>
static hipError_t fwd_dispatch(const ScanProblem& p, const KArgs& k, hipStream_t s) {
  constexpr int NT = cmax(D, M) / 16 * 64;
  const int64_t BH = p.B * p.H;
  if (p.nseg > 1) {
    timing_begin(GRADLEV_K_FWD_AGG, s);
    hipLaunchKernelGGL((agg_kernel<OP, D, M, C, false>), dim3((unsigned)(p.nseg - 1), (unsigned)BH), dim3(NT), 0, s, k);
    timing_end(GRADLEV_K_FWD_AGG, s);
    timing_begin(GRADLEV_K_FWD_CARRY, s);
    (void)launch_carry(k.aggA, nullptr, BH, p.nseg, (int64_t)D * M, 0, s);
    timing_end(GRADLEV_K_FWD_CARRY, s);
  }
  timing_begin(GRADLEV_K_FWD_MAIN, s);
  if (p.inclusive)
    hipLaunchKernelGGL((fwd_main_kernel<OP, D, M, C, true>), dim3((unsigned)p.nseg, (unsigned)BH), dim3(NT), 0, s, k);
  else
    hipLaunchKernelGGL((fwd_main_kernel<OP, D, M, C, false>), dim3((unsigned)p.nseg, (unsigned)BH), dim3(NT), 0, s, k);
  timing_end(GRADLEV_K_FWD_MAIN, s);
  return hipGetLastError();
}

template <class OP, int C>
static hipError_t fwd_by_dims(const ScanProblem& p, const KArgs& k, hipStream_t s) {
  if (p.d == 64 && p.m == 64) return fwd_dispatch<OP, 64, 64, C>(p, k, s);
  if (p.d == 64 && p.m == 128) return fwd_dispatch<OP, 64, 128, C>(p, k, s);
  if (p.d == 128 && p.m == 64) return fwd_dispatch<OP, 128, 64, C>(p, k, s);
  if (p.d == 128 && p.m == 128) return fwd_dispatch<OP, 128, 128, C>(p, k, s);
  return hipErrorInvalidValue;
}

hipError_t launch_scan_fwd(const ScanProblem& p, const FwdPtrs& f, hipStream_t s) {
  KArgs k{};
  k.W0 = f.W0;
  k.X = f.X;
  k.G = f.G;
  k.dY = nullptr;
  k.eta = f.eta;
  k.eta_scalar = f.eta_scalar;
  k.H = p.H;
  k.T = p.T;
  k.seg_len = p.seg_len;
  k.nseg = p.nseg;
  k.out0 = f.Y;
  k.aggA = p.nseg > 1 ? f.agg : nullptr;
  k.aggB = nullptr;
  if (p.bf16) {
    if (p.chunk == 128) return fwd_by_dims<OpBF16, 128>(p, k, s);
    return fwd_by_dims<OpBF16, 64>(p, k, s);
  }
  return fwd_by_dims<OpF32, 64>(p, k, s);
}

}  // namespace gradlev
