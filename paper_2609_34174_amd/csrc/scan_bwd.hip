// Backward of the GradLev forward scan on gfx950.
//
// For L = sum_t <dY_t, y_t> (dY is the upstream costate of Section 3 step 3):
//   read side  (Eq. 4; Appendix C, Eq. 16 second line):
//       gtilde_t = (W_0 + Delta_t)^T dY_t
//   reverse-time terms, with suffix R_t = sum_{u>t} dY_u x_u^T:
//       u_t = -R_t x_t,  dG_t = eta_t u_t,  deta_t = <g_t, u_t>,
//       dX_t = gtilde_t - eta_t R_t^T g_t,  dW_0 = sum_b sum_t dY_t x_t^T.
// (u >= t and Delta_{t+1} for the inclusive convention.)
//
// Chunk form, chunk n of C tokens, W_n = W_0 + Delta_{nC}, R_n = suffix after
// the chunk, V = diag(eta) G, M the causal mask:
//   gtilde = dY W_n - (M o dY V^T) X
//   U      = -(X R_n^T + (M o X X^T)^T dY)             dG = diag(eta) U
//   dXw    = -(V R_n + (M o dY V^T)^T X)                dX = gtilde + dXw
//   W_n    = W_{n+1} + V^T X     (the state is un-written chunk by chunk)
//   R_{n-1}= R_n + dY^T X
// A workgroup walks its segment's chunks from last to first, carrying R
// forward in reverse time and un-writing W from the state at the segment's
// end (W_0 minus the inclusive prefix of segment aggregates).  Waves own
// column blocks of W and R (for the products contracted over m) and row
// blocks of a second copy of R (for the product contracted over d), so every
// state operand is read straight from accumulator registers.
#include "../../include/gradlev.h"
#include "scan_common.hpp"

namespace gradlev {

struct BArgs {
  const float* W0;
  const void* X;
  const void* G;
  const void* dY;
  const float* eta;
  float eta_scalar;
  int64_t H, T, seg_len, nseg;
  float* gtilde;
  float* dX;
  float* dG;
  float* deta;
  const float* pin;   // [BH][nseg][m][d] inclusive prefix of write aggregates
  const float* sfx;   // [BH][nseg][m][d] exclusive suffix of dY x^T aggregates, or null
  float* rfin;        // [BH][m][d] full-sequence dY x^T (written by segment 0), or null
};

template <class OP, int D, int M, int C, bool INCL>
__global__ void __launch_bounds__(cmax(D, M) / 16 * 64)
bwd_main_kernel(const BArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int NW = cmax(D, M) / 16, NT = NW * 64;
  constexpr int TB = C / 16, JB = D / 16, IB = M / 16;
  constexpr int LDD = D + 4, LDM = M + 4, LDC = C + 4;
  __shared__ E Xr[C * LDD];  // X[t][j]
  __shared__ E Gr[C * LDM];  // G[t][i]
  __shared__ E Dr[C * LDM];  // dY[t][i]
  __shared__ E Xt[D * LDC];  // X^T[j][t]
  __shared__ E Gt[M * LDC];  // G^T[i][t]
  __shared__ E Dt[M * LDC];  // dY^T[i][t]
  __shared__ E Er[C * LDC];  // -E[t][s], E = eta_s dY_t.g_s (s before t), [t][s]
  __shared__ E Et[C * LDC];  // +E stored [s][t]
  __shared__ float et[C];
  __shared__ float dpart[IB][C];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, c = lane & 15, q = lane >> 4;
  const int64_t seg = blockIdx.x, bh = blockIdx.y, h = bh % a.H;
  const int64_t T = a.T;
  const int64_t t_begin = seg * a.seg_len;
  const int64_t t_end = t_begin + a.seg_len < T ? t_begin + a.seg_len : T;
  const E* X = static_cast<const E*>(a.X) + bh * T * D;
  const E* G = static_cast<const E*>(a.G) + bh * T * M;
  const E* Dy = static_cast<const E*>(a.dY) + bh * T * M;
  const bool need_gx = a.gtilde || a.dX;
  const bool need_u = a.dG || a.deta;
  const bool need_dxw = a.dX != nullptr;
  const bool need_ri = need_u || a.rfin;

  for (int i = tid; i < C * LDC; i += NT) {
    Er[i] = (E)0.f;
    Et[i] = (E)0.f;
  }

  // Column-block state (wave w < JB): Wj[ib], Rj[ib] hold W/R[i = 16ib + 4q + r][j = 16w + c].
  // Row-block copy of R (wave w < IB): Ri[jb] holds R[i = 16w + c][j = 16jb + 4q + r].
  f32x4 Wj[IB], Rj[IB], Ri[JB];
  {
    const float* w0 = a.W0 + h * M * D;
    const float* pin = a.pin ? a.pin + (bh * a.nseg + seg) * M * D : nullptr;
    const float* sfx = a.sfx ? a.sfx + (bh * a.nseg + seg) * M * D : nullptr;
    if (w < JB) {
#pragma unroll
      for (int ib = 0; ib < IB; ++ib) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t o = (int64_t)(16 * ib + 4 * q + r) * D + 16 * w + c;
          Wj[ib][r] = pin ? w0[o] - pin[o] : 0.f;
          Rj[ib][r] = sfx ? sfx[o] : 0.f;
        }
      }
    }
    if (w < IB) {
#pragma unroll
      for (int jb = 0; jb < JB; ++jb)
        Ri[jb] = sfx ? *reinterpret_cast<const f32x4*>(sfx + (int64_t)(16 * w + c) * D + 16 * jb + 4 * q) : zero4();
    }
  }

  const int64_t nch = (t_end - t_begin + C - 1) / C;
  TileRegs<OP, C, D, NT> xr;
  TileRegs<OP, C, M, NT> gr, dr;
  {
    const int64_t t0 = t_begin + (nch - 1) * C;
    const int rows = (int)(t_end - t0);
    xr.load(X + t0 * D, rows, tid);
    gr.load(G + t0 * M, rows, tid);
    dr.load(Dy + t0 * M, rows, tid);
  }
  for (int64_t n = nch - 1; n >= 0; --n) {
    const int64_t t0 = t_begin + n * C;
    const int nvalid = (int)(t_end - t0 < C ? t_end - t0 : C);
    __syncthreads();
    xr.store_rows(Xr, LDD, tid);
    xr.store_cols(Xt, LDC, tid);
    gr.store_rows(Gr, LDM, tid);
    gr.store_cols(Gt, LDC, tid);
    dr.store_rows(Dr, LDM, tid);
    dr.store_cols(Dt, LDC, tid);
    if (tid < C) et[tid] = tid < nvalid ? (a.eta ? a.eta[bh * T + t0 + tid] : a.eta_scalar) : 0.f;
    __syncthreads();
    if (n > 0) {
      xr.load(X + (t0 - C) * D, C, tid);
      gr.load(G + (t0 - C) * M, C, tid);
      dr.load(Dy + (t0 - C) * M, C, tid);
    }

    // (1) Un-write this chunk: W_n = W_{n+1} + (eta G)^T X.
    if (w < JB && need_gx) {
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
        const F xq = OP::load(Xt, LDC, 16 * w, 32 * kb, lane);
#pragma unroll
        for (int ib = 0; ib < IB; ++ib) {
          f32x8 gv = OP::load_f32(Gt, LDC, 16 * ib, 32 * kb, lane);
#pragma unroll
          for (int e = 0; e < 8; ++e) gv[e] *= et[32 * kb + slot_k(e, q)];
          F vh, vl;
          OP::split(gv, vh, vl);
          Wj[ib] = mma_split_a<OP>(Wj[ib], vh, vl, xq);
        }
      }
    }

    // (2) Intra-chunk tiles E[t][s] = eta_s dY_t . g_s (t after s), shared
    //     through LDS in both orientations.
    if (need_gx) {
      for (int idx = w; idx < TB * (TB + 1) / 2; idx += NW) {
        const int tb = tri_row(idx), sb = idx - tb * (tb + 1) / 2;
        // acc[r] holds entry (t = 16tb + 4q + r, s = 16sb + c).
        const int s = 16 * sb + c;
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < M / 32; ++kb)
          acc = OP::mma(acc, OP::load(Dr, LDM, 16 * tb, 32 * kb, lane), OP::load(Gr, LDM, 16 * sb, 32 * kb, lane));
        const float es = et[s];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * tb + 4 * q + r;
          const bool keep = INCL ? (t >= s) : (t > s);
          acc[r] = keep ? acc[r] * es : 0.f;
          OP::store1(Er + t * LDC + s, -acc[r]);
        }
        OP::store4(Et + s * LDC + 16 * tb + 4 * q, acc);
      }
    }
    __syncthreads();

    // (3) gtilde and dX for columns j in [16w, 16w+16).
    if (w < JB && need_gx) {
      F Wh[M / 32], Wl[M / 32], Rh[M / 32], Rl[M / 32];
#pragma unroll
      for (int kb = 0; kb < M / 32; ++kb) {
        OP::split(cat(Wj[2 * kb], Wj[2 * kb + 1]), Wh[kb], Wl[kb]);
        if (need_dxw) OP::split(cat(Rj[2 * kb], Rj[2 * kb + 1]), Rh[kb], Rl[kb]);
      }
      for (int tb = 0; tb < TB; ++tb) {
        // gtilde^T[j][t] = sum_i W[i][j] dY[t][i] - sum_s X[s][j] E[t][s]
        f32x4 ga = zero4();
#pragma unroll
        for (int kb = 0; kb < M / 32; ++kb)
          ga = mma_split_a<OP>(ga, Wh[kb], Wl[kb], OP::load(Dr, LDM, 16 * tb, 32 * kb, lane));
        for (int kb = 0; kb <= tb / 2; ++kb)
          ga = OP::mma(ga, OP::load(Xt, LDC, 16 * w, 32 * kb, lane), OP::load(Er, LDC, 16 * tb, 32 * kb, lane));
        // Lane holds row t = 16tb + c, columns j = 16w + 4q + r.
        const int t = 16 * tb + c;
        f32x4 dx = ga;
        if (need_dxw) {
          // dXw^T[j][s] = -(eta_s sum_i R[i][j] G[s][i] + sum_t X[t][j] E[t][s]), s = t here.
          f32x4 xa = zero4();
#pragma unroll
          for (int kb = 0; kb < M / 32; ++kb)
            xa = mma_split_a<OP>(xa, Rh[kb], Rl[kb], OP::load(Gr, LDM, 16 * tb, 32 * kb, lane));
          xa *= et[t];
          for (int kb = tb / 2; kb < C / 32; ++kb)
            xa = OP::mma(xa, OP::load(Xt, LDC, 16 * w, 32 * kb, lane), OP::load(Et, LDC, 16 * tb, 32 * kb, lane));
          dx = ga - xa;
        }
        if (t < nvalid) {
          const int64_t o = (t0 + t) * D + 16 * w + 4 * q;
          if (a.gtilde) *reinterpret_cast<f32x4*>(a.gtilde + bh * T * D + o) = ga;
          if (a.dX) *reinterpret_cast<f32x4*>(a.dX + bh * T * D + o) = dx;
        }
      }
    }

    // (4) U, dG and deta for rows i in [16w, 16w+16).
    if (w < IB && need_u) {
      F Rh[D / 32], Rl[D / 32];
#pragma unroll
      for (int kb = 0; kb < D / 32; ++kb) OP::split(cat(Ri[2 * kb], Ri[2 * kb + 1]), Rh[kb], Rl[kb]);
      for (int sb = 0; sb < TB; ++sb) {
        // -U^T[i][s] = sum_j R[i][j] X[s][j] + sum_t dY[t][i] S[t][s]
        f32x4 ua = zero4();
#pragma unroll
        for (int kb = 0; kb < D / 32; ++kb)
          ua = mma_split_a<OP>(ua, Rh[kb], Rl[kb], OP::load(Xr, LDD, 16 * sb, 32 * kb, lane));
        // Intra-chunk term with S[t][s] = x_t . x_s computed here, per pair of
        // t blocks, and kept in fp32 registers (split for the matrix core):
        // the tile (rows t, cols s) is directly the operand contracted over t.
        for (int kb = sb / 2; kb < C / 32; ++kb) {
          f32x8 sv;
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int tb = 2 * kb + hh;
            f32x4 st = zero4();
            if (tb >= sb) {
#pragma unroll
              for (int kj = 0; kj < D / 32; ++kj)
                st = OP::mma(st, OP::load(Xr, LDD, 16 * tb, 32 * kj, lane), OP::load(Xr, LDD, 16 * sb, 32 * kj, lane));
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const int t = 16 * tb + 4 * q + r, s = 16 * sb + c;
                if (!(INCL ? (t >= s) : (t > s))) st[r] = 0.f;
              }
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) sv[4 * hh + r] = st[r];
          }
          F sh, sl;
          OP::split(sv, sh, sl);
          ua = mma_split_b<OP>(ua, OP::load(Dt, LDC, 16 * w, 32 * kb, lane), sh, sl);
        }
        // Lane holds token s = 16sb + c, rows i = 16w + 4q + r; U = -ua.
        const int s = 16 * sb + c;
        const float es = et[s];
        if (a.dG && s < nvalid)
          *reinterpret_cast<f32x4*>(a.dG + (bh * T + t0 + s) * M + 16 * w + 4 * q) = -es * ua;
        if (a.deta) {
          const E* gp = Gr + s * LDM + 16 * w + 4 * q;
          float p = 0.f;
#pragma unroll
          for (int r = 0; r < 4; ++r) p -= (float)gp[r] * ua[r];
          p += __shfl_xor(p, 16);
          p += __shfl_xor(p, 32);
          if (q == 0) dpart[w][s] = p;
        }
      }
    }

    // (5) Suffix update: R_{n-1} = R_n + dY^T X (exact products).
    if (w < JB && need_dxw) {
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
        const F xq = OP::load(Xt, LDC, 16 * w, 32 * kb, lane);
#pragma unroll
        for (int ib = 0; ib < IB; ++ib) Rj[ib] = OP::mma(Rj[ib], OP::load(Dt, LDC, 16 * ib, 32 * kb, lane), xq);
      }
    }
    if (w < IB && need_ri) {
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
        const F dq = OP::load(Dt, LDC, 16 * w, 32 * kb, lane);
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) Ri[jb] = OP::mma(Ri[jb], OP::load(Xt, LDC, 16 * jb, 32 * kb, lane), dq);
      }
    }
    if (a.deta) {
      __syncthreads();
      if (tid < nvalid) {
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < IB; ++i) s += dpart[i][tid];
        a.deta[bh * T + t0 + tid] = s;
      }
    }
  }

  // Segment 0 ends holding sum over the whole sequence of dY x^T.
  if (a.rfin && seg == 0 && w < IB) {
    float* o = a.rfin + bh * M * D + (int64_t)(16 * w + c) * D;
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) *reinterpret_cast<f32x4*>(o + 16 * jb + 4 * q) = Ri[jb];
  }
}

// dW0[h] = sum_b rfin[b, h] in a fixed order.
static __global__ void __launch_bounds__(256)
reduce_dw0_kernel(const float* rfin, float* dW0, int64_t B, int64_t H, int64_t md4) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= H * md4) return;
  const int64_t h = gid / md4, e = gid % md4;
  f32x4 s = zero4();
  for (int64_t b = 0; b < B; ++b) s += reinterpret_cast<const f32x4*>(rfin)[(b * H + h) * md4 + e];
  reinterpret_cast<f32x4*>(dW0)[h * md4 + e] = s;
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
static int lds_bytes_bwd(int bf16, int d, int m, int C) {
  const int es = bf16 ? 2 : 4;
  return es * (C * (d + 4) + 2 * C * (m + 4) + d * (C + 4) + 2 * m * (C + 4) + 2 * C * (C + 4)) +
         4 * C + 4 * (m / 16) * C;
}

int bwd_chunk_for(int bf16, int d, int m, int requested) {
  (void)requested;
  int C = 64;
  if (lds_bytes_bwd(bf16, d, m, C) > 160 * 1024) C = 32;
  return C;
}

int bwd_wgs_per_cu(int bf16, int d, int m, int C) {
  int n = 160 * 1024 / lds_bytes_bwd(bf16, d, m, C);
  const int waves = cmax(d, m) / 16;
  if (n * waves > 32) n = 32 / waves;
  return n < 1 ? 1 : n;
}

template <class OP, int D, int M, int C>
static hipError_t bwd_dispatch(const ScanProblem& p, const BwdPtrs& f, hipStream_t s) {
  constexpr int NT = cmax(D, M) / 16 * 64;
  const int64_t BH = p.B * p.H;
  const bool need_gx = f.gtilde || f.dX;
  const bool need_sfx = p.nseg > 1 && (f.dX || f.dG || f.deta || f.dW0);

  KArgs k{};
  k.W0 = f.W0;
  k.X = f.X;
  k.G = f.G;
  k.dY = f.dY;
  k.eta = f.eta;
  k.eta_scalar = f.eta_scalar;
  k.H = p.H;
  k.T = p.T;
  k.seg_len = p.seg_len;
  k.nseg = p.nseg;
  k.aggA = f.aggA;
  k.aggB = f.aggB;
  // Segment aggregates: writes (for the un-write start state) and, when a
  // suffix is needed, dY x^T.  The write aggregate is skipped when only the
  // reverse-time outputs are requested; W is then never read.
  if (need_gx || need_sfx) {
    timing_begin(GRADLEV_K_BWD_AGG, s);
    if (need_sfx)
      hipLaunchKernelGGL((agg_kernel<OP, D, M, C, true>), dim3((unsigned)p.nseg, (unsigned)BH), dim3(NT), 0, s, k);
    else
      hipLaunchKernelGGL((agg_kernel<OP, D, M, C, false>), dim3((unsigned)p.nseg, (unsigned)BH), dim3(NT), 0, s, k);
    timing_end(GRADLEV_K_BWD_AGG, s);
    if (p.nseg > 1) {
      timing_begin(GRADLEV_K_BWD_CARRY, s);
      (void)launch_carry(f.aggA, need_sfx ? f.aggB : nullptr, BH, p.nseg, (int64_t)D * M, need_sfx ? 1 : 2, s);
      timing_end(GRADLEV_K_BWD_CARRY, s);
    }
  }
  BArgs b{};
  b.W0 = f.W0;
  b.X = f.X;
  b.G = f.G;
  b.dY = f.dY;
  b.eta = f.eta;
  b.eta_scalar = f.eta_scalar;
  b.H = p.H;
  b.T = p.T;
  b.seg_len = p.seg_len;
  b.nseg = p.nseg;
  b.gtilde = f.gtilde;
  b.dX = f.dX;
  b.dG = f.dG;
  b.deta = f.deta;
  b.pin = need_gx ? f.aggA : nullptr;
  b.sfx = need_sfx ? f.aggB : nullptr;
  b.rfin = f.dW0 ? f.rfin : nullptr;
  timing_begin(GRADLEV_K_BWD_MAIN, s);
  if (p.inclusive)
    hipLaunchKernelGGL((bwd_main_kernel<OP, D, M, C, true>), dim3((unsigned)p.nseg, (unsigned)BH), dim3(NT), 0, s, b);
  else
    hipLaunchKernelGGL((bwd_main_kernel<OP, D, M, C, false>), dim3((unsigned)p.nseg, (unsigned)BH), dim3(NT), 0, s, b);
  timing_end(GRADLEV_K_BWD_MAIN, s);
  if (f.dW0) {
    const int64_t md4 = (int64_t)D * M / 4, n = p.H * md4;
    timing_begin(GRADLEV_K_BWD_DW0, s);
    hipLaunchKernelGGL(reduce_dw0_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, f.rfin, f.dW0, p.B, p.H, md4);
    timing_end(GRADLEV_K_BWD_DW0, s);
  }
  return hipGetLastError();
}

template <class OP, int C>
static hipError_t bwd_by_dims(const ScanProblem& p, const BwdPtrs& f, hipStream_t s) {
  if (p.d == 64 && p.m == 64) return bwd_dispatch<OP, 64, 64, C>(p, f, s);
  if (p.d == 64 && p.m == 128) return bwd_dispatch<OP, 64, 128, C>(p, f, s);
  if (p.d == 128 && p.m == 64) return bwd_dispatch<OP, 128, 64, C>(p, f, s);
  if (p.d == 128 && p.m == 128) return bwd_dispatch<OP, 128, 128, C>(p, f, s);
  return hipErrorInvalidValue;
}

hipError_t launch_scan_bwd(const ScanProblem& p, const BwdPtrs& f, hipStream_t s) {
  if (p.bf16) return bwd_by_dims<OpBF16, 64>(p, f, s);
  // fp32 tiles double the LDS footprint: chunk 64 fits only the 64 x 64 map.
  if (p.d == 64 && p.m == 64 && p.chunk == 64) return bwd_dispatch<OpF32, 64, 64, 64>(p, f, s);
  if (p.chunk == 32) return bwd_by_dims<OpF32, 32>(p, f, s);
  return hipErrorInvalidValue;
}

}  // namespace gradlev
