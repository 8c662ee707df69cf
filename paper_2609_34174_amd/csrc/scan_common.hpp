// Pieces shared by the forward and backward scan launchers: kernel
// arguments, the segment-aggregate kernel and the cross-segment carry.
#pragma once

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
  int64_t H, T, seg_len, nseg;
  float* out0;   // fwd: Y
  float* aggA;
  float* aggB;
};

// ---------------------------------------------------------------------------
// Segment aggregates: A_k = sum_{t in seg k} eta_t g_t x_t^T   ([m][d], fp32)
// and, for the backward (BWD), B_k = sum_{t in seg k} dY_t x_t^T for k >= 1.
// Grid (segments to aggregate, B*H); wave w owns rows i in [16w, 16w+16).
// ---------------------------------------------------------------------------
template <class OP, int D, int M, int C, bool BWD>
__global__ void __launch_bounds__(cmax(D, M) / 16 * 64)
agg_kernel(const KArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int NW = cmax(D, M) / 16, NT = NW * 64;
  constexpr int JB = D / 16, IB = M / 16, LDC = C + 4;
  __shared__ E Xt[D * LDC];
  __shared__ E Gt[M * LDC];
  __shared__ E Dt[BWD ? M * LDC : 1];
  __shared__ float et[C];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, c = lane & 15, q = lane >> 4;
  const int64_t seg = blockIdx.x, bh = blockIdx.y;
  const int64_t T = a.T;
  const int64_t t_begin = seg * a.seg_len;
  const int64_t t_end = t_begin + a.seg_len < T ? t_begin + a.seg_len : T;
  const bool with_b = BWD && seg >= 1;
  const E* X = static_cast<const E*>(a.X) + bh * T * D;
  const E* G = static_cast<const E*>(a.G) + bh * T * M;
  const E* Dy = BWD ? static_cast<const E*>(a.dY) + bh * T * M : nullptr;

  f32x4 accA[JB], accB[JB];
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) accA[jb] = accB[jb] = zero4();

  TileRegs<OP, C, D, NT> xr;
  TileRegs<OP, C, M, NT> gr, dr;
  {
    const int rows = (int)(t_end - t_begin < C ? t_end - t_begin : C);
    xr.load(X + t_begin * D, rows, tid);
    gr.load(G + t_begin * M, rows, tid);
    if (with_b) dr.load(Dy + t_begin * M, rows, tid);
  }
  for (int64_t t0 = t_begin; t0 < t_end; t0 += C) {
    const int nvalid = (int)(t_end - t0 < C ? t_end - t0 : C);
    __syncthreads();
    xr.store_cols(Xt, LDC, tid);
    gr.store_cols(Gt, LDC, tid);
    if (with_b) dr.store_cols(Dt, LDC, tid);
    if (tid < C) et[tid] = tid < nvalid ? (a.eta ? a.eta[bh * T + t0 + tid] : a.eta_scalar) : 0.f;
    __syncthreads();
    if (t0 + C < t_end) {
      const int rows = (int)(t_end - t0 - C < C ? t_end - t0 - C : C);
      xr.load(X + (t0 + C) * D, rows, tid);
      gr.load(G + (t0 + C) * M, rows, tid);
      if (with_b) dr.load(Dy + (t0 + C) * M, rows, tid);
    }
    if (w < IB) {
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
        f32x8 gv = OP::load_f32(Gt, LDC, 16 * w, 32 * kb, lane);
#pragma unroll
        for (int e = 0; e < 8; ++e) gv[e] *= et[32 * kb + slot_k(e, q)];
        F vh, vl;
        OP::split(gv, vh, vl);
        F dv;
        if (with_b) dv = OP::load(Dt, LDC, 16 * w, 32 * kb, lane);
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) {
          const F xa = OP::load(Xt, LDC, 16 * jb, 32 * kb, lane);
          accA[jb] = mma_split_b<OP>(accA[jb], xa, vh, vl);
          if (with_b) accB[jb] = OP::mma(accB[jb], xa, dv);
        }
      }
    }
  }
  if (w < IB) {
    // accA[jb] holds A^T[j = 16jb + 4q + r][i = 16w + c].
    const int64_t off = (bh * a.nseg + seg) * M * D + (int64_t)(16 * w + c) * D;
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) {
      *reinterpret_cast<f32x4*>(a.aggA + off + 16 * jb + 4 * q) = accA[jb];
      if (with_b) *reinterpret_cast<f32x4*>(a.aggB + off + 16 * jb + 4 * q) = accB[jb];
    }
  }
}

// Carry across segments (defined in scan_fwd.hip).
//   mode 0 (forward):  A[k] <- sum_{j<k} A[j]        (A[nseg-1] is not read)
//   mode 1 (backward): A[k] <- sum_{j<=k} A[j];  B[k] <- sum_{j>k} B[j]
//                      (B[0] is not read)
//   mode 2 (backward, no suffix): A[k] <- sum_{j<=k} A[j]
hipError_t launch_carry(float* A, float* B, int64_t BH, int64_t nseg, int64_t md, int mode,
                        hipStream_t s);

}  // namespace gradlev
