// Deployment step of GradLev on gfx950 (Section 3, "Training objective", last
// sentences; Appendix A, last sentence): every (sequence, head) scores with
// its current fast weights and then writes its true costate,
//
//   y = W x   (before the write),      W <- W - eta g x^T,
//
// or, gated (Section 3, Eq. 2 general form), W <- W0 + alpha (W - W0) - eta g x^T
// with W first replaced by W0 when the step starts a new document.
//
// The step is a pure stream over the fp32 state (0.5 flop per byte), so the
// kernel is shaped for HBM: one workgroup per state matrix, each thread
// owning one 16-byte column group of D/4 lanes' rows, consecutive lanes on
// consecutive 16-byte words (fully coalesced loads and stores), four row
// passes' loads in flight at once, the row dot products reduced across the
// D/4 lanes that share a row, and the update written back from the same
// registers (each byte read once, written once).
#include "../../include/gradlev.h"
#include "device_common.hpp"
#include "internal.hpp"

namespace gradlev {

template <int D, bool GATED>
__global__ void __launch_bounds__(256)
decode_kernel(float* __restrict__ W, const float* __restrict__ x, const float* __restrict__ g,
              const float* __restrict__ eta, float eta_scalar, float* __restrict__ y, int M,
              const float* __restrict__ W0, int64_t H, const float* __restrict__ alpha,
              float alpha_scalar, const uint8_t* __restrict__ reset) {
  constexpr int LPR = D / 4;          // lanes per row (each holds 4 columns)
  constexpr int RPI = 256 / LPR;      // rows per pass of the workgroup
  constexpr int U = 4;                // passes whose loads are in flight together
  const int64_t sh = blockIdx.x;
  const int tid = threadIdx.x;
  const int col = 4 * (tid % LPR), row0 = tid / LPR;
  // The state of one (sequence, head) as a buffer: rows past M read zero and
  // their stores are dropped, so the passes need no branches.
  const rsrc_t Ws = make_rsrc(W + sh * (int64_t)M * D, (uint32_t)(M * D * 4));
  const rsrc_t Gs = make_rsrc(g + sh * (int64_t)M, (uint32_t)(M * 4));
  const rsrc_t Ys = make_rsrc(y + sh * (int64_t)M, (uint32_t)(M * 4));
  // Gated: the slow weights of this head (shared by all sequences, so they
  // are served from cache), the retention, and the document-start flag.
  const rsrc_t W0s = make_rsrc(GATED ? W0 + (sh % H) * (int64_t)M * D : nullptr, GATED ? (uint32_t)(M * D * 4) : 0u);
  const float al = GATED ? (alpha ? alpha[sh] : alpha_scalar) : 1.f;
  const bool fresh = GATED && reset && reset[sh / H] != 0;
  const f32x4 xv = *reinterpret_cast<const f32x4*>(x + sh * D + col);
  const float e = eta ? eta[sh] : eta_scalar;
  for (int i0 = row0; i0 < M; i0 += U * RPI) {
    f32x4 wv[U], w0[U];
    float gv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * RPI;
      wv[u] = buf_load4(Ws, (uint32_t)((i * D + col) * 4), (const float*)nullptr);
      if constexpr (GATED) w0[u] = buf_load4(W0s, (uint32_t)((i * D + col) * 4), (const float*)nullptr);
      gv[u] = buf_load1(Gs, (uint32_t)(i * 4));
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * RPI;
      if constexpr (GATED) {
        if (fresh) wv[u] = w0[u];
      }
      float s = wv[u][0] * xv[0] + wv[u][1] * xv[1] + wv[u][2] * xv[2] + wv[u][3] * xv[3];
#pragma unroll
      for (int o = LPR / 2; o >= 1; o >>= 1) s += __shfl_xor(s, o, LPR);
      buf_store1<kStoreDefault>(Ys, tid % LPR == 0 ? (uint32_t)(i * 4) : kOOB, s);
      f32x4 nw;
      if constexpr (GATED) nw = w0[u] + al * (wv[u] - w0[u]) - (e * gv[u]) * xv;
      else nw = wv[u] - (e * gv[u]) * xv;
      buf_store4<kStoreDefault>(Ws, (uint32_t)((i * D + col) * 4), nw);
    }
  }
}

hipError_t launch_decode(int64_t S, int64_t H, int d, int m, float* W, const float* x,
                         const float* g, const float* eta, float eta_scalar, float* y,
                         hipStream_t s, const DecodeGates* gt) {
  const dim3 grid((unsigned)(S * H)), block(256);
  const float* W0 = gt ? gt->W0 : nullptr;
  const float* al = gt ? gt->alpha : nullptr;
  const float as = gt ? gt->alpha_scalar : 1.f;
  const uint8_t* rs = gt ? gt->reset : nullptr;
#define GL_DECODE(DD)                                                                                   \
  if (gt)                                                                                               \
    hipLaunchKernelGGL((decode_kernel<DD, true>), grid, block, 0, s, W, x, g, eta, eta_scalar, y, m, W0, H, al, as, rs); \
  else                                                                                                  \
    hipLaunchKernelGGL((decode_kernel<DD, false>), grid, block, 0, s, W, x, g, eta, eta_scalar, y, m, W0, H, al, as, rs);
  timing_begin(GRADLEV_K_DECODE, s);
  switch (d) {
    case 16: GL_DECODE(16) break;
    case 32: GL_DECODE(32) break;
    case 64: GL_DECODE(64) break;
    case 128: GL_DECODE(128) break;
    case 256: GL_DECODE(256) break;
    default: timing_end(GRADLEV_K_DECODE, s); return hipErrorInvalidValue;
  }
#undef GL_DECODE
  timing_end(GRADLEV_K_DECODE, s);
  return hipGetLastError();
}

}  // namespace gradlev
