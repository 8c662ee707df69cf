// Deployment step of GradLev on gfx950 (Section 3, "Training objective", last
// sentences; Appendix A, last sentence): every (sequence, head) scores with
// its current fast weights and then writes its true costate,
//
//   y = W x   (before the write),      W <- W - eta g x^T.
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

template <int D>
__global__ void __launch_bounds__(256)
decode_kernel(float* __restrict__ W, const float* __restrict__ x, const float* __restrict__ g,
              const float* __restrict__ eta, float eta_scalar, float* __restrict__ y, int M) {
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
  const f32x4 xv = *reinterpret_cast<const f32x4*>(x + sh * D + col);
  const float e = eta ? eta[sh] : eta_scalar;
  for (int i0 = row0; i0 < M; i0 += U * RPI) {
    f32x4 wv[U];
    float gv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * RPI;
      wv[u] = buf_load4(Ws, (uint32_t)((i * D + col) * 4), (const float*)nullptr);
      gv[u] = buf_load1(Gs, (uint32_t)(i * 4));
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * RPI;
      float s = wv[u][0] * xv[0] + wv[u][1] * xv[1] + wv[u][2] * xv[2] + wv[u][3] * xv[3];
#pragma unroll
      for (int o = LPR / 2; o >= 1; o >>= 1) s += __shfl_xor(s, o, LPR);
      buf_store1<kStoreDefault>(Ys, tid % LPR == 0 ? (uint32_t)(i * 4) : kOOB, s);
      buf_store4<kStoreDefault>(Ws, (uint32_t)((i * D + col) * 4), wv[u] - (e * gv[u]) * xv);
    }
  }
}

hipError_t launch_decode(int64_t S, int64_t H, int d, int m, float* W, const float* x,
                         const float* g, const float* eta, float eta_scalar, float* y,
                         hipStream_t s) {
  const dim3 grid((unsigned)(S * H)), block(256);
  timing_begin(GRADLEV_K_DECODE, s);
  switch (d) {
    case 16: hipLaunchKernelGGL(decode_kernel<16>, grid, block, 0, s, W, x, g, eta, eta_scalar, y, m); break;
    case 32: hipLaunchKernelGGL(decode_kernel<32>, grid, block, 0, s, W, x, g, eta, eta_scalar, y, m); break;
    case 64: hipLaunchKernelGGL(decode_kernel<64>, grid, block, 0, s, W, x, g, eta, eta_scalar, y, m); break;
    case 128: hipLaunchKernelGGL(decode_kernel<128>, grid, block, 0, s, W, x, g, eta, eta_scalar, y, m); break;
    case 256: hipLaunchKernelGGL(decode_kernel<256>, grid, block, 0, s, W, x, g, eta, eta_scalar, y, m); break;
    default: timing_end(GRADLEV_K_DECODE, s); return hipErrorInvalidValue;
  }
  timing_end(GRADLEV_K_DECODE, s);
  return hipGetLastError();
}

}  // namespace gradlev
