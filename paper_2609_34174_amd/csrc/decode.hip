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

template <int D, bool GATED, bool STREAM>
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
      buf_store4<STREAM ? kStoreStream : kStoreDefault>(Ws, (uint32_t)((i * D + col) * 4), nw);
    }
  }
}

// Wide states (d_in = 256 NCH, NCH in {2, 4, ..., 32}): one wave per state
// row, the row streamed in 256-column chunks (lane l holds columns 4l..4l+3
// of each chunk: every load and store is a contiguous 1 KiB per wave).  A
// wave takes U rows at a time with all their chunks' loads issued together
// (U * NCH = 16 or more 16-byte loads in flight per lane), computes the dot
// products from the loaded (pre-update) values, writes the update from the
// same registers and reduces each row's dot product across the wave.  x sits
// in LDS, loaded once per workgroup.  Workgroup: 4 waves, 4 U rows.
template <int NCH, bool GATED, bool STREAM>
__global__ void __launch_bounds__(256)
decode_wide_kernel(float* __restrict__ W, const float* __restrict__ x, const float* __restrict__ g,
                   const float* __restrict__ eta, float eta_scalar, float* __restrict__ y, int M,
                   const float* __restrict__ W0, int64_t H, const float* __restrict__ alpha,
                   float alpha_scalar, const uint8_t* __restrict__ reset, int64_t blocks_per_state) {
  constexpr int D = 256 * NCH;
  constexpr int U = NCH >= 16 ? 1 : 16 / NCH;  // rows per wave per pass
  __shared__ __attribute__((aligned(16))) float xs[D];
  const int64_t sh = blockIdx.x / blocks_per_state;
  const int64_t rb = blockIdx.x % blocks_per_state;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int i = tid; i < D / 4; i += 256)
    reinterpret_cast<f32x4*>(xs)[i] = reinterpret_cast<const f32x4*>(x + sh * D)[i];
  __syncthreads();
  const rsrc_t Ws = make_rsrc(W + sh * (int64_t)M * D, (uint32_t)((int64_t)M * D * 4));
  const rsrc_t Gs = make_rsrc(g + sh * (int64_t)M, (uint32_t)(M * 4));
  const rsrc_t Ys = make_rsrc(y + sh * (int64_t)M, (uint32_t)(M * 4));
  const rsrc_t W0s = make_rsrc(GATED ? W0 + (sh % H) * (int64_t)M * D : nullptr,
                               GATED ? (uint32_t)((int64_t)M * D * 4) : 0u);
  const float al = GATED ? (alpha ? alpha[sh] : alpha_scalar) : 1.f;
  const bool fresh = GATED && reset && reset[sh / H] != 0;
  const float e = eta ? eta[sh] : eta_scalar;
  // Rows of this wave; rows past M read zero and their stores are dropped.
  const int r0 = (int)(rb * 4 * U) + w * U;
  f32x4 wv[U][NCH], w0[GATED ? U : 1][GATED ? NCH : 1];
  float gv[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    gv[u] = buf_load1(Gs, (uint32_t)((r0 + u) * 4));
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const uint32_t o = (uint32_t)((((int64_t)(r0 + u)) * D + 256 * c + 4 * lane) * 4);
      wv[u][c] = buf_load4(Ws, o, (const float*)nullptr);
      if constexpr (GATED) w0[u][c] = buf_load4(W0s, o, (const float*)nullptr);
    }
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const f32x4 xv = *reinterpret_cast<const f32x4*>(xs + 256 * c + 4 * lane);
      f32x4 v = wv[u][c];
      if constexpr (GATED) {
        if (fresh) v = w0[u][c];
      }
      s += v[0] * xv[0] + v[1] * xv[1] + v[2] * xv[2] + v[3] * xv[3];
      f32x4 nw;
      if constexpr (GATED) nw = w0[u][c] + al * (v - w0[u][c]) - (e * gv[u]) * xv;
      else nw = v - (e * gv[u]) * xv;
      buf_store4<STREAM ? kStoreStream : kStoreDefault>(Ws, (uint32_t)((((int64_t)(r0 + u)) * D + 256 * c + 4 * lane) * 4), nw);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
    buf_store1<kStoreDefault>(Ys, lane == 0 ? (uint32_t)((r0 + u) * 4) : kOOB, s);
  }
}

// State stores: a state that the 256 MB Infinity Cache can keep between
// steps is written with the default policy (the next step reads it back from
// the cache); a larger one is streamed past the L2, like the scans' outputs
// (measured at 256 x 16 states of 64 x 64: 64 MiB, 23.9 us per step either
// way; 2048 x 16: 512 MiB, 200 -> 189 us per step).
constexpr int64_t kDecodeStreamBytes = int64_t(128) << 20;
static bool decode_stream(int64_t S, int64_t H, int d, int m) { return S * H * (int64_t)d * m * 4 > kDecodeStreamBytes; }

static hipError_t launch_decode_wide(int64_t S, int64_t H, int d, int m, float* W, const float* x,
                                     const float* g, const float* eta, float eta_scalar, float* y,
                                     hipStream_t s, const DecodeGates* gt) {
  const float* W0 = gt ? gt->W0 : nullptr;
  const float* al = gt ? gt->alpha : nullptr;
  const float as = gt ? gt->alpha_scalar : 1.f;
  const uint8_t* rs = gt ? gt->reset : nullptr;
  const int nch = d / 256;
  const int U = nch >= 16 ? 1 : 16 / nch;
  const int64_t bps = (m + 4 * U - 1) / (4 * U);
  const dim3 grid((unsigned)(S * H * bps)), block(256);
  const bool st = decode_stream(S, H, d, m);
#define GL_DECODE_W1(N, G, ST)                                                                    \
  hipLaunchKernelGGL((decode_wide_kernel<N, G, ST>), grid, block, 0, s, W, x, g, eta, eta_scalar, \
                     y, m, W0, H, al, as, rs, bps)
#define GL_DECODE_W(N)              \
  if (gt && st)                     \
    GL_DECODE_W1(N, true, true);    \
  else if (gt)                      \
    GL_DECODE_W1(N, true, false);   \
  else if (st)                      \
    GL_DECODE_W1(N, false, true);   \
  else                              \
    GL_DECODE_W1(N, false, false);
  switch (nch) {
    case 2: GL_DECODE_W(2) break;
    case 4: GL_DECODE_W(4) break;
    case 8: GL_DECODE_W(8) break;
    case 16: GL_DECODE_W(16) break;
    case 32: GL_DECODE_W(32) break;
    default: return hipErrorInvalidValue;
  }
#undef GL_DECODE_W
#undef GL_DECODE_W1
  return hipGetLastError();
}

hipError_t launch_decode(int64_t S, int64_t H, int d, int m, float* W, const float* x,
                         const float* g, const float* eta, float eta_scalar, float* y,
                         hipStream_t s, const DecodeGates* gt) {
  const dim3 grid((unsigned)(S * H)), block(256);
  const float* W0 = gt ? gt->W0 : nullptr;
  const float* al = gt ? gt->alpha : nullptr;
  const float as = gt ? gt->alpha_scalar : 1.f;
  const uint8_t* rs = gt ? gt->reset : nullptr;
  const bool st = decode_stream(S, H, d, m);
#define GL_DECODE1(DD, G, ST)                                                                    \
  hipLaunchKernelGGL((decode_kernel<DD, G, ST>), grid, block, 0, s, W, x, g, eta, eta_scalar, y, m, \
                     W0, H, al, as, rs)
#define GL_DECODE(DD)            \
  if (gt && st)                  \
    GL_DECODE1(DD, true, true);  \
  else if (gt)                   \
    GL_DECODE1(DD, true, false); \
  else if (st)                   \
    GL_DECODE1(DD, false, true); \
  else                           \
    GL_DECODE1(DD, false, false);
  timing_begin(GRADLEV_K_DECODE, s);
  if (d > 256) {
    const hipError_t e = launch_decode_wide(S, H, d, m, W, x, g, eta, eta_scalar, y, s, gt);
    timing_end(GRADLEV_K_DECODE, s);
    return e;
  }
  switch (d) {
    case 16: GL_DECODE(16) break;
    case 32: GL_DECODE(32) break;
    case 64: GL_DECODE(64) break;
    case 128: GL_DECODE(128) break;
    case 256: GL_DECODE(256) break;
    default: timing_end(GRADLEV_K_DECODE, s); return hipErrorInvalidValue;
  }
#undef GL_DECODE
#undef GL_DECODE1
  timing_end(GRADLEV_K_DECODE, s);
  return hipGetLastError();
}

}  // namespace gradlev
