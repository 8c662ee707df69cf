// Elementwise stages of the two-map online MLP (Appendix A): the hidden
// activation between the two scans, h = sigma(z), the reverse target of the
// hidden layer, g_z = sigma'(z) * g_h, and the combination of the two scans'
// gate gradients into those of the shared gates.  All are pure streams (a few
// flops per 8-16 bytes); the activation stages handle 4 consecutive values
// per thread with 16-byte accesses in a grid-stride loop.
#include "../../include/gradlev.h"
#include "device_common.hpp"
#include "internal.hpp"

namespace gradlev {

// tanh; GELU in its Gaussian-CDF form z * Phi(z); or the tanh-approximate
// GELU z/2 (1 + tanh(u)), u = sqrt(2/pi) (z + 0.044715 z^3).
constexpr float kGeluK0 = 0.79788456080286536f;  // sqrt(2/pi)
constexpr float kGeluK1 = 0.044715f;
__device__ __forceinline__ float act_value(float z, int kind) {
  if (kind == GRADLEV_ACT_TANH) return tanhf(z);
  if (kind == GRADLEV_ACT_GELU_TANH) return 0.5f * z * (1.f + tanhf(kGeluK0 * (z + kGeluK1 * z * z * z)));
  return 0.5f * z * (1.f + erff(z * 0.70710678118654752f));
}
__device__ __forceinline__ float act_slope(float z, int kind) {
  if (kind == GRADLEV_ACT_TANH) {
    const float t = tanhf(z);
    return 1.f - t * t;
  }
  if (kind == GRADLEV_ACT_GELU_TANH) {
    const float t = tanhf(kGeluK0 * (z + kGeluK1 * z * z * z));
    return 0.5f * (1.f + t) + 0.5f * z * (1.f - t * t) * kGeluK0 * (1.f + 3.f * kGeluK1 * z * z);
  }
  // Phi(z) + z phi(z), phi the standard normal density.
  return 0.5f * (1.f + erff(z * 0.70710678118654752f)) + z * expf(-0.5f * z * z) * 0.39894228040143268f;
}

template <typename E>
__device__ __forceinline__ void store4e(E* p, f32x4 v);
template <>
__device__ __forceinline__ void store4e<float>(float* p, f32x4 v) {
  *reinterpret_cast<f32x4*>(p) = v;
}
template <>
__device__ __forceinline__ void store4e<bf16>(bf16* p, f32x4 v) {
  bf16x4 o;
#pragma unroll
  for (int r = 0; r < 4; ++r) o[r] = (bf16)v[r];
  *reinterpret_cast<bf16x4*>(p) = o;
}

template <typename E>
__global__ void __launch_bounds__(256)
act_fwd_kernel(const float* __restrict__ Z, E* __restrict__ H, int64_t n4, int kind) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    const f32x4 z = *reinterpret_cast<const f32x4*>(Z + 4 * i);
    f32x4 h;
#pragma unroll
    for (int r = 0; r < 4; ++r) h[r] = act_value(z[r], kind);
    store4e<E>(H + 4 * i, h);
  }
}

template <typename E>
__global__ void __launch_bounds__(256)
act_bwd_kernel(const float* __restrict__ Z, float* __restrict__ G, E* __restrict__ Gq, int64_t n4, int kind) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    const f32x4 z = *reinterpret_cast<const f32x4*>(Z + 4 * i);
    f32x4 g = *reinterpret_cast<const f32x4*>(G + 4 * i);
#pragma unroll
    for (int r = 0; r < 4; ++r) g[r] *= act_slope(z[r], kind);
    *reinterpret_cast<f32x4*>(G + 4 * i) = g;
    if (Gq) store4e<E>(Gq + 4 * i, g);
  }
}

static unsigned act_grid(int64_t n4) {
  const int64_t b = (n4 + 255) / 256;
  return (unsigned)(b < 8192 ? (b < 1 ? 1 : b) : 8192);
}

// The shared gates' gradients from the two scans' (Appendix A: both maps use
// the write strength mu, with eta_1 = mu / d_in and eta_2 = mu / hidden, and
// the same retention):  dmu = deta_1 / d_in + deta_2 / hidden,
// dalpha += dalpha_1 (dalpha already holds the second scan's).
__global__ void __launch_bounds__(256)
mlp_gate_grads_kernel(const float* __restrict__ de1, const float* __restrict__ de2, float s1, float s2,
                      float* __restrict__ dmu, const float* __restrict__ da1, float* __restrict__ dalpha, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    if (dmu) dmu[i] = de1[i] * s1 + de2[i] * s2;
    if (dalpha) dalpha[i] += da1[i];
  }
}

hipError_t launch_mlp_gate_grads(const float* de1, const float* de2, float s1, float s2, float* dmu,
                                 const float* da1, float* dalpha, int64_t n, hipStream_t s) {
  const int64_t b = (n + 255) / 256;
  hipLaunchKernelGGL(mlp_gate_grads_kernel, dim3((unsigned)(b < 4096 ? b : 4096)), dim3(256), 0, s, de1, de2, s1, s2,
                     dmu, da1, dalpha, n);
  return hipGetLastError();
}

hipError_t launch_act_fwd(int is_bf16, const float* Z, void* H, int64_t n, int kind, hipStream_t s) {
  const int64_t n4 = n / 4;
  if (is_bf16)
    hipLaunchKernelGGL(act_fwd_kernel<bf16>, dim3(act_grid(n4)), dim3(256), 0, s, Z, static_cast<bf16*>(H), n4, kind);
  else
    hipLaunchKernelGGL(act_fwd_kernel<float>, dim3(act_grid(n4)), dim3(256), 0, s, Z, static_cast<float*>(H), n4, kind);
  return hipGetLastError();
}

hipError_t launch_act_bwd(int is_bf16, const float* Z, float* G, void* Gq, int64_t n, int kind, hipStream_t s) {
  const int64_t n4 = n / 4;
  if (is_bf16)
    hipLaunchKernelGGL(act_bwd_kernel<bf16>, dim3(act_grid(n4)), dim3(256), 0, s, Z, G, static_cast<bf16*>(Gq), n4, kind);
  else
    hipLaunchKernelGGL(act_bwd_kernel<float>, dim3(act_grid(n4)), dim3(256), 0, s, Z, G, static_cast<float*>(Gq), n4, kind);
  return hipGetLastError();
}

}  // namespace gradlev
