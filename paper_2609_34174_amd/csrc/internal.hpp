// Host-side interface between the C ABI layer and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gradlev {

// One forward/backward problem after validation and planning.
struct ScanProblem {
  int64_t B, H, T;
  int d, m;          // d_in, d_out
  int bf16;          // 1: X, G, dY are bf16; 0: fp32
  int inclusive;     // 1: inclusive reads
  int chunk;         // effective tile length of the kernel in use
  int64_t seg_len;   // tokens per segment (multiple of chunk)
  int64_t nseg;      // segments per sequence
};

struct FwdPtrs {
  const float* W0;
  const void* X;
  const void* G;
  const float* eta;
  float eta_scalar;
  float* Y;
  float* agg;   // [B*H][nseg][m][d] workspace, or nullptr when nseg == 1
  float* wend;  // [B*H][nsave][m][d] weights after each save_len-token block (for a backward), or nullptr
  int64_t save_len, nsave;  // the backward's segment length and count (a multiple of the chunk)
  const uint8_t* reset;     // [B][T] document starts (unit retention with resets), or nullptr
  float* cstate;            // with resets: [B*H][ceil(T/64)][d][m] chunk-start states of reset chunks, transposed
  bool resets;              // run the reset kernels (reset may still be nullptr: no document starts)
  int* segreset;            // with resets: [B*H][nseg] workspace ints (each segment's last document start)
};

struct BwdPtrs {
  const float* W0;
  const void* X;
  const void* G;
  const float* eta;
  float eta_scalar;
  const void* dY;
  float* gtilde;
  float* dX;
  float* dG;
  float* deta;
  float* dW0;
  float* aggA;   // [B*H][nseg][d][m]: segment write aggregates (transposed)
  float* aggB;   // [B*H][nseg][d][m]: segment dY x^T aggregates (transposed)
  float* rfin;  // [B*H][m][d]: full-sequence sum of dY x^T per sequence
  const float* wend;  // the forward's saved segment-end weights (same segments), or nullptr
  const uint8_t* reset;  // document starts, with `resets`
  const float* cstate;   // the forward's chunk-start states of reset chunks, with `resets`
  float* aggF;           // with resets: [B*H][nseg][d][m] full dY x^T per segment (for dW0)
  bool resets;
  int* segreset;         // with resets: [B*H][nseg] workspace ints (each segment's first document start)
};

// Gated scans (retention and resets).  Workspace: segment aggregates
// A_k = sum eta_s (prod_{s<j<end} alpha_j) g_s x_s^T, B_k = sum (prod_{start<=j<u}
// alpha_j) dY_u x_u^T, Bu_k = sum dY_u x_u^T (all [m][d]), the segment decays
// D_k = prod alpha, and for the backward the state at every chunk start.
struct GatedPtrs {
  const float* W0;
  const void* X;
  const void* G;
  const void* dY;
  const float* eta;
  float eta_scalar;
  float eta_mul;  // step size = eta_mul * (eta ? eta[t] : eta_scalar)
  const float* alpha;
  float alpha_scalar;
  const uint8_t* reset;
  float* Y;
  float* gtilde;
  float* dX;
  float* dG;
  float* deta;
  float* dalpha;
  float* dW0;
  float* aggA;    // [B*H][nseg][m][d]
  float* aggB;    // [B*H][nseg][m][d] (backward)
  float* aggBu;   // [B*H][nseg][m][d] (backward)
  float* aggD;    // [B*H][nseg]
  float* states;  // [B*H][ceil(T/chunk)][m*d] (backward), in the backward's register order
  bool saved_states;  // backward: states were written by a saving forward (no state pass, no A)
};

struct DecodeGates {
  const float* W0;
  const float* alpha;
  float alpha_scalar;
  const uint8_t* reset;
};

// Two-map MLP elementwise stages (n values, a multiple of 4).
hipError_t launch_act_fwd(int bf16, const float* Z, void* H, int64_t n, int kind, hipStream_t s);
hipError_t launch_act_bwd(int bf16, const float* Z, float* G, void* Gq, int64_t n, int kind, hipStream_t s);
hipError_t launch_mlp_gate_grads(const float* de1, const float* de2, float s1, float s2, float* dmu,
                                 const float* da1, float* dalpha, int64_t n, hipStream_t s);

int gated_fwd_chunk(int bf16, int d, int m);
int gated_bwd_chunk(int bf16, int d, int m);
int gated_wgs_per_cu(int fwd, int bf16, int d, int m);
hipError_t launch_scan_fwd_gated(const ScanProblem& p, const GatedPtrs& a, hipStream_t s);
hipError_t launch_scan_bwd_gated(const ScanProblem& p, const GatedPtrs& a, hipStream_t s);

// Tile lengths each kernel family supports for a shape (LDS budget).
int fwd_chunk_for(int bf16, int d, int m, int requested);
int bwd_chunk_for(int bf16, int d, int m, int requested);
// Resident workgroups per CU for the main kernels (LDS bound).
int fwd_wgs_per_cu(int bf16, int d, int m, int chunk);
int bwd_wgs_per_cu(int bf16, int d, int m, int chunk);

// Wide maps (parallel form, scan_wide.hip): d and m multiples of 128, at
// least one above 128; exclusive reads.  fmode: 0 no retention or resets
// (F = 1), 1 resets only (F in {0, 1}), 2 general retention.
struct WideProblem {
  int64_t B, H, T, Tp;  // Tp: T rounded up to a multiple of 128
  int d, m;
  int bf16;
  int fmode;
};

struct WidePtrs {
  const float* W0;
  const void* X;
  const void* G;
  const void* dY;
  const float* eta;
  float eta_scalar;
  float eta_mul;
  const float* alpha;
  float alpha_scalar;
  const uint8_t* reset;
  float* Y;
  float* gtilde;
  float* dX;
  float* dG;
  float* deta;
  float* dalpha;
  float* dW0;
  void* ws;  // wide_workspace_bytes
};

size_t wide_workspace_bytes(const WideProblem& p);
hipError_t launch_wide_fwd(const WideProblem& p, const WidePtrs& a, hipStream_t s);
// Backward of a wide map: gtilde, dX, dG, deta, dalpha and dW0 (each when non-null).
hipError_t launch_wide_read(const WideProblem& p, const WidePtrs& a, hipStream_t s);

// Optional event timing around each kernel launch (see gradlev_timing_*).
void timing_begin(int family, hipStream_t s);
void timing_end(int family, hipStream_t s);

hipError_t launch_scan_fwd(const ScanProblem& p, const FwdPtrs& a, hipStream_t s);
hipError_t launch_scan_bwd(const ScanProblem& p, const BwdPtrs& a, hipStream_t s);
hipError_t launch_decode(int64_t S, int64_t H, int d, int m, float* W, const float* x,
                         const float* g, const float* eta, float eta_scalar, float* y,
                         hipStream_t s, const DecodeGates* gates = nullptr);

}  // namespace gradlev
