// C ABI of the GradLev scan library: argument validation, work planning,
// workspace layout and dispatch to the gfx950 kernels.  Every check runs on
// the host before any HIP runtime call, so invalid calls return a status code
// without touching a device.
#include <stddef.h>
#include <stdint.h>

#include <mutex>

#include "../../include/gradlev.h"
#include "internal.hpp"

// Device scratch of gradlev_scan_fwd_static: one copy per GPU, at its own
// address on each.  Host code never uses this name as an address (on the host
// it is only a stand-in for the symbol); it uses the pointer that
// static_scratch() looks up per device.
static __device__ __align__(256) unsigned char scratch[GRADLEV_STATIC_SCRATCH_BYTES];

namespace gradlev {
namespace {

constexpr int kNumCU = 256;           // MI355X compute units
constexpr int64_t kMaxElems = int64_t(1) << 40;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// The scan kernels run a 1-D grid of 8 * nseg * ceil(BH / 8) workgroups of
// at most 1024 work-items (the widest, 16-wave kernels); the grid's
// work-item count must stay below 2^32.
constexpr int64_t kMaxBlockThreads = 1024;
bool grid_fits(int64_t BH, int64_t nseg) {
  return 8 * nseg * ((BH + 7) / 8) <= ((int64_t(1) << 32) - 1) / kMaxBlockThreads;
}

struct Plan {
  ScanProblem fwd, bwd;
  int64_t save_len;  // save-for-backward pair: tokens per saved state (the backward's segment)
  size_t ws_fwd, ws_bwd;
  // Offsets (bytes) inside the workspace.
  size_t off_aggA, off_aggB, off_rfin;
};

int64_t pick_nseg(int64_t BH, int64_t T, int C, int wgs_per_cu, int64_t hint) {
  const int64_t nchunks = (T + C - 1) / C;
  int64_t seg_chunks;
  if (hint > 0) {
    seg_chunks = (hint + C - 1) / C;
  } else {
    const int64_t target = (int64_t)kNumCU * wgs_per_cu;
    int64_t nseg = (target + BH - 1) / BH;
    if (nseg < 1) nseg = 1;
    if (nseg > nchunks) nseg = nchunks;
    if (nseg > 16) nseg = 16;  // a main workgroup sums at most 15 predecessor aggregates
    seg_chunks = (nchunks + nseg - 1) / nseg;
  }
  if (seg_chunks < 1) seg_chunks = 1;
  return seg_chunks;
}

// Workspace of a plan: forward segment aggregates; backward aggregates A_k,
// B_k and the per-sequence dY x^T sums.
void layout_ws(Plan* out, int64_t BH, size_t md) {
  out->ws_fwd = out->fwd.nseg > 1 ? round_up((size_t)BH * out->fwd.nseg * md, 256) : 0;
  const size_t agg_b = out->bwd.nseg > 1 ? round_up((size_t)BH * out->bwd.nseg * md, 256) : 0;
  out->off_aggA = 0;
  out->off_aggB = round_up((size_t)BH * out->bwd.nseg * md, 256);
  out->off_rfin = out->off_aggB + agg_b;
  out->ws_bwd = out->off_rfin + round_up((size_t)BH * md, 256);
}

int make_plan(const gradlev_shape* s, Plan* out) {
  if (!s || !out) return GRADLEV_ERR_INVALID;
  if (s->B < 1 || s->H < 1 || s->T < 1 || s->d_in < 1 || s->d_out < 1) return GRADLEV_ERR_INVALID;
  if (s->in_dtype != GRADLEV_F32 && s->in_dtype != GRADLEV_BF16) return GRADLEV_ERR_INVALID;
  if (s->prefix != GRADLEV_EXCLUSIVE && s->prefix != GRADLEV_INCLUSIVE) return GRADLEV_ERR_INVALID;
  if (s->chunk < 0 || s->segment < 0) return GRADLEV_ERR_INVALID;
  if ((s->d_in != 64 && s->d_in != 128) || (s->d_out != 64 && s->d_out != 128)) return GRADLEV_ERR_UNSUPPORTED;
  if (s->chunk != 0 && s->chunk != 64 && s->chunk != 128) return GRADLEV_ERR_UNSUPPORTED;
  if (s->segment % 64 != 0) return GRADLEV_ERR_UNSUPPORTED;
  const int64_t BH = s->B * s->H;
  if (s->B > kMaxElems / s->H || BH > kMaxElems / s->T) return GRADLEV_ERR_UNSUPPORTED;
  const int64_t wmax = s->d_in > s->d_out ? s->d_in : s->d_out;
  if (BH * s->T > kMaxElems / wmax) return GRADLEV_ERR_UNSUPPORTED;
  // Per-sequence byte offsets are 32-bit (buffer addressing): T * width * 4 < 2^31.
  if (s->T > (int64_t(1) << 31) / (4 * wmax) - 1) return GRADLEV_ERR_UNSUPPORTED;
  if (BH > (int64_t(1) << 26)) return GRADLEV_ERR_UNSUPPORTED;  // 1-D grid of 8 * nseg * ceil(BH / 8) blocks

  const int bf = s->in_dtype == GRADLEV_BF16;
  const int d = (int)s->d_in, m = (int)s->d_out;
  const size_t md = (size_t)m * d * sizeof(float);

  ScanProblem base{};
  base.B = s->B;
  base.H = s->H;
  base.T = s->T;
  base.d = d;
  base.m = m;
  base.bf16 = bf;
  base.inclusive = s->prefix == GRADLEV_INCLUSIVE;

  out->fwd = base;
  out->fwd.chunk = fwd_chunk_for(bf, d, m, (int)s->chunk);
  int64_t sc = pick_nseg(BH, s->T, out->fwd.chunk, fwd_wgs_per_cu(bf, d, m, out->fwd.chunk), s->segment);
  out->fwd.seg_len = sc * out->fwd.chunk;
  out->fwd.nseg = (s->T + out->fwd.seg_len - 1) / out->fwd.seg_len;
  if (out->fwd.nseg > 16) return GRADLEV_ERR_UNSUPPORTED;

  out->bwd = base;
  out->bwd.chunk = bwd_chunk_for(bf, d, m, (int)s->chunk);
  sc = pick_nseg(BH, s->T, out->bwd.chunk, bwd_wgs_per_cu(bf, d, m, out->bwd.chunk), s->segment);
  out->bwd.seg_len = sc * out->bwd.chunk;
  out->bwd.nseg = (s->T + out->bwd.seg_len - 1) / out->bwd.seg_len;
  if (out->bwd.nseg > 16) return GRADLEV_ERR_UNSUPPORTED;
  if (!grid_fits(BH, out->fwd.nseg) || !grid_fits(BH, out->bwd.nseg)) return GRADLEV_ERR_UNSUPPORTED;

  out->save_len = out->bwd.seg_len;
  layout_ws(out, BH, md);
  return GRADLEV_OK;
}

// The save-for-backward pair: the forward saves the weights after each of
// the backward's segments and the backward starts its segments from them.
// The backward keeps its own segmentation, rounded up to the forward's tile
// so that no forward tile straddles a saved boundary (the backward tile, 32
// or 64 tokens, divides the forward's, 64 or 128); the forward's segments
// are rounded up to whole backward segments.
int make_saved_plan(const gradlev_shape* s, Plan* out, size_t* saved_bytes) {
  const int rc = make_plan(s, out);
  if (rc != GRADLEV_OK) return rc;
  const int64_t fc = out->fwd.chunk;
  const int64_t sb = (out->bwd.seg_len + fc - 1) / fc * fc;
  out->bwd.seg_len = sb;
  out->bwd.nseg = (s->T + sb - 1) / sb;
  const int64_t sf = (out->fwd.seg_len + sb - 1) / sb * sb;
  out->fwd.seg_len = sf;
  out->fwd.nseg = (s->T + sf - 1) / sf;
  if (!grid_fits(s->B * s->H, out->bwd.nseg)) return GRADLEV_ERR_UNSUPPORTED;
  out->save_len = sb;
  const size_t md = (size_t)s->d_out * s->d_in * sizeof(float);
  layout_ws(out, s->B * s->H, md);
  *saved_bytes = (size_t)(s->B * s->H) * out->bwd.nseg * md;
  return GRADLEV_OK;
}

// The save-for-backward pair with document resets at unit retention: the
// saved plan at 64-token tiles for both directions (the backward restarts its
// un-write at the forward's chunk-start states, so the two share the tile).
// Saved: segment-end weights [BH][nseg_b][m][d], then the chunk-start states
// [BH][ceil(T/64)][d][m], transposed (written only for chunks that hold a reset).
// Workspace: forward aggregates [BH][nseg_f][m][d]; backward pre-reset and
// full dY x^T aggregates [BH][nseg_b][d][m] each; then one int per segment
// (its last / first document start, recorded by the aggregate passes).
struct ResetPlan {
  Plan p;
  size_t off_cstate, saved_bytes;
  size_t off_aggF, off_seg, ws;
};

int make_reset_plan(const gradlev_shape* s, ResetPlan* out) {
  if (!s) return GRADLEV_ERR_INVALID;
  if (s->B < 1 || s->H < 1 || s->T < 1 || s->d_in < 1 || s->d_out < 1) return GRADLEV_ERR_INVALID;
  if (s->d_in != 64 || s->d_out != 64 || s->prefix != GRADLEV_EXCLUSIVE) return GRADLEV_ERR_UNSUPPORTED;
  gradlev_shape s64 = *s;
  s64.chunk = 64;
  size_t sv = 0;
  const int rc = make_saved_plan(&s64, &out->p, &sv);
  if (rc != GRADLEV_OK) return rc;
  if (out->p.fwd.chunk != 64 || out->p.bwd.chunk != 64) return GRADLEV_ERR_UNSUPPORTED;
  const int64_t BH = s->B * s->H;
  const size_t md = (size_t)64 * 64 * sizeof(float);
  // One sequence's chunk-start states stay under 2 GiB (32-bit offsets).
  const int64_t nch = (s->T + 63) / 64;
  if (nch > ((int64_t(1) << 31) - 1) / (int64_t)md) return GRADLEV_ERR_UNSUPPORTED;
  out->off_cstate = round_up(sv, 256);
  out->saved_bytes = out->off_cstate + (size_t)BH * nch * md;
  const size_t agg_f = out->p.fwd.nseg > 1 ? round_up((size_t)BH * out->p.fwd.nseg * md, 256) : 0;
  const size_t agg_b = round_up((size_t)BH * out->p.bwd.nseg * md, 256);
  out->off_aggF = agg_b;
  out->off_seg = agg_f > 2 * agg_b ? agg_f : 2 * agg_b;
  const int64_t nseg = out->p.fwd.nseg > out->p.bwd.nseg ? out->p.fwd.nseg : out->p.bwd.nseg;
  out->ws = out->off_seg + round_up((size_t)BH * nseg * sizeof(int), 256);
  return GRADLEV_OK;
}

// Wide maps: widths that are multiples of 128 with one of them above 128 run
// the parallel form (scan_wide.hip).  Its workspace holds the gate prefixes
// and the causal score matrix, B*H*Tp*Tp*4 bytes, so the sequence length is
// capped; reads are exclusive (the paper's convention).
constexpr int64_t kWideMaxWidth = 8192;
constexpr int64_t kWideMaxT = 16384;

bool wide_shape(const gradlev_shape* s) { return s && (s->d_in > 128 || s->d_out > 128); }

int make_wide(const gradlev_shape* s, WideProblem* out) {
  if (!s || !out) return GRADLEV_ERR_INVALID;
  if (s->B < 1 || s->H < 1 || s->T < 1 || s->d_in < 1 || s->d_out < 1) return GRADLEV_ERR_INVALID;
  if (s->in_dtype != GRADLEV_F32 && s->in_dtype != GRADLEV_BF16) return GRADLEV_ERR_INVALID;
  if (s->prefix != GRADLEV_EXCLUSIVE && s->prefix != GRADLEV_INCLUSIVE) return GRADLEV_ERR_INVALID;
  if (s->chunk < 0 || s->segment < 0) return GRADLEV_ERR_INVALID;
  if (s->prefix != GRADLEV_EXCLUSIVE) return GRADLEV_ERR_UNSUPPORTED;
  if (s->d_in % 128 != 0 || s->d_out % 128 != 0) return GRADLEV_ERR_UNSUPPORTED;
  if (s->d_in > kWideMaxWidth || s->d_out > kWideMaxWidth || s->T > kWideMaxT) return GRADLEV_ERR_UNSUPPORTED;
  if (s->B > kMaxElems / s->H || s->B * s->H > (int64_t(1) << 20)) return GRADLEV_ERR_UNSUPPORTED;
  out->B = s->B;
  out->H = s->H;
  out->T = s->T;
  out->Tp = (s->T + 127) / 128 * 128;
  out->d = (int)s->d_in;
  out->m = (int)s->d_out;
  out->bf16 = s->in_dtype == GRADLEV_BF16;
  out->fmode = 0;
  // Grid sizes (work-items are counted in 32 bits) and 32-bit byte offsets
  // within one sequence's score matrix and rows.
  const int64_t BH = s->B * s->H, Kp = out->Tp / 128;
  const int64_t wmax = s->d_in > s->d_out ? s->d_in : s->d_out;
  if (BH * Kp * (wmax / 128) > (int64_t(1) << 23) || BH * 2 * Kp * (Kp + 1) > (int64_t(1) << 24))
    return GRADLEV_ERR_UNSUPPORTED;
  return GRADLEV_OK;
}

WidePtrs wide_ptrs(const gradlev_gates* g, const float* W0, const void* X, const void* G, const float* eta,
                   float eta_scalar, float eta_mul, void* ws) {
  WidePtrs f{};
  f.W0 = W0;
  f.X = X;
  f.G = G;
  f.eta = eta;
  f.eta_scalar = eta_scalar;
  f.eta_mul = eta_mul;
  f.alpha = g ? g->alpha : nullptr;
  f.alpha_scalar = g ? g->alpha_scalar : 1.f;
  f.reset = g ? g->reset : nullptr;
  f.ws = ws;
  return f;
}

// Retention mode of the wide kernels: products of ones, resets only, or
// general retentions.
int wide_fmode(const gradlev_gates* g) {
  if (!g) return 0;
  if (g->alpha || g->alpha_scalar != 1.f) return 2;
  return g->reset ? 1 : 0;
}

// Gated plan: tile lengths of the gated kernels, segments picked as for the
// unit-retention scans, and the workspace layout of GatedPtrs.
struct GatedPlan {
  ScanProblem fwd, bwd;
  size_t ws_fwd, ws_bwd;
  size_t off_A, off_B, off_Bu, off_D, off_S;  // backward layout (forward: A then D)
};

int make_gated_plan(const gradlev_shape* s, GatedPlan* out) {
  Plan base;
  const int rc = make_plan(s, &base);
  if (rc != GRADLEV_OK) return rc;
  if (s->prefix != GRADLEV_EXCLUSIVE) return GRADLEV_ERR_UNSUPPORTED;
  const int64_t BH = s->B * s->H;
  const size_t md = (size_t)s->d_out * s->d_in * sizeof(float);
  const int bf = s->in_dtype == GRADLEV_BF16;
  const int d = (int)s->d_in, m = (int)s->d_out;
  for (int k = 0; k < 2; ++k) {
    ScanProblem& q = k == 0 ? out->fwd : out->bwd;
    q = k == 0 ? base.fwd : base.bwd;
    q.chunk = k == 0 ? gated_fwd_chunk(bf, d, m) : gated_bwd_chunk(bf, d, m);
    const int64_t sc = pick_nseg(BH, s->T, q.chunk, gated_wgs_per_cu(k == 0, bf, d, m), s->segment);
    q.seg_len = sc * q.chunk;
    q.nseg = (s->T + q.seg_len - 1) / q.seg_len;
    if (q.nseg > 16 || !grid_fits(BH, q.nseg)) return GRADLEV_ERR_UNSUPPORTED;
  }
  // The backward addresses one sequence's chunk-start states with 32-bit
  // buffer offsets: ceil(T / chunk) * m * d * 4 < 2^31.
  const int64_t nchunk = (s->T + out->bwd.chunk - 1) / out->bwd.chunk;
  if (nchunk > ((int64_t(1) << 31) - 1) / (int64_t)md) return GRADLEV_ERR_UNSUPPORTED;
  const size_t nf = (size_t)BH * out->fwd.nseg, nb = (size_t)BH * out->bwd.nseg;
  out->ws_fwd = out->fwd.nseg > 1 ? round_up(nf * md, 256) + round_up(nf * 4, 256) : 0;
  const size_t nch = (size_t)BH * ((s->T + out->bwd.chunk - 1) / out->bwd.chunk);
  out->off_A = 0;
  out->off_B = round_up(nb * md, 256);
  out->off_Bu = out->off_B + round_up(nb * md, 256);
  out->off_D = out->off_Bu + round_up(nb * md, 256);
  out->off_S = out->off_D + round_up(nb * 4, 256);
  out->ws_bwd = out->off_S + round_up(nch * md, 256);
  return GRADLEV_OK;
}

// The gated save-for-backward pair: the forward runs on the backward's tile
// and writes Delta at every tile start into the saved buffer, in the order
// the backward loads it; the backward then needs no state pass and no write
// aggregates (its workspace ends before the state region).
int make_gated_saved_plan(const gradlev_shape* s, GatedPlan* out, size_t* saved_bytes) {
  const int rc = make_gated_plan(s, out);
  if (rc != GRADLEV_OK) return rc;
  const int64_t BH = s->B * s->H;
  const size_t md = (size_t)s->d_out * s->d_in * sizeof(float);
  const int bf = s->in_dtype == GRADLEV_BF16;
  out->fwd.chunk = out->bwd.chunk;
  const int64_t sc = pick_nseg(BH, s->T, out->fwd.chunk, gated_wgs_per_cu(1, bf, (int)s->d_in, (int)s->d_out),
                               s->segment);
  out->fwd.seg_len = sc * out->fwd.chunk;
  out->fwd.nseg = (s->T + out->fwd.seg_len - 1) / out->fwd.seg_len;
  if (out->fwd.nseg > 16 || !grid_fits(BH, out->fwd.nseg)) return GRADLEV_ERR_UNSUPPORTED;
  const size_t nf = (size_t)BH * out->fwd.nseg;
  out->ws_fwd = out->fwd.nseg > 1 ? round_up(nf * md, 256) + round_up(nf * 4, 256) : 0;
  *saved_bytes = (size_t)BH * ((s->T + out->bwd.chunk - 1) / out->bwd.chunk) * md;
  out->ws_bwd = out->off_S;
  return GRADLEV_OK;
}

int gated_fwd_planned(const gradlev_shape* s, const GatedPlan& p, const gradlev_gates* gates, const float* W0,
                      const void* X, const void* G, const float* eta, float eta_scalar, float* Y, float* states,
                      void* workspace, size_t workspace_bytes, void* stream);
int gated_bwd_planned(const GatedPlan& p, const gradlev_gates* gates, const float* W0, const void* X,
                      const void* G, const float* eta, float eta_scalar, const void* dY, const float* states,
                      float* gtilde, float* dX, float* dG, float* deta, float* dalpha, float* dW0, void* workspace,
                      size_t workspace_bytes, void* stream);

int check_gates(const gradlev_gates* g) {
  if (!g) return GRADLEV_ERR_INVALID;
  if (g->alpha && !aligned16(g->alpha)) return GRADLEV_ERR_ALIGN;
  return GRADLEV_OK;
}

// The two scans of the MLP, as gated scan shapes.
int make_mlp_shapes(const gradlev_mlp_shape* m, gradlev_shape* s1, gradlev_shape* s2) {
  if (!m) return GRADLEV_ERR_INVALID;
  if (m->act != GRADLEV_ACT_TANH && m->act != GRADLEV_ACT_GELU && m->act != GRADLEV_ACT_GELU_TANH) return GRADLEV_ERR_INVALID;
  *s1 = gradlev_shape{m->B, m->H, m->T, m->d_in, m->hidden, 0, m->segment, m->in_dtype, GRADLEV_EXCLUSIVE};
  *s2 = gradlev_shape{m->B, m->H, m->T, m->hidden, m->d_out, 0, m->segment, m->in_dtype, GRADLEV_EXCLUSIVE};
  return GRADLEV_OK;
}

struct MlpPlan {
  GatedPlan p1, p2;
  bool wide1, wide2;  // the scan runs the wide-map kernels (w1, w2) instead
  WideProblem w1, w2;
  size_t scan_ws;  // the larger of the two scans' workspaces (they run in turn)
  size_t off_q;    // in_dtype copy of the hidden target (queries the first scan)
  size_t off_g;    // the first scan's deta and dalpha, the second's deta ([B*H*T] fp32 each)
  size_t total;
};

int make_mlp_plan(const gradlev_mlp_shape* m, MlpPlan* out) {
  gradlev_shape s1, s2;
  int rc = make_mlp_shapes(m, &s1, &s2);
  if (rc != GRADLEV_OK) return rc;
  size_t w = 0;
  const gradlev_shape* sh[2] = {&s1, &s2};
  GatedPlan* gp[2] = {&out->p1, &out->p2};
  WideProblem* wp[2] = {&out->w1, &out->w2};
  bool* wd[2] = {&out->wide1, &out->wide2};
  for (int k = 0; k < 2; ++k) {
    *wd[k] = wide_shape(sh[k]);
    size_t need;
    if (*wd[k]) {
      rc = make_wide(sh[k], wp[k]);
      need = rc == GRADLEV_OK ? wide_workspace_bytes(*wp[k]) : 0;
    } else {
      rc = make_gated_plan(sh[k], gp[k]);
      need = gp[k]->ws_fwd > gp[k]->ws_bwd ? gp[k]->ws_fwd : gp[k]->ws_bwd;
    }
    if (rc != GRADLEV_OK) return rc;
    w = need > w ? need : w;
  }
  out->scan_ws = round_up(w, 256);
  out->off_q = out->scan_ws;
  const size_t es = m->in_dtype == GRADLEV_BF16 ? 2 : 4;
  out->off_g = out->off_q + round_up((size_t)(m->B * m->H * m->T * m->hidden) * es, 256);
  out->total = out->off_g + 3 * round_up((size_t)(m->B * m->H * m->T) * 4, 256);
  return GRADLEV_OK;
}

GatedPtrs gated_ptrs(const GatedPlan& p, const gradlev_gates* g, const float* W0, const void* X,
                     const void* G, const float* mu, float mu_scalar, float eta_mul, void* ws, bool bwd,
                     int64_t BH) {
  GatedPtrs f{};
  f.W0 = W0;
  f.X = X;
  f.G = G;
  f.eta = mu;
  f.eta_scalar = mu_scalar;
  f.eta_mul = eta_mul;
  f.alpha = g->alpha;
  f.alpha_scalar = g->alpha_scalar;
  f.reset = g->reset;
  char* w = static_cast<char*>(ws);
  if (bwd) {
    f.aggA = reinterpret_cast<float*>(w + p.off_A);
    f.aggB = reinterpret_cast<float*>(w + p.off_B);
    f.aggBu = reinterpret_cast<float*>(w + p.off_Bu);
    f.aggD = reinterpret_cast<float*>(w + p.off_D);
    f.states = reinterpret_cast<float*>(w + p.off_S);
  } else if (p.fwd.nseg > 1) {
    const size_t nf = (size_t)BH * p.fwd.nseg;
    f.aggA = reinterpret_cast<float*>(w);
    f.aggD = reinterpret_cast<float*>(w + round_up(nf * (size_t)p.fwd.m * p.fwd.d * sizeof(float), 256));
  }
  return f;
}

// Decode shapes: d_in in {16, ..., 256} with d_out <= 1024, or a wide state
// with d_in in {512, 1024, 2048, 4096, 8192} and d_out <= 65536 (one state
// must stay under 2 GiB for 32-bit buffer offsets, and the grid of
// S * H * ceil(d_out / rows per workgroup) workgroups within 2^31 work-items).
bool decode_shape_ok(int64_t S, int64_t H, int64_t d_in, int64_t d_out) {
  if (S > kMaxElems / H || S * H > 0x7fffffff) return false;
  // One 256-work-item workgroup per state: S * H * 256 work-items < 2^32.
  if (d_in == 16 || d_in == 32 || d_in == 64 || d_in == 128 || d_in == 256)
    return d_out <= 1024 && S * H < (int64_t(1) << 24);
  if (d_in != 512 && d_in != 1024 && d_in != 2048 && d_in != 4096 && d_in != 8192) return false;
  if (d_out > 65536 || d_in * d_out * 4 >= (int64_t(1) << 31)) return false;
  const int64_t nch = d_in / 256, rows = 4 * (nch >= 16 ? 1 : 16 / nch);
  return S * H * ((d_out + rows - 1) / rows) * 256 < (int64_t(1) << 31);
}

int check_workspace(void* ws, size_t have, size_t need) {
  if (need == 0) return GRADLEV_OK;
  if (!ws || have < need) return GRADLEV_ERR_WORKSPACE;
  if (!aligned16(ws)) return GRADLEV_ERR_ALIGN;
  return GRADLEV_OK;
}

// Device address of `scratch` on the current device, looked up once per
// device with that device current.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

int static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return GRADLEV_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return GRADLEV_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return GRADLEV_OK;
}

}  // namespace
}  // namespace gradlev

using namespace gradlev;

extern "C" {

int gradlev_version(void) { return 100; }

const char* gradlev_error_string(int code) {
  switch (code) {
    case GRADLEV_OK: return "success";
    case GRADLEV_ERR_INVALID: return "invalid argument (null pointer, non-positive size or unknown enum)";
    case GRADLEV_ERR_UNSUPPORTED: return "unsupported shape (d_in/d_out 64 or 128, or multiples of 128 up to 8192 with T <= 16384 and exclusive reads for wide maps; chunk 0/64/128, segment a multiple of 64 giving at most 16 segments; gated scans read exclusively)";
    case GRADLEV_ERR_ALIGN: return "a pointer is not 16-byte aligned";
    case GRADLEV_ERR_WORKSPACE: return "workspace missing or too small";
    case GRADLEV_ERR_HIP: return "HIP launch failed";
    case GRADLEV_ERR_SCRATCH: return "the call needs more device scratch than GRADLEV_STATIC_SCRATCH_BYTES (use gradlev_scan_fwd with a workspace)";
    default: return "unknown status code";
  }
}

int gradlev_scan_plan(const gradlev_shape* s, gradlev_plan* plan) {
  if (!plan) return GRADLEV_ERR_INVALID;
  if (wide_shape(s)) {
    WideProblem w;
    const int rc = make_wide(s, &w);
    if (rc != GRADLEV_OK) return rc;
    plan->fwd_chunk = plan->bwd_chunk = w.Tp;
    plan->fwd_segment = plan->bwd_segment = w.Tp;
    plan->fwd_nseg = plan->bwd_nseg = 1;
    plan->workspace_bytes = wide_workspace_bytes(w);
    return GRADLEV_OK;
  }
  Plan p;
  const int rc = make_plan(s, &p);
  if (rc != GRADLEV_OK) return rc;
  plan->fwd_chunk = p.fwd.chunk;
  plan->fwd_segment = p.fwd.seg_len;
  plan->fwd_nseg = p.fwd.nseg;
  plan->bwd_chunk = p.bwd.chunk;
  plan->bwd_segment = p.bwd.seg_len;
  plan->bwd_nseg = p.bwd.nseg;
  plan->workspace_bytes = p.ws_fwd > p.ws_bwd ? p.ws_fwd : p.ws_bwd;
  return GRADLEV_OK;
}

int gradlev_scan_workspace_bytes(const gradlev_shape* s, size_t* bytes) {
  if (!bytes) return GRADLEV_ERR_INVALID;
  if (wide_shape(s)) {
    WideProblem w;
    const int rc = make_wide(s, &w);
    if (rc == GRADLEV_OK) *bytes = wide_workspace_bytes(w);
    return rc;
  }
  Plan p;
  const int rc = make_plan(s, &p);
  if (rc != GRADLEV_OK) return rc;
  *bytes = p.ws_fwd > p.ws_bwd ? p.ws_fwd : p.ws_bwd;
  return GRADLEV_OK;
}

}  // extern "C"

namespace gradlev {
namespace {

// Forward with a validated plan; wend (saved segment-end weights) or null.
int scan_fwd_planned(const Plan& p, const float* W0, const void* X, const void* G, const float* eta,
                     float eta_scalar, float* Y, float* wend, void* workspace, size_t workspace_bytes,
                     void* stream) {
  int rc;
  if (!W0 || !X || !G || !Y) return GRADLEV_ERR_INVALID;
  if (!aligned16(W0) || !aligned16(X) || !aligned16(G) || !aligned16(Y) || (eta && !aligned16(eta)))
    return GRADLEV_ERR_ALIGN;
  rc = check_workspace(workspace, workspace_bytes, p.ws_fwd);
  if (rc != GRADLEV_OK) return rc;
  FwdPtrs f{};
  f.W0 = W0;
  f.X = X;
  f.G = G;
  f.eta = eta;
  f.eta_scalar = eta_scalar;
  f.Y = Y;
  f.agg = static_cast<float*>(workspace);
  f.wend = wend;
  f.save_len = p.save_len;
  f.nsave = p.bwd.nseg;
  const hipError_t e = launch_scan_fwd(p.fwd, f, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GRADLEV_OK : GRADLEV_ERR_HIP;
}

// Backward with a validated plan; wend (the forward's saved weights) or null.
int scan_bwd_planned(const Plan& p, const float* W0, const void* X, const void* G, const float* eta,
                     float eta_scalar, const void* dY, const float* wend, float* gtilde, float* dX, float* dG,
                     float* deta, float* dW0, void* workspace, size_t workspace_bytes, void* stream) {
  int rc;
  if (!W0 || !X || !G || !dY) return GRADLEV_ERR_INVALID;
  if (!gtilde && !dX && !dG && !deta && !dW0) return GRADLEV_ERR_INVALID;
  const void* ptrs[] = {W0, X, G, dY, eta, gtilde, dX, dG, deta, dW0};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return GRADLEV_ERR_ALIGN;
  rc = check_workspace(workspace, workspace_bytes, p.ws_bwd);
  if (rc != GRADLEV_OK) return rc;
  char* ws = static_cast<char*>(workspace);
  BwdPtrs b{};
  b.W0 = W0;
  b.X = X;
  b.G = G;
  b.eta = eta;
  b.eta_scalar = eta_scalar;
  b.dY = dY;
  b.gtilde = gtilde;
  b.dX = dX;
  b.dG = dG;
  b.deta = deta;
  b.dW0 = dW0;
  b.aggA = reinterpret_cast<float*>(ws + p.off_aggA);
  b.aggB = reinterpret_cast<float*>(ws + p.off_aggB);
  b.rfin = reinterpret_cast<float*>(ws + p.off_rfin);
  b.wend = wend;
  const hipError_t e = launch_scan_bwd(p.bwd, b, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GRADLEV_OK : GRADLEV_ERR_HIP;
}

}  // namespace
}  // namespace gradlev

extern "C" {

int gradlev_scan_fwd(const gradlev_shape* s, const float* W0, const void* X, const void* G,
                     const float* eta, float eta_scalar, float* Y, void* workspace,
                     size_t workspace_bytes, void* stream) {
  if (wide_shape(s)) {
    const gradlev_gates none{nullptr, 1.f, nullptr};
    return gradlev_scan_fwd_gated(s, &none, W0, X, G, eta, eta_scalar, Y, workspace, workspace_bytes, stream);
  }
  Plan p;
  const int rc = make_plan(s, &p);
  if (rc != GRADLEV_OK) return rc;
  return scan_fwd_planned(p, W0, X, G, eta, eta_scalar, Y, nullptr, workspace, workspace_bytes, stream);
}

int gradlev_scan_fwd_static(const gradlev_shape* s, const float* W0, const void* X, const void* G,
                            const float* eta, float eta_scalar, float* Y, void* stream) {
  // Host validation first (the same checks gradlev_scan_fwd makes), then the
  // scratch lookup, the only HIP call before the launches.
  size_t need = 0;
  const int rc = gradlev_scan_workspace_bytes(s, &need);
  if (rc != GRADLEV_OK) return rc;
  if (!W0 || !X || !G || !Y) return GRADLEV_ERR_INVALID;
  if (!aligned16(W0) || !aligned16(X) || !aligned16(G) || !aligned16(Y) || (eta && !aligned16(eta)))
    return GRADLEV_ERR_ALIGN;
  if (need > GRADLEV_STATIC_SCRATCH_BYTES) return GRADLEV_ERR_SCRATCH;
  void* ws = nullptr;
  const int rs = static_scratch(&ws);
  if (rs != GRADLEV_OK) return rs;
  return gradlev_scan_fwd(s, W0, X, G, eta, eta_scalar, Y, ws, GRADLEV_STATIC_SCRATCH_BYTES, stream);
}

int gradlev_scan_bwd(const gradlev_shape* s, const float* W0, const void* X, const void* G,
                     const float* eta, float eta_scalar, const void* dY, float* gtilde,
                     float* dX, float* dG, float* deta, float* dW0, void* workspace,
                     size_t workspace_bytes, void* stream) {
  if (wide_shape(s)) {
    const gradlev_gates none{nullptr, 1.f, nullptr};
    return gradlev_scan_bwd_gated(s, &none, W0, X, G, eta, eta_scalar, dY, gtilde, dX, dG, deta, nullptr, dW0,
                                  workspace, workspace_bytes, stream);
  }
  Plan p;
  const int rc = make_plan(s, &p);
  if (rc != GRADLEV_OK) return rc;
  return scan_bwd_planned(p, W0, X, G, eta, eta_scalar, dY, nullptr, gtilde, dX, dG, deta, dW0, workspace,
                          workspace_bytes, stream);
}

int gradlev_scan_saved_bytes(const gradlev_shape* s, size_t* saved_bytes, size_t* workspace_bytes) {
  if (!saved_bytes || !workspace_bytes) return GRADLEV_ERR_INVALID;
  if (wide_shape(s)) return s && s->B >= 1 ? GRADLEV_ERR_UNSUPPORTED : GRADLEV_ERR_INVALID;
  Plan p;
  size_t sb = 0;
  const int rc = make_saved_plan(s, &p, &sb);
  if (rc != GRADLEV_OK) return rc;
  *saved_bytes = sb;
  *workspace_bytes = p.ws_fwd > p.ws_bwd ? p.ws_fwd : p.ws_bwd;
  return GRADLEV_OK;
}

int gradlev_scan_fwd_save(const gradlev_shape* s, const float* W0, const void* X, const void* G,
                          const float* eta, float eta_scalar, float* Y, float* saved, size_t saved_bytes,
                          void* workspace, size_t workspace_bytes, void* stream) {
  if (wide_shape(s)) return s && s->B >= 1 ? GRADLEV_ERR_UNSUPPORTED : GRADLEV_ERR_INVALID;
  Plan p;
  size_t need = 0;
  const int rc = make_saved_plan(s, &p, &need);
  if (rc != GRADLEV_OK) return rc;
  if (!saved) return GRADLEV_ERR_INVALID;
  if (!aligned16(saved)) return GRADLEV_ERR_ALIGN;
  if (saved_bytes < need) return GRADLEV_ERR_WORKSPACE;
  return scan_fwd_planned(p, W0, X, G, eta, eta_scalar, Y, saved, workspace, workspace_bytes, stream);
}

int gradlev_scan_bwd_saved(const gradlev_shape* s, const float* W0, const void* X, const void* G,
                           const float* eta, float eta_scalar, const void* dY, const float* saved,
                           size_t saved_bytes, float* gtilde, float* dX, float* dG, float* deta, float* dW0,
                           void* workspace, size_t workspace_bytes, void* stream) {
  if (wide_shape(s)) return s && s->B >= 1 ? GRADLEV_ERR_UNSUPPORTED : GRADLEV_ERR_INVALID;
  Plan p;
  size_t need = 0;
  const int rc = make_saved_plan(s, &p, &need);
  if (rc != GRADLEV_OK) return rc;
  if (!saved) return GRADLEV_ERR_INVALID;
  if (!aligned16(saved)) return GRADLEV_ERR_ALIGN;
  if (saved_bytes < need) return GRADLEV_ERR_WORKSPACE;
  return scan_bwd_planned(p, W0, X, G, eta, eta_scalar, dY, saved, gtilde, dX, dG, deta, dW0, workspace,
                          workspace_bytes, stream);
}

int gradlev_scan_reset_saved_bytes(const gradlev_shape* s, size_t* saved_bytes, size_t* workspace_bytes) {
  if (!saved_bytes || !workspace_bytes) return GRADLEV_ERR_INVALID;
  ResetPlan r;
  const int rc = make_reset_plan(s, &r);
  if (rc != GRADLEV_OK) return rc;
  *saved_bytes = r.saved_bytes;
  *workspace_bytes = r.ws;
  return GRADLEV_OK;
}

int gradlev_scan_fwd_reset_save(const gradlev_shape* s, const float* W0, const void* X, const void* G,
                                const float* eta, float eta_scalar, const uint8_t* reset, float* Y, float* saved,
                                size_t saved_bytes, void* workspace, size_t workspace_bytes, void* stream) {
  ResetPlan r;
  int rc = make_reset_plan(s, &r);
  if (rc != GRADLEV_OK) return rc;
  if (!W0 || !X || !G || !Y || !saved) return GRADLEV_ERR_INVALID;
  if (!aligned16(W0) || !aligned16(X) || !aligned16(G) || !aligned16(Y) || !aligned16(saved) ||
      (eta && !aligned16(eta)))
    return GRADLEV_ERR_ALIGN;
  if (saved_bytes < r.saved_bytes) return GRADLEV_ERR_WORKSPACE;
  rc = check_workspace(workspace, workspace_bytes, r.ws);
  if (rc != GRADLEV_OK) return rc;
  FwdPtrs f{};
  f.W0 = W0;
  f.X = X;
  f.G = G;
  f.eta = eta;
  f.eta_scalar = eta_scalar;
  f.Y = Y;
  f.agg = static_cast<float*>(workspace);
  f.wend = saved;
  f.save_len = r.p.save_len;
  f.nsave = r.p.bwd.nseg;
  f.reset = reset;
  f.cstate = reinterpret_cast<float*>(reinterpret_cast<char*>(saved) + r.off_cstate);
  f.resets = true;
  f.segreset = reinterpret_cast<int*>(static_cast<char*>(workspace) + r.off_seg);
  const hipError_t e = launch_scan_fwd(r.p.fwd, f, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GRADLEV_OK : GRADLEV_ERR_HIP;
}

int gradlev_scan_bwd_reset_saved(const gradlev_shape* s, const float* W0, const void* X, const void* G,
                                 const float* eta, float eta_scalar, const void* dY, const uint8_t* reset,
                                 const float* saved, size_t saved_bytes, float* gtilde, float* dX, float* dG,
                                 float* deta, float* dW0, void* workspace, size_t workspace_bytes, void* stream) {
  ResetPlan r;
  int rc = make_reset_plan(s, &r);
  if (rc != GRADLEV_OK) return rc;
  if (!W0 || !X || !G || !dY || !saved) return GRADLEV_ERR_INVALID;
  if (!gtilde && !dX && !dG && !deta && !dW0) return GRADLEV_ERR_INVALID;
  const void* ptrs[] = {W0, X, G, dY, eta, saved, gtilde, dX, dG, deta, dW0};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return GRADLEV_ERR_ALIGN;
  if (saved_bytes < r.saved_bytes) return GRADLEV_ERR_WORKSPACE;
  rc = check_workspace(workspace, workspace_bytes, r.ws);
  if (rc != GRADLEV_OK) return rc;
  char* ws = static_cast<char*>(workspace);
  BwdPtrs b{};
  b.W0 = W0;
  b.X = X;
  b.G = G;
  b.eta = eta;
  b.eta_scalar = eta_scalar;
  b.dY = dY;
  b.gtilde = gtilde;
  b.dX = dX;
  b.dG = dG;
  b.deta = deta;
  b.dW0 = dW0;
  b.aggB = reinterpret_cast<float*>(ws);
  b.aggF = reinterpret_cast<float*>(ws + r.off_aggF);
  b.wend = saved;
  b.reset = reset;
  b.cstate = reinterpret_cast<const float*>(reinterpret_cast<const char*>(saved) + r.off_cstate);
  b.resets = true;
  b.segreset = reinterpret_cast<int*>(ws + r.off_seg);
  const hipError_t e = launch_scan_bwd(r.p.bwd, b, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GRADLEV_OK : GRADLEV_ERR_HIP;
}

int gradlev_scan_gated_workspace_bytes(const gradlev_shape* s, size_t* bytes) {
  if (!bytes) return GRADLEV_ERR_INVALID;
  if (wide_shape(s)) return gradlev_scan_workspace_bytes(s, bytes);
  GatedPlan p;
  const int rc = make_gated_plan(s, &p);
  if (rc != GRADLEV_OK) return rc;
  *bytes = p.ws_fwd > p.ws_bwd ? p.ws_fwd : p.ws_bwd;
  return GRADLEV_OK;
}

int gradlev_scan_fwd_gated(const gradlev_shape* s, const gradlev_gates* gates, const float* W0,
                           const void* X, const void* G, const float* eta, float eta_scalar, float* Y,
                           void* workspace, size_t workspace_bytes, void* stream) {
  if (wide_shape(s)) {
    WideProblem w;
    int rc = make_wide(s, &w);
    if (rc != GRADLEV_OK) return rc;
    rc = check_gates(gates);
    if (rc != GRADLEV_OK) return rc;
    if (!W0 || !X || !G || !Y) return GRADLEV_ERR_INVALID;
    if (!aligned16(W0) || !aligned16(X) || !aligned16(G) || !aligned16(Y) || (eta && !aligned16(eta)))
      return GRADLEV_ERR_ALIGN;
    rc = check_workspace(workspace, workspace_bytes, wide_workspace_bytes(w));
    if (rc != GRADLEV_OK) return rc;
    w.fmode = wide_fmode(gates);
    WidePtrs f = wide_ptrs(gates, W0, X, G, eta, eta_scalar, 1.f, workspace);
    f.Y = Y;
    return launch_wide_fwd(w, f, static_cast<hipStream_t>(stream)) == hipSuccess ? GRADLEV_OK : GRADLEV_ERR_HIP;
  }
  GatedPlan p;
  const int rc = make_gated_plan(s, &p);
  if (rc != GRADLEV_OK) return rc;
  return gated_fwd_planned(s, p, gates, W0, X, G, eta, eta_scalar, Y, nullptr, workspace, workspace_bytes, stream);
}

}  // extern "C"

namespace gradlev {
namespace {

// Gated forward with a validated plan; states (saved chunk-start states) or null.
int gated_fwd_planned(const gradlev_shape* s, const GatedPlan& p, const gradlev_gates* gates, const float* W0,
                      const void* X, const void* G, const float* eta, float eta_scalar, float* Y, float* states,
                      void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_gates(gates);
  if (rc != GRADLEV_OK) return rc;
  if (!W0 || !X || !G || !Y) return GRADLEV_ERR_INVALID;
  if (!aligned16(W0) || !aligned16(X) || !aligned16(G) || !aligned16(Y) || (eta && !aligned16(eta)))
    return GRADLEV_ERR_ALIGN;
  rc = check_workspace(workspace, workspace_bytes, p.ws_fwd);
  if (rc != GRADLEV_OK) return rc;
  GatedPtrs f{};
  f.W0 = W0;
  f.X = X;
  f.G = G;
  f.eta = eta;
  f.eta_scalar = eta_scalar;
  f.eta_mul = 1.f;
  f.alpha = gates->alpha;
  f.alpha_scalar = gates->alpha_scalar;
  f.reset = gates->reset;
  f.Y = Y;
  if (p.fwd.nseg > 1) {
    char* ws = static_cast<char*>(workspace);
    const size_t nf = (size_t)(s->B * s->H) * p.fwd.nseg;
    f.aggA = reinterpret_cast<float*>(ws);
    f.aggD = reinterpret_cast<float*>(ws + round_up(nf * (size_t)s->d_out * s->d_in * sizeof(float), 256));
  }
  f.states = states;
  const hipError_t e = launch_scan_fwd_gated(p.fwd, f, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GRADLEV_OK : GRADLEV_ERR_HIP;
}

// Gated backward with a validated plan; states: the saving forward's states,
// or null (then the workspace's state region, filled by the state pass).
int gated_bwd_planned(const GatedPlan& p, const gradlev_gates* gates, const float* W0, const void* X,
                      const void* G, const float* eta, float eta_scalar, const void* dY, const float* states,
                      float* gtilde, float* dX, float* dG, float* deta, float* dalpha, float* dW0, void* workspace,
                      size_t workspace_bytes, void* stream) {
  int rc = check_gates(gates);
  if (rc != GRADLEV_OK) return rc;
  if (!W0 || !X || !G || !dY) return GRADLEV_ERR_INVALID;
  if (!gtilde && !dX && !dG && !deta && !dalpha && !dW0) return GRADLEV_ERR_INVALID;
  const void* ptrs[] = {W0, X, G, dY, eta, gtilde, dX, dG, deta, dalpha, dW0};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return GRADLEV_ERR_ALIGN;
  rc = check_workspace(workspace, workspace_bytes, p.ws_bwd);
  if (rc != GRADLEV_OK) return rc;
  char* ws = static_cast<char*>(workspace);
  GatedPtrs b{};
  b.W0 = W0;
  b.X = X;
  b.G = G;
  b.dY = dY;
  b.eta = eta;
  b.eta_scalar = eta_scalar;
  b.eta_mul = 1.f;
  b.alpha = gates->alpha;
  b.alpha_scalar = gates->alpha_scalar;
  b.reset = gates->reset;
  b.gtilde = gtilde;
  b.dX = dX;
  b.dG = dG;
  b.deta = deta;
  b.dalpha = dalpha;
  b.dW0 = dW0;
  b.aggA = reinterpret_cast<float*>(ws + p.off_A);
  b.aggB = reinterpret_cast<float*>(ws + p.off_B);
  b.aggBu = reinterpret_cast<float*>(ws + p.off_Bu);
  b.aggD = reinterpret_cast<float*>(ws + p.off_D);
  b.states = states ? const_cast<float*>(states) : reinterpret_cast<float*>(ws + p.off_S);
  b.saved_states = states != nullptr;
  const hipError_t e = launch_scan_bwd_gated(p.bwd, b, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GRADLEV_OK : GRADLEV_ERR_HIP;
}

}  // namespace
}  // namespace gradlev

extern "C" {

int gradlev_scan_bwd_gated(const gradlev_shape* s, const gradlev_gates* gates, const float* W0,
                           const void* X, const void* G, const float* eta, float eta_scalar,
                           const void* dY, float* gtilde, float* dX, float* dG, float* deta,
                           float* dalpha, float* dW0, void* workspace, size_t workspace_bytes,
                           void* stream) {
  if (wide_shape(s)) {
    // Wide maps: the parallel form's backward (transpose read, write-side
    // terms, gate gradients and dW0), each output when requested.
    WideProblem w;
    int rc = make_wide(s, &w);
    if (rc != GRADLEV_OK) return rc;
    rc = check_gates(gates);
    if (rc != GRADLEV_OK) return rc;
    if (!W0 || !X || !G || !dY) return GRADLEV_ERR_INVALID;
    if (!gtilde && !dX && !dG && !deta && !dalpha && !dW0) return GRADLEV_ERR_INVALID;
    const void* ptrs[] = {W0, X, G, dY, eta, gtilde, dX, dG, deta, dalpha, dW0};
    for (const void* q : ptrs)
      if (q && !aligned16(q)) return GRADLEV_ERR_ALIGN;
    rc = check_workspace(workspace, workspace_bytes, wide_workspace_bytes(w));
    if (rc != GRADLEV_OK) return rc;
    w.fmode = wide_fmode(gates);
    WidePtrs f = wide_ptrs(gates, W0, X, G, eta, eta_scalar, 1.f, workspace);
    f.dY = dY;
    f.gtilde = gtilde;
    f.dX = dX;
    f.dG = dG;
    f.deta = deta;
    f.dalpha = dalpha;
    f.dW0 = dW0;
    return launch_wide_read(w, f, static_cast<hipStream_t>(stream)) == hipSuccess ? GRADLEV_OK : GRADLEV_ERR_HIP;
  }
  GatedPlan p;
  const int rc = make_gated_plan(s, &p);
  if (rc != GRADLEV_OK) return rc;
  return gated_bwd_planned(p, gates, W0, X, G, eta, eta_scalar, dY, nullptr, gtilde, dX, dG, deta, dalpha, dW0,
                           workspace, workspace_bytes, stream);
}

int gradlev_scan_gated_saved_bytes(const gradlev_shape* s, size_t* saved_bytes, size_t* workspace_bytes) {
  if (!saved_bytes || !workspace_bytes) return GRADLEV_ERR_INVALID;
  if (wide_shape(s)) return s && s->B >= 1 ? GRADLEV_ERR_UNSUPPORTED : GRADLEV_ERR_INVALID;
  GatedPlan p;
  size_t sb = 0;
  const int rc = make_gated_saved_plan(s, &p, &sb);
  if (rc != GRADLEV_OK) return rc;
  *saved_bytes = sb;
  *workspace_bytes = p.ws_fwd > p.ws_bwd ? p.ws_fwd : p.ws_bwd;
  return GRADLEV_OK;
}

int gradlev_scan_fwd_gated_save(const gradlev_shape* s, const gradlev_gates* gates, const float* W0,
                                const void* X, const void* G, const float* eta, float eta_scalar, float* Y,
                                float* saved, size_t saved_bytes, void* workspace, size_t workspace_bytes,
                                void* stream) {
  if (wide_shape(s)) return s && s->B >= 1 ? GRADLEV_ERR_UNSUPPORTED : GRADLEV_ERR_INVALID;
  GatedPlan p;
  size_t need = 0;
  const int rc = make_gated_saved_plan(s, &p, &need);
  if (rc != GRADLEV_OK) return rc;
  if (!saved) return GRADLEV_ERR_INVALID;
  if (!aligned16(saved)) return GRADLEV_ERR_ALIGN;
  if (saved_bytes < need) return GRADLEV_ERR_WORKSPACE;
  return gated_fwd_planned(s, p, gates, W0, X, G, eta, eta_scalar, Y, saved, workspace, workspace_bytes, stream);
}

int gradlev_scan_bwd_gated_saved(const gradlev_shape* s, const gradlev_gates* gates, const float* W0,
                                 const void* X, const void* G, const float* eta, float eta_scalar, const void* dY,
                                 const float* saved, size_t saved_bytes, float* gtilde, float* dX, float* dG,
                                 float* deta, float* dalpha, float* dW0, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  if (wide_shape(s)) return s && s->B >= 1 ? GRADLEV_ERR_UNSUPPORTED : GRADLEV_ERR_INVALID;
  GatedPlan p;
  size_t need = 0;
  const int rc = make_gated_saved_plan(s, &p, &need);
  if (rc != GRADLEV_OK) return rc;
  if (!saved) return GRADLEV_ERR_INVALID;
  if (!aligned16(saved)) return GRADLEV_ERR_ALIGN;
  if (saved_bytes < need) return GRADLEV_ERR_WORKSPACE;
  return gated_bwd_planned(p, gates, W0, X, G, eta, eta_scalar, dY, saved, gtilde, dX, dG, deta, dalpha, dW0,
                           workspace, workspace_bytes, stream);
}

int gradlev_mlp_workspace_bytes(const gradlev_mlp_shape* s, size_t* bytes) {
  if (!bytes) return GRADLEV_ERR_INVALID;
  MlpPlan p;
  const int rc = make_mlp_plan(s, &p);
  if (rc != GRADLEV_OK) return rc;
  *bytes = p.total;
  return GRADLEV_OK;
}

int gradlev_mlp_fwd(const gradlev_mlp_shape* s, const gradlev_gates* gates, const float* W1_0,
                    const float* W2_0, const void* X, const void* Gz, const void* Gy, const float* mu,
                    float mu_scalar, float* Z, void* Hid, float* Y, void* workspace,
                    size_t workspace_bytes, void* stream) {
  MlpPlan p;
  int rc = make_mlp_plan(s, &p);
  if (rc != GRADLEV_OK) return rc;
  rc = check_gates(gates);
  if (rc != GRADLEV_OK) return rc;
  if (!W1_0 || !W2_0 || !X || !Gz || !Gy || !Z || !Hid || !Y) return GRADLEV_ERR_INVALID;
  const void* ptrs[] = {W1_0, W2_0, X, Gz, Gy, mu, Z, Hid, Y};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return GRADLEV_ERR_ALIGN;
  rc = check_workspace(workspace, workspace_bytes, p.total);
  if (rc != GRADLEV_OK) return rc;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t BH = s->B * s->H;
  const int fm = wide_fmode(gates);
  if (p.wide1) {
    WidePtrs f1 = wide_ptrs(gates, W1_0, X, Gz, mu, mu_scalar, 1.f / (float)s->d_in, workspace);
    f1.Y = Z;
    p.w1.fmode = fm;
    if (launch_wide_fwd(p.w1, f1, st) != hipSuccess) return GRADLEV_ERR_HIP;
  } else {
    GatedPtrs f1 = gated_ptrs(p.p1, gates, W1_0, X, Gz, mu, mu_scalar, 1.f / (float)s->d_in, workspace, false, BH);
    f1.Y = Z;
    if (launch_scan_fwd_gated(p.p1.fwd, f1, st) != hipSuccess) return GRADLEV_ERR_HIP;
  }
  if (launch_act_fwd(s->in_dtype == GRADLEV_BF16, Z, Hid, BH * s->T * s->hidden, s->act, st) != hipSuccess)
    return GRADLEV_ERR_HIP;
  if (p.wide2) {
    WidePtrs f2 = wide_ptrs(gates, W2_0, Hid, Gy, mu, mu_scalar, 1.f / (float)s->hidden, workspace);
    f2.Y = Y;
    p.w2.fmode = fm;
    if (launch_wide_fwd(p.w2, f2, st) != hipSuccess) return GRADLEV_ERR_HIP;
  } else {
    GatedPtrs f2 = gated_ptrs(p.p2, gates, W2_0, Hid, Gy, mu, mu_scalar, 1.f / (float)s->hidden, workspace, false, BH);
    f2.Y = Y;
    if (launch_scan_fwd_gated(p.p2.fwd, f2, st) != hipSuccess) return GRADLEV_ERR_HIP;
  }
  return GRADLEV_OK;
}

int gradlev_mlp_reverse(const gradlev_mlp_shape* s, const gradlev_gates* gates, const float* W1_0,
                        const float* W2_0, const void* X, const void* Gz, const void* Gy, const float* mu,
                        float mu_scalar, const float* Z, const void* Hid, const void* gY, float* gZ,
                        float* gX, float* dMu, float* dAlpha, float* dW1_0, float* dW2_0, void* workspace,
                        size_t workspace_bytes, void* stream) {
  MlpPlan p;
  int rc = make_mlp_plan(s, &p);
  if (rc != GRADLEV_OK) return rc;
  rc = check_gates(gates);
  if (rc != GRADLEV_OK) return rc;
  if (!W1_0 || !W2_0 || !X || !Gz || !Gy || !Z || !Hid || !gY || !gZ) return GRADLEV_ERR_INVALID;
  const void* ptrs[] = {W1_0, W2_0, X, Gz, Gy, mu, Z, Hid, gY, gZ, gX, dMu, dAlpha, dW1_0, dW2_0};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return GRADLEV_ERR_ALIGN;
  rc = check_workspace(workspace, workspace_bytes, p.total);
  if (rc != GRADLEV_OK) return rc;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t BH = s->B * s->H, n = BH * s->T;
  char* ws = static_cast<char*>(workspace);
  const size_t gstride = round_up((size_t)n * 4, 256);
  float* de1 = reinterpret_cast<float*>(ws + p.off_g);
  float* de2 = reinterpret_cast<float*>(ws + p.off_g + gstride);
  float* da1 = reinterpret_cast<float*>(ws + p.off_g + 2 * gstride);
  // The second scan with the output costate: its transpose read g_h (written
  // into gZ), and with the training gradients its deta, dalpha and dW0.
  const int fm = wide_fmode(gates);
  if (p.wide2) {
    WidePtrs b2 = wide_ptrs(gates, W2_0, Hid, Gy, mu, mu_scalar, 1.f / (float)s->hidden, workspace);
    b2.dY = gY;
    b2.gtilde = gZ;
    b2.deta = dMu ? de2 : nullptr;
    b2.dalpha = dAlpha;
    b2.dW0 = dW2_0;
    p.w2.fmode = fm;
    if (launch_wide_read(p.w2, b2, st) != hipSuccess) return GRADLEV_ERR_HIP;
  } else {
    GatedPtrs b2 = gated_ptrs(p.p2, gates, W2_0, Hid, Gy, mu, mu_scalar, 1.f / (float)s->hidden, workspace, true, BH);
    b2.dY = gY;
    b2.gtilde = gZ;
    b2.deta = dMu ? de2 : nullptr;
    b2.dalpha = dAlpha;
    b2.dW0 = dW2_0;
    if (launch_scan_bwd_gated(p.p2.bwd, b2, st) != hipSuccess) return GRADLEV_ERR_HIP;
  }
  // g_z = sigma'(z) g_h, and its in_dtype copy for the first scan's queries.
  const bool first = gX || dMu || dAlpha || dW1_0;
  void* q = first ? static_cast<void*>(ws + p.off_q) : nullptr;
  if (launch_act_bwd(s->in_dtype == GRADLEV_BF16, Z, gZ, q, BH * s->T * s->hidden, s->act, st) != hipSuccess)
    return GRADLEV_ERR_HIP;
  if (first && p.wide1) {
    WidePtrs b1 = wide_ptrs(gates, W1_0, X, Gz, mu, mu_scalar, 1.f / (float)s->d_in, workspace);
    b1.dY = q;
    b1.gtilde = gX;
    b1.deta = dMu ? de1 : nullptr;
    b1.dalpha = dAlpha ? da1 : nullptr;
    b1.dW0 = dW1_0;
    p.w1.fmode = fm;
    if (launch_wide_read(p.w1, b1, st) != hipSuccess) return GRADLEV_ERR_HIP;
  } else if (first) {
    GatedPtrs b1 = gated_ptrs(p.p1, gates, W1_0, X, Gz, mu, mu_scalar, 1.f / (float)s->d_in, workspace, true, BH);
    b1.dY = q;
    b1.gtilde = gX;
    b1.deta = dMu ? de1 : nullptr;
    b1.dalpha = dAlpha ? da1 : nullptr;
    b1.dW0 = dW1_0;
    if (launch_scan_bwd_gated(p.p1.bwd, b1, st) != hipSuccess) return GRADLEV_ERR_HIP;
  }
  if ((dMu || dAlpha) &&
      launch_mlp_gate_grads(de1, de2, 1.f / (float)s->d_in, 1.f / (float)s->hidden, dMu, da1, dAlpha, n, st) !=
          hipSuccess)
    return GRADLEV_ERR_HIP;
  return GRADLEV_OK;
}

int gradlev_decode_step_gated(int64_t S, int64_t H, int64_t d_in, int64_t d_out, float* W,
                              const float* W0, const float* x, const float* g, const float* eta,
                              float eta_scalar, const float* alpha, float alpha_scalar,
                              const uint8_t* reset, float* y, void* stream) {
  if (S < 1 || H < 1 || d_in < 1 || d_out < 1) return GRADLEV_ERR_INVALID;
  if (!W || !W0 || !x || !g || !y) return GRADLEV_ERR_INVALID;
  if (!decode_shape_ok(S, H, d_in, d_out)) return GRADLEV_ERR_UNSUPPORTED;
  if (!aligned16(W) || !aligned16(W0) || !aligned16(x) || !aligned16(g) || !aligned16(y) ||
      (eta && !aligned16(eta)) || (alpha && !aligned16(alpha)))
    return GRADLEV_ERR_ALIGN;
  DecodeGates gt{W0, alpha, alpha_scalar, reset};
  const hipError_t e = launch_decode(S, H, (int)d_in, (int)d_out, W, x, g, eta, eta_scalar, y,
                                     static_cast<hipStream_t>(stream), &gt);
  return e == hipSuccess ? GRADLEV_OK : GRADLEV_ERR_HIP;
}

int gradlev_decode_step(int64_t S, int64_t H, int64_t d_in, int64_t d_out, float* W, const float* x,
                        const float* g, const float* eta, float eta_scalar, float* y, void* stream) {
  if (S < 1 || H < 1 || d_in < 1 || d_out < 1) return GRADLEV_ERR_INVALID;
  if (!W || !x || !g || !y) return GRADLEV_ERR_INVALID;
  if (!decode_shape_ok(S, H, d_in, d_out)) return GRADLEV_ERR_UNSUPPORTED;
  if (!aligned16(W) || !aligned16(x) || !aligned16(g) || !aligned16(y) || (eta && !aligned16(eta)))
    return GRADLEV_ERR_ALIGN;
  const hipError_t e = launch_decode(S, H, (int)d_in, (int)d_out, W, x, g, eta, eta_scalar, y,
                                     static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GRADLEV_OK : GRADLEV_ERR_HIP;
}

}  // extern "C"
