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
// the chunk, V = diag(eta) G, M the causal mask, E = M o (dY V^T):
//   gtilde = dY W_n - E X
//   U      = -(X R_n^T + (M o X X^T)^T dY)             dG = diag(eta) U
//   dXw    = -(V R_n + E^T X)                           dX = gtilde + dXw
//   W_n    = W_{n+1} + V^T X     (the state is un-written chunk by chunk)
//   R_{n-1}= R_n + dY^T X
// A workgroup walks its segment's chunks from last to first, carrying R in
// reverse time and un-writing W from the state at the segment's end (both
// summed in its prologue from the aggregate pass).  Waves own column blocks of
// W and R in registers; R is also published each chunk to LDS (transposed,
// split into bf16 hi + lo) for the products contracted over d, so no second
// register copy is needed.
#include "scan_common.hpp"

namespace gradlev {

struct BArgs {
  const float* W0;
  const void* X;
  const void* G;
  const void* dY;
  const float* eta;
  float eta_scalar;
  int64_t BH, H, T, seg_len, nseg;
  float* gtilde;
  float* dX;
  float* dG;
  float* deta;
  const float* aggA;  // [BH][nseg][d][m]: per-segment write aggregates A_k, transposed
  const float* aggB;  // [BH][nseg][d][m]: per-segment dY x^T aggregates B_k (k >= 1), or null
  float* rfin;        // [BH][m][d]: full-sequence dY x^T (written by segment 0), or null
  const float* wend;  // [BH][nseg][m][d]: the forward's segment-end weights, or null (then W_0 - sum A)
  const uint8_t* reset;  // [B][T] document starts (RST kernels)
  const float* cstate;   // [BH][ceil(T/C)][d][m]: chunk-start states of the chunks holding a reset, transposed
  const int* segreset;   // RST, or null: each work item's first document start (-1: none), from the aggregate pass
};

// Output modes compiled separately so that no accumulator crosses a runtime
// branch: kOutFull computes every backward term (stores are skipped for NULL
// outputs); kOutRead computes only the read-side gtilde.
enum OutMode { kOutFull = 0, kOutRead = 1 };

// LDS bytes of the main backward kernel (without the shared score tiles) and
// whether the split score tiles fit beside it.
static constexpr int lds_bytes_bwd(int bf16, int d, int m, int C, int etav) {
  const int es = bf16 ? 2 : 4;
  const int v = etav ? (bf16 ? 2 : 1) * C * m : 0;
  const int r = (bf16 ? 2 : 1) * d * m;
  return es * (C * d + 2 * C * m + C * C + v + r) + 4 * C + 4 * 4 * (m / 16) * C;  // last: deta partials, at most
}
static constexpr bool s_shared_fits(bool bf16, int d, int m, int C, bool etav) {
  return lds_bytes_bwd(bf16, d, m, C, etav) + (bf16 ? 2 : 1) * C * C * (bf16 ? 2 : 4) <= 160 * 1024;
}

// RST (document resets at unit retention, with the forward's saved states;
// exclusive reads, 64 x 64 maps, 64-token chunks): intra-chunk tiles pair
// tokens of one document; a chunk holding a reset takes its start state from
// cstate (writes before a reset cannot be taken back), its rows at or after
// the first reset read W_0, only its last document's tokens see the suffix
// R_n, and the suffix passed to the previous chunk keeps the tokens before
// the first reset only.
template <class OP, int D, int M, int C, bool INCL, bool ETAV, int OUT, bool RST = false>
__global__ void __launch_bounds__(cmax(D, M) / 16 * 64, 128 / cmax(D, M))
bwd_main_kernel(const BArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int NW = cmax(D, M) / 16, NT = NW * 64;
  constexpr int TB = C / 16, JB = D / 16, IB = M / 16;
  constexpr bool SPLITV = ETAV && OP::kSplit == 2;
  constexpr bool FULL = OUT == kOutFull;
  // Paired column blocks (64x64 maps, 64-token chunks): waves 2p and 2p+1
  // both keep W's column blocks 2p and 2p+1 and split the chunk's token
  // blocks between them, so that each wave holds adjacent column blocks of
  // the same rows and writes gtilde, dX and dG as whole 128-byte rows
  // (pair_rows).  The pair's duplicated un-write costs a few matrix-core
  // steps; the stores run at the full-line rate.
  constexpr bool PAIR = D == 64 && M == 64 && C == 64;
  constexpr int NWB = PAIR ? 2 : 1;   // W column blocks (and U row blocks) per wave
  constexpr int TBW = PAIR ? 2 : TB;  // token blocks per wave in the output phases
  __shared__ E Xs[C * D];                  // X[t][j]
  __shared__ E Gs[C * M];                  // G[t][i]
  __shared__ E Ds[C * M];                  // dY[t][i]
  __shared__ E Es[C * C];                  // E[t][s] = eta_s dY_t . g_s (s before t)
  __shared__ E Vh[ETAV ? C * M : 1];       // (eta G)[t][i] hi (per-token eta)
  __shared__ E Vl[SPLITV ? C * M : 1];     // (eta G)[t][i] lo
  __shared__ E Rh[FULL ? D * M : 1];       // R^T[j][i] hi
  __shared__ E Rl[FULL && OP::kSplit == 2 ? D * M : 1];  // R^T[j][i] lo
  // Intra-chunk scores S[t][s] = x_t . x_s (masked), split hi + lo, built once
  // per chunk and shared by the waves (when they fit the LDS budget; with
  // per-token eta the extra live tiles would cost the second workgroup per CU).
  constexpr bool SSH = FULL && !ETAV && s_shared_fits(OP::kSplit == 2, D, M, C, ETAV);
  __shared__ E Sh[SSH ? C * C : 1];
  __shared__ E Sl[SSH && OP::kSplit == 2 ? C * C : 1];
  __shared__ __attribute__((aligned(16))) float et[C];
  __shared__ float dpart[PAIR ? 2 : IB][4][C];  // deta partial sums per wave (pair) and lane group
  static_assert(!RST || (C == 64 && D == 64 && M == 64 && !INCL), "resets: exclusive 64 x 64 maps, 64-token chunks");
  __shared__ int red[1];

  int64_t bh, seg;
  if (!map_block(a.BH, a.nseg, bh, seg)) return;
  const int tid = threadIdx.x, lane = tid & 63, c = lane & 15, q = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: block indices stay scalar
  // Column block of W (and row block of U) e of this wave.
  auto blk = [&](int e) { return PAIR ? 2 * (w >> 1) + e : w; };
  const int64_t T = a.T;
  const int64_t t_begin = seg * a.seg_len;
  const int64_t t_end = t_begin + a.seg_len < T ? t_begin + a.seg_len : T;
  const rsrc_t X = make_rsrc(static_cast<const E*>(a.X) + bh * T * D, (uint32_t)(T * D * sizeof(E)));
  const rsrc_t G = make_rsrc(static_cast<const E*>(a.G) + bh * T * M, (uint32_t)(T * M * sizeof(E)));
  const rsrc_t Dy = make_rsrc(static_cast<const E*>(a.dY) + bh * T * M, (uint32_t)(T * M * sizeof(E)));
  // Outputs: rows past T are dropped by the resource bounds.
  const rsrc_t Og = make_rsrc(a.gtilde ? a.gtilde + bh * T * D : nullptr, a.gtilde ? (uint32_t)(T * D * 4) : 0u);
  const rsrc_t Ox = make_rsrc(a.dX ? a.dX + bh * T * D : nullptr, a.dX ? (uint32_t)(T * D * 4) : 0u);
  const rsrc_t Od = make_rsrc(a.dG ? a.dG + bh * T * M : nullptr, a.dG ? (uint32_t)(T * M * 4) : 0u);
  const rsrc_t Oe = make_rsrc(a.deta ? a.deta + bh * T : nullptr, a.deta ? (uint32_t)(T * 4) : 0u);
  const rsrc_t none = make_rsrc(nullptr, 0u);  // every access out of range
  const int64_t nch = (t_end - t_begin + C - 1) / C;

  // Register staging, DEPTH chunks ahead (chunks are visited last to first).
  // Two chunks ahead keep more bytes in flight, which pays once the inputs
  // come from HBM rather than the Infinity Cache.  fp32 tiles take twice the
  // registers, and the full backward of maps with a 128-wide side keeps more
  // accumulators: those stage one chunk ahead, which keeps them free of spills.
  constexpr int DEPTH = (OP::kSplit == 2 && (!FULL || (D == 64 && M == 64 && !PAIR))) ? 2 : 1;
  Tile4<OP, C, D, NT> xa, xb;
  Tile4<OP, C, M, NT> ga, gb, da, db;
  EtaReg<ETAV> ea, eb;
  RstReg<RST> ra, rb;
  const rsrc_t Et = eta_rsrc(a.eta, bh, T);
  const rsrc_t Rrow = reset_rsrc(RST ? a.reset : nullptr, bh / a.H, T);
  const float* W0h = a.W0 + (bh % a.H) * M * D;  // this head's W_0 (rows after a reset read it)
  typedef Tile4<OP, C, D, NT> TX;
  typedef Tile4<OP, C, M, NT> TM;
  auto fetch = [&](TX& xr, TM& gr, TM& dr, EtaReg<ETAV>& er, RstReg<RST>& rr, int64_t n) {
    const int64_t t0 = t_begin + n * C;
    er.load(Et, n >= 0 ? (uint32_t)(t0 * 4) : kOOB, tid, C);
    rr.load(Rrow, t0, n >= 0, tid, C);
    xr.load(X, n >= 0 ? (uint32_t)(t0 * D * sizeof(E)) : kOOB, tid);
    gr.load(G, n >= 0 ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
    dr.load(Dy, n >= 0 ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
  };
  // With resets the suffix at the segment end holds the dY x^T of the tokens
  // up to the next document start: none if it is t_end itself, else the
  // (pre-reset) aggregates up to that document start's segment.
  fetch(xa, ga, da, ea, ra, nch - 1);
  if (DEPTH == 2) fetch(xb, gb, db, eb, rb, nch - 2);
  int64_t j_last = a.nseg - 1;
  bool no_sfx = false;
  if constexpr (RST) {
    // The first document start after the segment: that of the nearest later
    // segment holding one, as the aggregate pass found them.
    int64_t fr = -1;
    if (a.segreset) {
      // Lane j > seg reads segment j's record (one load each, in parallel).
      const int v = lane > seg && lane < a.nseg ? a.segreset[bh * a.nseg + lane] : -1;
      const uint64_t m = __ballot(v >= 0);
      if (m) fr = __builtin_amdgcn_readlane(v, __builtin_ctzll(m));
    } else {
      fr = first_reset_in<NT>(Rrow, t_end, T, tid, red);
    }
    if (fr == t_end) no_sfx = true;
    else if (fr > 0) j_last = fr / a.seg_len;
  }

  // Column-block state (wave w < JB): Wj[e][ib] holds W[i = 16ib + 4q + r][j = 16 blk(e) + c]
  // and Rj[ib] holds R[i][j = 16w + c], at the segment's end: W_0 - sum_{j<=seg} A_j
  // (subtracted in segment order) and R = sum_{j>seg} B_j (added from the last segment down).
  f32x4 Wj[NWB][IB], Rj[IB];
  constexpr int PU = IB <= 4 ? 4 : 1;  // aggregates summed per batch of loads (register budget)
  if (w < JB) {
    // The segment's end state: saved by the forward, or W_0 minus the
    // aggregated writes up to and including this segment.
    const float* w0 = a.wend ? a.wend + (bh * a.nseg + seg) * M * D : a.W0 + (bh % a.H) * M * D;
#pragma unroll
    for (int e = 0; e < NWB; ++e) {
#pragma unroll
      for (int ib = 0; ib < IB; ++ib)
#pragma unroll
        for (int r = 0; r < 4; ++r) Wj[e][ib][r] = w0[(int64_t)(16 * ib + 4 * q + r) * D + 16 * blk(e) + c];
      const int64_t o = bh * a.nseg * M * D + (int64_t)(16 * blk(e) + c) * M + 4 * q;
      for (int64_t j0 = 0; !a.wend && j0 <= seg; j0 += PU) {
        f32x4 v[PU][IB];
#pragma unroll
        for (int u = 0; u < PU; ++u)
#pragma unroll
          for (int ib = 0; ib < IB; ++ib)
            v[u][ib] = j0 + u <= seg ? *reinterpret_cast<const f32x4*>(a.aggA + o + (j0 + u) * M * D + 16 * ib) : zero4();
#pragma unroll
        for (int u = 0; u < PU; ++u)
#pragma unroll
          for (int ib = 0; ib < IB; ++ib)
            if (j0 + u <= seg) Wj[e][ib] -= v[u][ib];
      }
    }
    const int64_t o = bh * a.nseg * M * D + (int64_t)(16 * w + c) * M + 4 * q;
#pragma unroll
    for (int ib = 0; ib < IB; ++ib) Rj[ib] = zero4();
    if (FULL && a.aggB && !no_sfx) {
      for (int64_t j0 = j_last; j0 > seg; j0 -= PU) {
        f32x4 v[PU][IB];
#pragma unroll
        for (int u = 0; u < PU; ++u)
#pragma unroll
          for (int ib = 0; ib < IB; ++ib)
            v[u][ib] = j0 - u > seg ? *reinterpret_cast<const f32x4*>(a.aggB + o + (j0 - u) * M * D + 16 * ib) : zero4();
#pragma unroll
        for (int u = 0; u < PU; ++u)
#pragma unroll
          for (int ib = 0; ib < IB; ++ib)
            if (j0 - u > seg) Rj[ib] += v[u][ib];
      }
    }
  }
  for (int i = tid; i < C * C; i += NT) Es[i] = (E)0.f;
  if constexpr (SSH) {
    for (int i = tid; i < C * C; i += NT) Sh[i] = (E)0.f;
    if constexpr (OP::kSplit == 2)
      for (int i = tid; i < C * C; i += NT) Sl[i] = (E)0.f;
  }

  auto chunk = [&](TX& xr, TM& gr, TM& dr, EtaReg<ETAV>& er, RstReg<RST>& rr, int64_t n) {
    // A step before the segment start (the second of a pair) sees zero
    // tiles, leaves W and R unchanged and stores nothing.
    // Lane and thread indices as the chunk sees them: opaque to the compiler,
    // so that LDS addresses are formed per use instead of being hoisted out
    // of the loop into dozens of live registers.
    int ln = lane, td = tid;
    asm volatile("" : "+v"(ln), "+v"(td));
    const int c = ln & 15, q = ln >> 4;
    // Fragment address offsets of this lane for the tile widths in use, and
    // those of the wave's own column blocks (known only at run time).
    // Precomputed for square maps; with d != m the extra offset sets would
    // cost more registers than they save.
    constexpr bool PRE = D == M;
    const LaneOff<D, sizeof(E), PRE> lD = lane_off<D, sizeof(E), PRE>(ln);
    const LaneOff<M, sizeof(E), PRE> lM = lane_off_like<M>(lD);
    const LaneOff<C, sizeof(E), PRE> lC = lane_off_like<C>(lM);
    typename OP::tcol tD[NWB], tM[NWB];
    int nM[NWB];
#pragma unroll
    for (int e = 0; e < NWB; ++e) {
      tD[e] = OP::make_tcol(lD, 16 * blk(e));
      if constexpr (D == M) tM[e] = tD[e];
      else tM[e] = OP::make_tcol(lM, 16 * blk(e));
      nM[e] = PRE ? lM.nat_rt(0, 16 * blk(e)) : 0;
    }
    const int64_t t0 = t_begin + n * C;
    const bool live = n >= 0;
    const int nvalid = live ? (int)(t_end - t0 < C ? t_end - t0 : C) : 0;
    const rsrc_t Ogc = live ? Og : none, Oxc = live ? Ox : none, Odc = live ? Od : none, Oec = live ? Oe : none;
    __syncthreads();
    er.stage(et, C, a.eta_scalar, nvalid, 1.f, td);
    xr.store(Xs, td);
    gr.store(Gs, td);
    dr.store(Ds, td);
    __syncthreads();
    // Reset masks of this chunk (fr = C, lr = -1 without a reset).
    const uint64_t dm = rr.mask();
    const int fr = first_flag(dm), lr = last_flag(dm);
    const bool has = RST && lr >= 0 && live;
    if (ETAV) gr.store_scaled(Vh, Vl, td, et);  // read after the next barrier
    fetch(xr, gr, dr, er, rr, n - DEPTH);
    // The chunk's compute, compiled with the reset masks (HAS) for the chunks
    // that hold a reset and without them for the others.
    auto compute = [&](auto hc) {
    constexpr bool HAS = decltype(hc)::value;
    // A chunk holding a reset starts from the forward's saved state, not from
    // the un-write: loaded here into the state registers (unused until the
    // un-write step), so the loads overlap the score-tile phase.
    if constexpr (HAS) {
      if (w < JB) {
        const float* cs = a.cstate + (bh * ((T + C - 1) / C) + t0 / C) * M * D;
#pragma unroll
        for (int e = 0; e < NWB; ++e)
#pragma unroll
          for (int ib = 0; ib < IB; ++ib)
            Wj[e][ib] = *reinterpret_cast<const f32x4*>(cs + (int64_t)(16 * blk(e) + c) * M + 16 * ib + 4 * q);
      }
    }

    // (1) Intra-chunk tiles E[t][s], shared through LDS, and R_n^T (split).
#pragma unroll
    for (int idx = 0; idx < TB * (TB + 1) / 2; ++idx) {
      if (idx % NW != w) continue;
      int tb = 0;
      while ((tb + 1) * (tb + 2) / 2 <= idx) ++tb;
      const int sb = idx - tb * (tb + 1) / 2;
      // acc[r] = g_s . dY_t with s = 16sb + 4q + r, t = 16tb + c.
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < M / 32; ++kb)
        acc = OP::mma(acc, OP::load_n(Gs, lM, 16 * sb, 32 * kb), OP::load_n(Ds, lM, 16 * tb, 32 * kb));
      const int t = 16 * tb + c;
      // eta of the four s of this lane, read unconditionally (a select, not a branch per element).
      const f32x4 es = *reinterpret_cast<const f32x4*>(et + 16 * sb + 4 * q);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int s = 16 * sb + 4 * q + r;
        bool keep = tb > sb || (INCL ? (t >= s) : (t > s));
        if constexpr (HAS) keep = keep && same_doc(dm, s, t);
        acc[r] = keep ? acc[r] * es[r] : 0.f;
      }
      OP::store4(ptr_byte<E>(Es, lC.nat(16 * tb, 16 * sb)), acc);
    }
    if constexpr (SSH) {
      // Score tiles st[r] = x_s . x_t for the same (s, t) pairs, masked alike.
#pragma unroll
      for (int idx = 0; idx < TB * (TB + 1) / 2; ++idx) {
        if ((idx + NW / 2) % NW != w) continue;
        int tb = 0;
        while ((tb + 1) * (tb + 2) / 2 <= idx) ++tb;
        const int sb = idx - tb * (tb + 1) / 2;
        f32x4 st = zero4();
#pragma unroll
        for (int kb = 0; kb < D / 32; ++kb)
          st = OP::mma(st, OP::load_n(Xs, lD, 16 * sb, 32 * kb), OP::load_n(Xs, lD, 16 * tb, 32 * kb));
        const int t = 16 * tb + c;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int s = 16 * sb + 4 * q + r;
          bool keep = tb > sb || (INCL ? (t >= s) : (t > s));
          if constexpr (HAS) keep = keep && same_doc(dm, s, t);
          if (!keep) st[r] = 0.f;
        }
        const int o = lC.nat(16 * tb, 16 * sb);
        OP::store4_split(ptr_byte<E>(Sh, o), ptr_byte<E>(Sl, o), st);
      }
    }
    if (FULL && w < JB) {
#pragma unroll
      for (int ib = 0; ib < IB; ++ib) {
        const int o = lM.nat(16 * w, 16 * ib);
        OP::store4_split(ptr_byte<E>(Rh, o), ptr_byte<E>(Rl, o), Rj[ib]);
      }
    }
    __syncthreads();

    // X^T rows j of this wave's column block over the chunk's tokens: shared
    // by the un-write, both intra-chunk terms and the suffix update.
    F xt[NWB][C / 32];
    if (w < JB) {
#pragma unroll
      for (int e = 0; e < NWB; ++e)
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) xt[e][kb] = OP::load_t(Xs, lD, 32 * kb, tD[e]);
    }

    // (2) Un-write this chunk: W_n = W_{n+1} + (eta G)^T X (a chunk holding a
    // reset already holds W_n, loaded above).
    if (!HAS && w < JB) {
      if constexpr (ETAV) {
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
#pragma unroll
          for (int ib = 0; ib < IB; ++ib) {
            const F vh = OP::load_t(Vh, lM, 32 * kb, 16 * ib);
            F vl = vh;
            if constexpr (SPLITV) vl = OP::load_t(Vl, lM, 32 * kb, 16 * ib);
#pragma unroll
            for (int e = 0; e < NWB; ++e) Wj[e][ib] = mma_split_a<OP>(Wj[e][ib], vh, vl, xt[e][kb]);
          }
        }
      } else {
        f32x4 dw[NWB][IB];
#pragma unroll
        for (int e = 0; e < NWB; ++e)
#pragma unroll
          for (int ib = 0; ib < IB; ++ib) dw[e][ib] = zero4();
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
#pragma unroll
          for (int ib = 0; ib < IB; ++ib) {
            const F gq = OP::load_t(Gs, lM, 32 * kb, 16 * ib);
#pragma unroll
            for (int e = 0; e < NWB; ++e) dw[e][ib] = OP::mma(dw[e][ib], gq, xt[e][kb]);
          }
        }
        const float es = a.eta_scalar;
#pragma unroll
        for (int e = 0; e < NWB; ++e)
#pragma unroll
          for (int ib = 0; ib < IB; ++ib) Wj[e][ib] += es * dw[e][ib];
      }
    }

    // Token block hh of this wave in the gtilde/dX phase (tok3) and in the
    // U/dG phase (tok4).  In a pair, wave 2p + H takes token blocks {2H, 2H+1}
    // for gtilde/dX and {H, 3-H} for U/dG, which balances the causal
    // intra-chunk terms; H is a template constant so that those terms'
    // conditions fold at compile time.
    auto outputs = [&](auto hc) {
    constexpr int H = decltype(hc)::value;
    auto tok3 = [&](int hh) { return PAIR ? 2 * H + hh : hh; };
    auto tok4 = [&](int hh) { return PAIR ? (hh == 0 ? H : TB - 1 - H) : hh; };
    // (3) gtilde and dX for columns j of blocks blk(e), token blocks tok3(hh).
    if (w < JB) {
      f32x4 ga[NWB][TBW], xa2[NWB][TBW];
#pragma unroll
      for (int e = 0; e < NWB; ++e)
#pragma unroll
        for (int hh = 0; hh < TBW; ++hh) ga[e][hh] = xa2[e][hh] = zero4();
      // gtilde^T[j][t] += sum_i W[i][j] dY[t][i];  dXw^T[j][s] += sum_i R[i][j] G[s][i]
#pragma unroll
      for (int kb = 0; kb < M / 32; ++kb) {
        F wh[NWB], wl[NWB], rh[NWB], rl[NWB];  // R^T rows as published (split) in step (1)
#pragma unroll
        for (int e = 0; e < NWB; ++e) {
          OP::split(cat(Wj[e][2 * kb], Wj[e][2 * kb + 1]), wh[e], wl[e]);
          if (FULL) {
            rh[e] = OP::load_n(Rh, lM, 16 * blk(e), 32 * kb);
            rl[e] = rh[e];
            if constexpr (OP::kSplit == 2) rl[e] = OP::load_n(Rl, lM, 16 * blk(e), 32 * kb);
          }
        }
#pragma unroll
        for (int hh = 0; hh < TBW; ++hh) {
          const int tb = tok3(hh);
          F dq = OP::load_n(Ds, lM, 16 * tb, 32 * kb);
          F gq;
          if (FULL) gq = OP::load_n(Gs, lM, 16 * tb, 32 * kb);
          if constexpr (HAS) {
            dq = keep_row<OP>(dq, 16 * tb + c < fr);  // rows after the first reset read W_0 (below)
            if (FULL) gq = keep_row<OP>(gq, 16 * tb + c >= lr);  // only the last document sees R_n
          }
#pragma unroll
          for (int e = 0; e < NWB; ++e) {
            ga[e][hh] = mma_split_a<OP>(ga[e][hh], wh[e], wl[e], dq);
            if (FULL) xa2[e][hh] = mma_split_a<OP>(xa2[e][hh], rh[e], rl[e], gq);
          }
        }
      }
      if constexpr (HAS) {
        {
          const float* w0 = W0h;
#pragma unroll
          for (int kb = 0; kb < M / 32; ++kb) {
            F wh[NWB], wl[NWB];
#pragma unroll
            for (int e = 0; e < NWB; ++e) {
              f32x8 v;
#pragma unroll
              for (int r = 0; r < 8; ++r)
                v[r] = w0[(int64_t)(32 * kb + 16 * (r >> 2) + 4 * q + (r & 3)) * D + 16 * blk(e) + c];
              OP::split(v, wh[e], wl[e]);
            }
#pragma unroll
            for (int hh = 0; hh < TBW; ++hh) {
              const int tb = tok3(hh);
              const F dq = keep_row<OP>(OP::load_n(Ds, lM, 16 * tb, 32 * kb), 16 * tb + c >= fr);
#pragma unroll
              for (int e = 0; e < NWB; ++e) ga[e][hh] = mma_split_a<OP>(ga[e][hh], wh[e], wl[e], dq);
            }
          }
        }
      }
      if (FULL) {
#pragma unroll
        for (int hh = 0; hh < TBW; ++hh) {
          const float s = et[16 * tok3(hh) + c];
#pragma unroll
          for (int e = 0; e < NWB; ++e) xa2[e][hh] *= s;
        }
      }
      // Intra-chunk terms: gtilde -= sum_{s<t} X[s][j] E[t][s];  dXw += sum_{t>s} X[t][j] E[t][s]
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
#pragma unroll
        for (int hh = 0; hh < TBW; ++hh) {
          const int tb = tok3(hh);
          if (kb <= tb / 2) {
            const F ef = OP::load_n(Es, lC, 16 * tb, 32 * kb);
#pragma unroll
            for (int e = 0; e < NWB; ++e) ga[e][hh] = OP::mma(ga[e][hh], OP::neg(xt[e][kb]), ef);
          }
          if (FULL && kb >= tb / 2) {
            const F ef = OP::load_t(Es, lC, 32 * kb, 16 * tb);
#pragma unroll
            for (int e = 0; e < NWB; ++e) xa2[e][hh] = OP::mma(xa2[e][hh], xt[e][kb], ef);
          }
        }
      }
      // Lane holds row t = 16 tok3(hh) + c, columns j = 16 blk(e) + 4q + r; dX = gtilde - xa2.
#pragma unroll
      for (int hh = 0; hh < TBW; ++hh) {
        const int tb = tok3(hh);
        if constexpr (PAIR) {
          const uint32_t o = pair_off(t0 + 16 * tb, 32 * (w >> 1), D, c, q), o8 = o + 8 * D * 4;
          f32x4 lo, hi;
          if (a.gtilde) {
            pair_rows(ga[0][hh], ga[1][hh], lo, hi);
            buf_store4(Ogc, o, lo);
            buf_store4(Ogc, o8, hi);
          }
          if (FULL && a.dX) {
            pair_rows(ga[0][hh] - xa2[0][hh], ga[1][hh] - xa2[1][hh], lo, hi);
            buf_store4(Oxc, o, lo);
            buf_store4(Oxc, o8, hi);
          }
        } else {
          const uint32_t o = (uint32_t)(((t0 + 16 * tb + c) * D + 16 * w + 4 * q) * 4);
          if (a.gtilde) buf_store4(Ogc, o, ga[0][hh]);
          if (FULL && a.dX) buf_store4(Oxc, o, ga[0][hh] - xa2[0][hh]);
        }
      }
    }

    if constexpr (FULL) {
      // (4) U, dG and deta for rows i of blocks blk(e), token blocks tok4(hh).
      if (w < IB) {
        f32x4 ua[NWB][TBW];
#pragma unroll
        for (int e = 0; e < NWB; ++e)
#pragma unroll
          for (int hh = 0; hh < TBW; ++hh) ua[e][hh] = zero4();
        // Row fragments of X (rows t over j) serve both the R term and, when
        // the scores are not shared, the intra-chunk scores; they are then read
        // once when they fit the register budget (32 VGPRs), else per use.
        constexpr bool XCACHE = !SSH && TB * (D / 32) * (int)(sizeof(F) / 4) <= 32;
        F xr[XCACHE ? TB : 1][XCACHE ? D / 32 : 1];
        if constexpr (XCACHE) {
#pragma unroll
          for (int tb = 0; tb < TB; ++tb)
#pragma unroll
            for (int kb = 0; kb < D / 32; ++kb) xr[tb][kb] = OP::load_n(Xs, lD, 16 * tb, 32 * kb);
        }
        auto xrow = [&](int tb, int kb) -> F {
          if constexpr (XCACHE) return xr[tb][kb];
          else return OP::load_n(Xs, lD, 16 * tb, 32 * kb);
        };
        // -U^T[i][s] = sum_j R[i][j] X[s][j] + sum_t dY[t][i] S[t][s]
#pragma unroll
        for (int kb = 0; kb < D / 32; ++kb) {
          F rh[NWB], rl[NWB];
#pragma unroll
          for (int e = 0; e < NWB; ++e) {
            rh[e] = OP::load_t(Rh, lM, 32 * kb, tM[e]);
            rl[e] = rh[e];
            if constexpr (OP::kSplit == 2) rl[e] = OP::load_t(Rl, lM, 32 * kb, tM[e]);
          }
#pragma unroll
          for (int hh = 0; hh < TBW; ++hh) {
            F xq = xrow(tok4(hh), kb);
            if constexpr (HAS) xq = keep_row<OP>(xq, 16 * tok4(hh) + c >= lr);  // only the last document sees R_n
#pragma unroll
            for (int e = 0; e < NWB; ++e) ua[e][hh] = mma_split_a<OP>(ua[e][hh], rh[e], rl[e], xq);
          }
        }
        if constexpr (SSH) {
          // Intra-chunk term from the shared split scores: the operand for
          // row s over k = t is a transposing read of the [t][s] tile.
#pragma unroll
          for (int kb = 0; kb < C / 32; ++kb) {
            F dq[NWB];
#pragma unroll
            for (int e = 0; e < NWB; ++e) dq[e] = OP::load_t(Ds, lM, 32 * kb, tM[e]);
#pragma unroll
            for (int hh = 0; hh < TBW; ++hh) {
              const int sb = tok4(hh);
              if (sb > 2 * kb + 1) continue;
              const F sh = OP::load_t(Sh, lC, 32 * kb, 16 * sb);
              F sl = sh;
              if constexpr (OP::kSplit == 2) sl = OP::load_t(Sl, lC, 32 * kb, 16 * sb);
#pragma unroll
              for (int e = 0; e < NWB; ++e) ua[e][hh] = mma_split_b<OP>(ua[e][hh], dq[e], sh, sl);
            }
          }
        } else {
        // Intra-chunk term with S[t][s] = x_t . x_s computed here, per pair of
        // t blocks, and kept in fp32 registers (split for the matrix core):
        // the tile (rows t, cols s) is directly the operand contracted over t.
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
          F dq[NWB];
#pragma unroll
          for (int e = 0; e < NWB; ++e) dq[e] = OP::load_t(Ds, lM, 32 * kb, tM[e]);
#pragma unroll
          for (int hh = 0; hh < TBW; ++hh) {
            const int sb = tok4(hh);
            if (sb > 2 * kb + 1) continue;
            f32x8 sv;
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
              const int tb = 2 * kb + h2;
              f32x4 st = zero4();
              if (tb >= sb) {
#pragma unroll
                for (int kj = 0; kj < D / 32; ++kj) st = OP::mma(st, xrow(tb, kj), xrow(sb, kj));
                if (tb == sb) {
#pragma unroll
                  for (int r = 0; r < 4; ++r) {
                    const int t = 4 * q + r;
                    if (!(INCL ? (t >= c) : (t > c))) st[r] = 0.f;
                  }
                }
                if constexpr (HAS) {
#pragma unroll
                  for (int r = 0; r < 4; ++r)
                    if (!same_doc(dm, 16 * tb + 4 * q + r, 16 * sb + c)) st[r] = 0.f;
                }
              }
#pragma unroll
              for (int r = 0; r < 4; ++r) sv[4 * h2 + r] = st[r];
            }
            F sh, sl;
            OP::split(sv, sh, sl);
#pragma unroll
            for (int e = 0; e < NWB; ++e) ua[e][hh] = mma_split_b<OP>(ua[e][hh], dq[e], sh, sl);
          }
        }
        }
#pragma unroll
        for (int hh = 0; hh < TBW; ++hh) {
          // Lane holds token s = 16 tok4(hh) + c, rows i = 16 blk(e) + 4q + r; U = -ua.
          const int sb = tok4(hh);
          const int s = 16 * sb + c;
          const float es = et[s];
          if (a.dG) {
            if constexpr (PAIR) {
              const uint32_t o = pair_off(t0 + 16 * sb, 32 * (w >> 1), M, c, q);
              f32x4 lo, hi;
              pair_rows(-es * ua[0][hh], -es * ua[1][hh], lo, hi);
              buf_store4(Odc, o, lo);
              buf_store4(Odc, o + 8 * M * 4, hi);
            } else {
              buf_store4(Odc, (uint32_t)(((t0 + s) * M + 16 * w + 4 * q) * 4), -es * ua[0][hh]);
            }
          }
          if (a.deta) {
            typedef typename Vec4<E>::type vec4;
            float p = 0.f;
#pragma unroll
            for (int e = 0; e < NWB; ++e) {
              const vec4 gv = at_byte<vec4>(Gs, PRE ? 16 * sb * M * (int)sizeof(E) + nM[e] : lM.nat(16 * sb, 16 * blk(e)));
#pragma unroll
              for (int r = 0; r < 4; ++r) p -= (float)gv[r] * ua[e][hh][r];
            }
            // The four lane groups' partial sums are added after the barrier
            // below (no cross-lane shuffles here).
            dpart[PAIR ? (w >> 1) : w][q][s] = p;
          }
        }
      }

    }
    if constexpr (FULL) {
      // (5) Suffix update: R_{n-1} = R_n + dY^T X (exact products).
      if (w < JB) {
        // With a reset the previous chunk's document ends at the first reset:
        // the suffix restarts from the tokens before it.
        if (HAS)
#pragma unroll
          for (int ib = 0; ib < IB; ++ib) Rj[ib] = zero4();
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
#pragma unroll
          for (int ib = 0; ib < IB; ++ib) {
            F dsf = OP::load_t(Ds, lM, 32 * kb, 16 * ib);
            if constexpr (HAS) dsf = mask_k<OP>(dsf, 32 * kb, q, 0, fr);
            Rj[ib] = OP::mma(Rj[ib], dsf, xt[PAIR ? H : 0][kb]);
          }
        }
      }
    }
    };
    if (PAIR && (w & 1)) outputs(IntC<1>{});
    else outputs(IntC<0>{});

    if constexpr (FULL) {
      if (a.deta) {
        __syncthreads();
        const int tt = td < C ? td : 0;
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < (PAIR ? 2 : IB); ++i)
          s += (dpart[i][0][tt] + dpart[i][1][tt]) + (dpart[i][2][tt] + dpart[i][3][tt]);
        buf_store1(Oec, td < C ? (uint32_t)((t0 + td) * 4) : kOOB, s);
      }
    }
      };
    if (RST && has) compute(IntC<RST ? 1 : 0>{});
    else compute(IntC<0>{});
  };

  if constexpr (DEPTH == 2) {
    for (int64_t n = nch - 1; n >= 0; n -= 2) {
      chunk(xa, ga, da, ea, ra, n);
      chunk(xb, gb, db, eb, rb, n - 1);
    }
  } else {
    for (int64_t n = nch - 1; n >= 0; --n) chunk(xa, ga, da, ea, ra, n);
  }

  // Segment 0 ends holding the sum over the whole sequence of dY x^T.
  if (FULL && a.rfin && seg == 0 && w < JB) {
    float* o = a.rfin + bh * M * D;
#pragma unroll
    for (int ib = 0; ib < IB; ++ib)
#pragma unroll
      for (int r = 0; r < 4; ++r) o[(int64_t)(16 * ib + 4 * q + r) * D + 16 * w + c] = Rj[ib][r];
  }
}

// Wave-specialised full backward for square maps (d == m).  Waves [0, JB)
// own column blocks of W: the un-write, gtilde and dX.  Waves [JB, 2JB) own
// the same column blocks of R: its publication to LDS, the suffix update, and
// the row blocks of U (dG, deta).  Each wave keeps half the state of
// bwd_main_kernel's waves, so twice as many waves share a CU and hide each
// other's LDS and matrix-core latency.  Same chunk equations, same rounding.
template <class OP, int D, int M, int C, bool INCL, bool ETAV>
__global__ void __launch_bounds__(2 * (D / 16) * 64, 128 / D)
bwd_split_kernel(const BArgs a) {
  static_assert(D == M, "the wave-specialised backward takes square maps");
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int JB = D / 16, IB = M / 16, NW = 2 * JB, NT = NW * 64, TB = C / 16;
  constexpr bool SPLITV = ETAV && OP::kSplit == 2;
  __shared__ E Xs[C * D];                  // X[t][j]
  __shared__ E Gs[C * M];                  // G[t][i]
  __shared__ E Ds[C * M];                  // dY[t][i]
  __shared__ E Es[C * C];                  // E[t][s] = eta_s dY_t . g_s (s before t)
  __shared__ E Vh[ETAV ? C * M : 1];       // (eta G)[t][i] hi (per-token eta)
  __shared__ E Vl[SPLITV ? C * M : 1];     // (eta G)[t][i] lo
  __shared__ E Rh[D * M];                  // R^T[j][i] hi
  __shared__ E Rl[OP::kSplit == 2 ? D * M : 1];  // R^T[j][i] lo
  constexpr bool SSH = !ETAV && s_shared_fits(OP::kSplit == 2, D, M, C, ETAV);
  __shared__ E Sh[SSH ? C * C : 1];
  __shared__ E Sl[SSH && OP::kSplit == 2 ? C * C : 1];
  __shared__ __attribute__((aligned(16))) float et[C];
  __shared__ float dpart[IB][C];

  int64_t bh, seg;
  if (!map_block(a.BH, a.nseg, bh, seg)) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, c = lane & 15, q = lane >> 4;
  const bool gw = w < JB;          // owner of W's column block wb (else of R's)
  const int wb = gw ? w : w - JB;
  const int64_t T = a.T;
  const int64_t t_begin = seg * a.seg_len;
  const int64_t t_end = t_begin + a.seg_len < T ? t_begin + a.seg_len : T;
  const rsrc_t X = make_rsrc(static_cast<const E*>(a.X) + bh * T * D, (uint32_t)(T * D * sizeof(E)));
  const rsrc_t G = make_rsrc(static_cast<const E*>(a.G) + bh * T * M, (uint32_t)(T * M * sizeof(E)));
  const rsrc_t Dy = make_rsrc(static_cast<const E*>(a.dY) + bh * T * M, (uint32_t)(T * M * sizeof(E)));
  const rsrc_t Og = make_rsrc(a.gtilde ? a.gtilde + bh * T * D : nullptr, a.gtilde ? (uint32_t)(T * D * 4) : 0u);
  const rsrc_t Ox = make_rsrc(a.dX ? a.dX + bh * T * D : nullptr, a.dX ? (uint32_t)(T * D * 4) : 0u);
  const rsrc_t Od = make_rsrc(a.dG ? a.dG + bh * T * M : nullptr, a.dG ? (uint32_t)(T * M * 4) : 0u);
  const rsrc_t Oe = make_rsrc(a.deta ? a.deta + bh * T : nullptr, a.deta ? (uint32_t)(T * 4) : 0u);
  const int64_t nch = (t_end - t_begin + C - 1) / C;

  // Register staging one chunk ahead (chunks are visited last to first).
  typedef TileRow<OP, C, D, NT> TX;
  typedef TileRow<OP, C, M, NT> TM;
  TX xr;
  TM gr, dr;
  EtaReg<ETAV> er;
  const rsrc_t Et = eta_rsrc(a.eta, bh, T);
  auto fetch = [&](int64_t n) {
    const int64_t t0 = t_begin + n * C;
    er.load(Et, n >= 0 ? (uint32_t)(t0 * 4) : kOOB, tid, C);
    xr.load(X, n >= 0 ? (uint32_t)(t0 * D * sizeof(E)) : kOOB, tid);
    gr.load(G, n >= 0 ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
    dr.load(Dy, n >= 0 ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
  };
  fetch(nch - 1);

  // St[ib][r] = W (owners of W) or R (owners of R) at [i = 16ib + 4q + r][j = 16wb + c],
  // at the segment's end: the saved state or W_0 - sum_{k<=seg} A_k, and
  // R = sum_{k>seg} B_k (added from the last segment down).
  f32x4 St[IB];
  constexpr int PU = IB <= 4 ? 4 : 1;  // aggregates summed per batch of loads (register budget)
  const int64_t ao = bh * a.nseg * M * D + (int64_t)(16 * wb + c) * M + 4 * q;
  if (gw) {
    const float* w0 = a.wend ? a.wend + (bh * a.nseg + seg) * M * D : a.W0 + (bh % a.H) * M * D;
#pragma unroll
    for (int ib = 0; ib < IB; ++ib)
#pragma unroll
      for (int r = 0; r < 4; ++r) St[ib][r] = w0[(int64_t)(16 * ib + 4 * q + r) * D + 16 * wb + c];
    for (int64_t j0 = 0; !a.wend && j0 <= seg; j0 += PU) {
      f32x4 v[PU][IB];
#pragma unroll
      for (int u = 0; u < PU; ++u)
#pragma unroll
        for (int ib = 0; ib < IB; ++ib)
          v[u][ib] = j0 + u <= seg ? *reinterpret_cast<const f32x4*>(a.aggA + ao + (j0 + u) * M * D + 16 * ib) : zero4();
#pragma unroll
      for (int u = 0; u < PU; ++u)
#pragma unroll
        for (int ib = 0; ib < IB; ++ib)
          if (j0 + u <= seg) St[ib] -= v[u][ib];
    }
  } else {
#pragma unroll
    for (int ib = 0; ib < IB; ++ib) St[ib] = zero4();
    for (int64_t j0 = a.nseg - 1; a.aggB && j0 > seg; j0 -= PU) {
      f32x4 v[PU][IB];
#pragma unroll
      for (int u = 0; u < PU; ++u)
#pragma unroll
        for (int ib = 0; ib < IB; ++ib)
          v[u][ib] = j0 - u > seg ? *reinterpret_cast<const f32x4*>(a.aggB + ao + (j0 - u) * M * D + 16 * ib) : zero4();
#pragma unroll
      for (int u = 0; u < PU; ++u)
#pragma unroll
        for (int ib = 0; ib < IB; ++ib)
          if (j0 - u > seg) St[ib] += v[u][ib];
    }
  }
  for (int i = tid; i < C * C; i += NT) Es[i] = (E)0.f;
  if constexpr (SSH) {
    for (int i = tid; i < C * C; i += NT) Sh[i] = (E)0.f;
    if constexpr (OP::kSplit == 2)
      for (int i = tid; i < C * C; i += NT) Sl[i] = (E)0.f;
  }

  for (int64_t n = nch - 1; n >= 0; --n) {
    const int64_t t0 = t_begin + n * C;
    const int nvalid = (int)(t_end - t0 < C ? t_end - t0 : C);
    // Lane and thread indices as the loop sees them: kept opaque to the
    // compiler so that LDS addresses are formed per use instead of being
    // hoisted out of the loop into dozens of live registers.
    int ln = lane, td = tid;
    asm volatile("" : "+v"(ln), "+v"(td));
    const int c = ln & 15, q = ln >> 4;
    __syncthreads();
    er.stage(et, C, a.eta_scalar, nvalid, 1.f, td);
    xr.store(Xs, td);
    gr.store(Gs, td);
    dr.store(Ds, td);
    __syncthreads();
    if (ETAV) gr.store_scaled(Vh, Vl, td, et);  // read after the next barrier
    fetch(n - 1);

    // (1) Intra-chunk tiles E[t][s] and the masked scores, shared through
    // LDS; the owners of R publish R_n^T (split).
#pragma unroll
    for (int idx = 0; idx < TB * (TB + 1) / 2; ++idx) {
      if (idx % NW != w) continue;
      int tb = 0;
      while ((tb + 1) * (tb + 2) / 2 <= idx) ++tb;
      const int sb = idx - tb * (tb + 1) / 2;
      // acc[r] = g_s . dY_t with s = 16sb + 4q + r, t = 16tb + c.
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < M / 32; ++kb)
        acc = OP::mma(acc, OP::load_n(Gs, M, 16 * sb, 32 * kb, ln), OP::load_n(Ds, M, 16 * tb, 32 * kb, ln));
      const int t = 16 * tb + c;
      const f32x4 es = *reinterpret_cast<const f32x4*>(et + 16 * sb + 4 * q);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int s = 16 * sb + 4 * q + r;
        const bool keep = tb > sb || (INCL ? (t >= s) : (t > s));
        acc[r] = keep ? acc[r] * es[r] : 0.f;
      }
      OP::store4(Es + lds_off(t, 16 * sb + 4 * q, C), acc);
    }
    if constexpr (SSH) {
#pragma unroll
      for (int idx = 0; idx < TB * (TB + 1) / 2; ++idx) {
        if ((idx + NW / 2) % NW != w) continue;
        int tb = 0;
        while ((tb + 1) * (tb + 2) / 2 <= idx) ++tb;
        const int sb = idx - tb * (tb + 1) / 2;
        f32x4 st = zero4();
#pragma unroll
        for (int kb = 0; kb < D / 32; ++kb)
          st = OP::mma(st, OP::load_n(Xs, D, 16 * sb, 32 * kb, ln), OP::load_n(Xs, D, 16 * tb, 32 * kb, ln));
        const int t = 16 * tb + c;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int s = 16 * sb + 4 * q + r;
          if (!(tb > sb || (INCL ? (t >= s) : (t > s)))) st[r] = 0.f;
        }
        const int o = lds_off(t, 16 * sb + 4 * q, C);
        OP::store4_split(Sh + o, Sl + o, st);
      }
    }
    if (!gw) {
#pragma unroll
      for (int ib = 0; ib < IB; ++ib) {
        const int o = lds_off(16 * wb + c, 16 * ib + 4 * q, M);
        OP::store4_split(Rh + o, Rl + o, St[ib]);
      }
    }
    __syncthreads();

    // X^T rows j of this wave's column block over the chunk's tokens.
    F xt[C / 32];
#pragma unroll
    for (int kb = 0; kb < C / 32; ++kb) xt[kb] = OP::load_t(Xs, D, 32 * kb, 16 * wb, ln);

    if (gw) {
      // (2) Un-write this chunk: W_n = W_{n+1} + (eta G)^T X.
      if constexpr (ETAV) {
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
#pragma unroll
          for (int ib = 0; ib < IB; ++ib) {
            const F vh = OP::load_t(Vh, M, 32 * kb, 16 * ib, ln);
            F vl = vh;
            if constexpr (SPLITV) vl = OP::load_t(Vl, M, 32 * kb, 16 * ib, ln);
            St[ib] = mma_split_a<OP>(St[ib], vh, vl, xt[kb]);
          }
        }
      } else {
        f32x4 dw[IB];
#pragma unroll
        for (int ib = 0; ib < IB; ++ib) dw[ib] = zero4();
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
#pragma unroll
          for (int ib = 0; ib < IB; ++ib) dw[ib] = OP::mma(dw[ib], OP::load_t(Gs, M, 32 * kb, 16 * ib, ln), xt[kb]);
        }
        const float e = a.eta_scalar;
#pragma unroll
        for (int ib = 0; ib < IB; ++ib) St[ib] += e * dw[ib];
      }

      // (3) gtilde and dX for columns j in [16wb, 16wb+16), all t blocks at once.
      f32x4 ga[TB], xa2[TB];
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) ga[tb] = xa2[tb] = zero4();
      // gtilde^T[j][t] += sum_i W[i][j] dY[t][i];  dXw^T[j][s] += sum_i R[i][j] G[s][i]
#pragma unroll
      for (int kb = 0; kb < M / 32; ++kb) {
        F wh, wl;
        OP::split(cat(St[2 * kb], St[2 * kb + 1]), wh, wl);
        const F rh = OP::load_n(Rh, M, 16 * wb, 32 * kb, ln);
        F rl = rh;
        if constexpr (OP::kSplit == 2) rl = OP::load_n(Rl, M, 16 * wb, 32 * kb, ln);
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          ga[tb] = mma_split_a<OP>(ga[tb], wh, wl, OP::load_n(Ds, M, 16 * tb, 32 * kb, ln));
          xa2[tb] = mma_split_a<OP>(xa2[tb], rh, rl, OP::load_n(Gs, M, 16 * tb, 32 * kb, ln));
        }
        __builtin_amdgcn_sched_barrier(0);  // bound the operands in flight (register budget)
      }
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) xa2[tb] *= et[16 * tb + c];
      // Intra-chunk terms: gtilde -= sum_{s<t} X[s][j] E[t][s];  dXw += sum_{t>s} X[t][j] E[t][s]
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
        const F xq = xt[kb];
        const F xn = OP::neg(xq);
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          if (kb <= tb / 2) ga[tb] = OP::mma(ga[tb], xn, OP::load_n(Es, C, 16 * tb, 32 * kb, ln));
          if (kb >= tb / 2) xa2[tb] = OP::mma(xa2[tb], xq, OP::load_t(Es, C, 32 * kb, 16 * tb, ln));
        }
      }
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        const uint32_t o = (uint32_t)(((t0 + 16 * tb + c) * D + 16 * wb + 4 * q) * 4);
        if (a.gtilde) buf_store4(Og, o, ga[tb]);
        if (a.dX) buf_store4(Ox, o, ga[tb] - xa2[tb]);
      }
    } else {
      // (4) U, dG and deta for rows i in [16wb, 16wb+16), all s blocks at once.
      f32x4 ua[TB];
#pragma unroll
      for (int sb = 0; sb < TB; ++sb) ua[sb] = zero4();
      constexpr bool XCACHE = !SSH && TB * (D / 32) * (int)(sizeof(F) / 4) <= 32;
      F xc[XCACHE ? TB : 1][XCACHE ? D / 32 : 1];
      if constexpr (XCACHE) {
#pragma unroll
        for (int tb = 0; tb < TB; ++tb)
#pragma unroll
          for (int kb = 0; kb < D / 32; ++kb) xc[tb][kb] = OP::load_n(Xs, D, 16 * tb, 32 * kb, ln);
      }
      auto xrow = [&](int tb, int kb) -> F {
        if constexpr (XCACHE) return xc[tb][kb];
        else return OP::load_n(Xs, D, 16 * tb, 32 * kb, ln);
      };
      // -U^T[i][s] = sum_j R[i][j] X[s][j] + sum_t dY[t][i] S[t][s]
#pragma unroll
      for (int kb = 0; kb < D / 32; ++kb) {
        const F rh = OP::load_t(Rh, M, 32 * kb, 16 * wb, ln);
        F rl = rh;
        if constexpr (OP::kSplit == 2) rl = OP::load_t(Rl, M, 32 * kb, 16 * wb, ln);
#pragma unroll
        for (int sb = 0; sb < TB; ++sb) ua[sb] = mma_split_a<OP>(ua[sb], rh, rl, xrow(sb, kb));
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (SSH) {
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
          const F dq = OP::load_t(Ds, M, 32 * kb, 16 * wb, ln);
#pragma unroll
          for (int sb = 0; sb <= 2 * kb + 1 && sb < TB; ++sb) {
            const F sh = OP::load_t(Sh, C, 32 * kb, 16 * sb, ln);
            F sl = sh;
            if constexpr (OP::kSplit == 2) sl = OP::load_t(Sl, C, 32 * kb, 16 * sb, ln);
            ua[sb] = mma_split_b<OP>(ua[sb], dq, sh, sl);
          }
        }
      } else {
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
          const F dq = OP::load_t(Ds, M, 32 * kb, 16 * wb, ln);
#pragma unroll
          for (int sb = 0; sb <= 2 * kb + 1 && sb < TB; ++sb) {
            f32x8 sv;
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
              const int tb = 2 * kb + hh;
              f32x4 st = zero4();
              if (tb >= sb) {
#pragma unroll
                for (int kj = 0; kj < D / 32; ++kj) st = OP::mma(st, xrow(tb, kj), xrow(sb, kj));
                if (tb == sb) {
#pragma unroll
                  for (int r = 0; r < 4; ++r) {
                    const int t = 4 * q + r;
                    if (!(INCL ? (t >= c) : (t > c))) st[r] = 0.f;
                  }
                }
              }
#pragma unroll
              for (int r = 0; r < 4; ++r) sv[4 * hh + r] = st[r];
            }
            F sh, sl;
            OP::split(sv, sh, sl);
            ua[sb] = mma_split_b<OP>(ua[sb], dq, sh, sl);
          }
        }
      }
#pragma unroll
      for (int sb = 0; sb < TB; ++sb) {
        // Lane holds token s = 16sb + c, rows i = 16wb + 4q + r; U = -ua.
        const int s = 16 * sb + c;
        const float es = et[s];
        if (a.dG) buf_store4(Od, (uint32_t)(((t0 + s) * M + 16 * wb + 4 * q) * 4), -es * ua[sb]);
        if (a.deta) {
          typedef typename Vec4<E>::type vec4;
          const vec4 gv = *reinterpret_cast<const vec4*>(Gs + lds_off(s, 16 * wb + 4 * q, M));
          float p = 0.f;
#pragma unroll
          for (int r = 0; r < 4; ++r) p -= (float)gv[r] * ua[sb][r];
          p += __shfl_xor(p, 16);
          p += __shfl_xor(p, 32);
          if (q == 0) dpart[wb][s] = p;
        }
      }
      // (5) Suffix update: R_{n-1} = R_n + dY^T X (exact products).
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
#pragma unroll
        for (int ib = 0; ib < IB; ++ib) St[ib] = OP::mma(St[ib], OP::load_t(Ds, M, 32 * kb, 16 * ib, ln), xt[kb]);
      }
    }
    if (a.deta) {
      __syncthreads();
      const int tt = td < C ? td : 0;
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < IB; ++i) s += dpart[i][tt];
      buf_store1(Oe, td < C ? (uint32_t)((t0 + td) * 4) : kOOB, s);
    }
  }

  // Segment 0 ends holding the sum over the whole sequence of dY x^T.
  if (!gw && a.rfin && seg == 0) {
    float* o = a.rfin + bh * M * D;
#pragma unroll
    for (int ib = 0; ib < IB; ++ib)
#pragma unroll
      for (int r = 0; r < 4; ++r) o[(int64_t)(16 * ib + 4 * q + r) * D + 16 * wb + c] = St[ib][r];
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

// With resets: dW0[h][i][j] = sum_b sum_k aggF[b, h, k][j][i] (the full
// dY x^T of every segment, transposed), in a fixed order.  Four threads per
// (h, j, 4 consecutive i) each sum a quarter of the (b, k) terms, eight
// 16-byte reads in flight, and the quarters are added in order through LDS.
static __global__ void __launch_bounds__(256)
reduce_dw0_segs_kernel(const float* aggF, float* dW0, int64_t B, int64_t H, int64_t nseg, int D, int M) {
  __shared__ f32x4 part[4][64];
  const int M4 = M / 4;
  const int64_t g = (int64_t)blockIdx.x * 64 + (threadIdx.x & 63);
  const int quarter = threadIdx.x >> 6;
  const bool ok = g < H * (int64_t)D * M4;
  const int64_t h = ok ? g / ((int64_t)D * M4) : 0, j = g / M4 % D, i = 4 * (g % M4);
  const int64_t n = B * nseg, md = (int64_t)M * D, per = (n + 3) / 4;
  const int64_t k0 = quarter * per, k1 = k0 + per < n ? k0 + per : n;
  const float* p = aggF + j * M + i;
  f32x4 s = zero4();
  for (int64_t u0 = k0; ok && u0 < k1; u0 += 8) {
    f32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int64_t k = u0 + u, b = k / nseg, sg = k % nseg;
      v[u] = k < k1 ? *reinterpret_cast<const f32x4*>(p + ((b * H + h) * nseg + sg) * md) : zero4();
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  part[quarter][threadIdx.x & 63] = s;
  __syncthreads();
  if (quarter == 0 && ok) {
    const f32x4 t = ((part[0][threadIdx.x] + part[1][threadIdx.x]) + part[2][threadIdx.x]) + part[3][threadIdx.x];
#pragma unroll
    for (int r = 0; r < 4; ++r) dW0[(h * M + i + r) * D + j] = t[r];
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
// Tile length of the backward (the same for both eta forms): 64 for the
// 64 x 64 map; 32 for maps with a 128-wide side, whose per-wave state and
// accumulators do not fit the register budget at 64 (measured: the 128 x 128
// bf16 backward runs 1.85x faster at 32).  launch_scan_bwd dispatches on
// exactly this value.
int bwd_chunk_for(int bf16, int d, int m, int requested) {
  (void)bf16;
  (void)requested;
  return (d == 64 && m == 64) ? 64 : 32;
}
static_assert(lds_bytes_bwd(1, 64, 64, 64, 1) <= 160 * 1024, "bf16 backward tile does not fit LDS");
static_assert(lds_bytes_bwd(1, 128, 128, 32, 1) <= 160 * 1024, "bf16 backward tile does not fit LDS");
static_assert(lds_bytes_bwd(0, 64, 64, 64, 1) <= 160 * 1024, "fp32 backward tile does not fit LDS");
static_assert(lds_bytes_bwd(0, 128, 128, 32, 1) <= 160 * 1024, "fp32 backward tile does not fit LDS");

int bwd_wgs_per_cu(int bf16, int d, int m, int C) {
  const int s = s_shared_fits(bf16, d, m, C, false) ? (bf16 ? 2 : 1) * C * C * (bf16 ? 2 : 4) : 0;
  int n = 160 * 1024 / (lds_bytes_bwd(bf16, d, m, C, 0) + s);
  const int waves = cmax(d, m) / 16;
  if (n * waves > 8) n = 8 / waves;  // two waves per SIMD (register budget)
  return n < 1 ? 1 : n;
}

template <class OP, int D, int M, int C, bool ETAV>
static hipError_t bwd_dispatch2(const ScanProblem& p, const BwdPtrs& f, hipStream_t s) {
  constexpr int NT = cmax(D, M) / 16 * 64;
  const int64_t BH = p.B * p.H;
  const unsigned grid = (unsigned)seg_grid(BH, p.nseg);
  // Only gtilde requested: the reverse-time suffix is never needed.
  const bool read_only = !f.dX && !f.dG && !f.deta && !f.dW0;
  const bool need_sfx = p.nseg > 1 && !read_only;

  KArgs k{};
  k.W0 = f.W0;
  k.X = f.X;
  k.G = f.G;
  k.dY = f.dY;
  k.eta = f.eta;
  k.eta_scalar = f.eta_scalar;
  k.BH = BH;
  k.H = p.H;
  k.T = p.T;
  k.seg_len = p.seg_len;
  k.nseg = p.nseg;
  k.aggA = f.aggA;
  k.aggB = f.aggB;
  k.reset = f.reset;
  k.aggF = f.aggF;
  k.segreset = f.resets && !read_only ? f.segreset : nullptr;  // the pass that records them runs only then
  if (f.resets) {
    // Document resets at unit retention (the saved pair; exclusive 64 x 64
    // maps, 64-token chunks): pre-reset suffix aggregates and full per-segment
    // sums for dW0, then the reset kernel.
    if constexpr (D == 64 && M == 64 && C == 64) {
      if (p.inclusive || !f.wend || !f.cstate) return hipErrorInvalidValue;
      if (!read_only) {
        timing_begin(GRADLEV_K_BWD_AGG, s);
        hipLaunchKernelGGL((agg_kernel<OP, D, M, C, kAggBwdB, ETAV, true>), dim3(grid), dim3(NT), 0, s, k, p.nseg);
        timing_end(GRADLEV_K_BWD_AGG, s);
      }
      BArgs b{};
      b.W0 = f.W0;
      b.X = f.X;
      b.G = f.G;
      b.dY = f.dY;
      b.eta = f.eta;
      b.eta_scalar = f.eta_scalar;
      b.BH = BH;
      b.H = p.H;
      b.T = p.T;
      b.seg_len = p.seg_len;
      b.nseg = p.nseg;
      b.gtilde = f.gtilde;
      b.dX = f.dX;
      b.dG = f.dG;
      b.deta = f.deta;
      b.aggB = need_sfx ? f.aggB : nullptr;
      b.rfin = nullptr;
      b.wend = f.wend;
      b.reset = f.reset;
      b.cstate = f.cstate;
      b.segreset = k.segreset;
      timing_begin(GRADLEV_K_BWD_MAIN, s);
      if (read_only)
        hipLaunchKernelGGL((bwd_main_kernel<OP, D, M, C, false, ETAV, kOutRead, true>), dim3(grid), dim3(NT), 0, s, b);
      else
        hipLaunchKernelGGL((bwd_main_kernel<OP, D, M, C, false, ETAV, kOutFull, true>), dim3(grid), dim3(NT), 0, s, b);
      timing_end(GRADLEV_K_BWD_MAIN, s);
      if (f.dW0) {
        const int64_t n = p.H * (int64_t)D * M / 4;
        timing_begin(GRADLEV_K_BWD_DW0, s);
        hipLaunchKernelGGL(reduce_dw0_segs_kernel, dim3((unsigned)((n + 63) / 64)), dim3(256), 0, s, f.aggF, f.dW0,
                           p.B, p.H, p.nseg, D, M);
        timing_end(GRADLEV_K_BWD_DW0, s);
      }
      return hipGetLastError();
    } else {
      return hipErrorInvalidValue;
    }
  }
  // Segment aggregates (writes, and dY x^T when a suffix is needed); each
  // workgroup of the main kernel sums the ones it needs in its prologue.
  // With the forward's saved segment-end weights only the dY x^T aggregates
  // are left to compute (none when the suffix is not needed).
  if (f.wend) {
    if (need_sfx) {
      timing_begin(GRADLEV_K_BWD_AGG, s);
      hipLaunchKernelGGL((agg_kernel<OP, D, M, C, kAggBwdB, ETAV>), dim3(grid), dim3(NT), 0, s, k, p.nseg);
      timing_end(GRADLEV_K_BWD_AGG, s);
    }
  } else {
    timing_begin(GRADLEV_K_BWD_AGG, s);
    if (need_sfx)
      hipLaunchKernelGGL((agg_kernel<OP, D, M, C, kAggBwdAB, ETAV>), dim3(grid), dim3(NT), 0, s, k, p.nseg);
    else
      hipLaunchKernelGGL((agg_kernel<OP, D, M, C, kAggBwdA, ETAV>), dim3(grid), dim3(NT), 0, s, k, p.nseg);
    timing_end(GRADLEV_K_BWD_AGG, s);
  }

  BArgs b{};
  b.W0 = f.W0;
  b.X = f.X;
  b.G = f.G;
  b.dY = f.dY;
  b.eta = f.eta;
  b.eta_scalar = f.eta_scalar;
  b.BH = BH;
  b.H = p.H;
  b.T = p.T;
  b.seg_len = p.seg_len;
  b.nseg = p.nseg;
  b.gtilde = f.gtilde;
  b.dX = f.dX;
  b.dG = f.dG;
  b.deta = f.deta;
  b.aggA = f.aggA;
  b.aggB = need_sfx ? f.aggB : nullptr;
  b.rfin = f.dW0 ? f.rfin : nullptr;
  b.wend = f.wend;
  timing_begin(GRADLEV_K_BWD_MAIN, s);
  if (read_only) {
    if (p.inclusive)
      hipLaunchKernelGGL((bwd_main_kernel<OP, D, M, C, true, ETAV, kOutRead>), dim3(grid), dim3(NT), 0, s, b);
    else
      hipLaunchKernelGGL((bwd_main_kernel<OP, D, M, C, false, ETAV, kOutRead>), dim3(grid), dim3(NT), 0, s, b);
  } else {
    // 128 x 128 maps: the wave-specialised kernel (twice the waves per CU;
    // measured 428 -> 343 us per launch at B=2, H=16, T=16384).  Smaller maps
    // keep the single-role kernel, which two workgroups per CU already feed.
    if constexpr (D == 128 && M == 128) {
      if (p.inclusive)
        hipLaunchKernelGGL((bwd_split_kernel<OP, D, M, C, true, ETAV>), dim3(grid), dim3(2 * NT), 0, s, b);
      else
        hipLaunchKernelGGL((bwd_split_kernel<OP, D, M, C, false, ETAV>), dim3(grid), dim3(2 * NT), 0, s, b);
    } else {
      if (p.inclusive)
        hipLaunchKernelGGL((bwd_main_kernel<OP, D, M, C, true, ETAV, kOutFull>), dim3(grid), dim3(NT), 0, s, b);
      else
        hipLaunchKernelGGL((bwd_main_kernel<OP, D, M, C, false, ETAV, kOutFull>), dim3(grid), dim3(NT), 0, s, b);
    }
  }
  timing_end(GRADLEV_K_BWD_MAIN, s);
  if (f.dW0) {
    const int64_t md4 = (int64_t)D * M / 4, n = p.H * md4;
    timing_begin(GRADLEV_K_BWD_DW0, s);
    hipLaunchKernelGGL(reduce_dw0_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, f.rfin, f.dW0, p.B, p.H, md4);
    timing_end(GRADLEV_K_BWD_DW0, s);
  }
  return hipGetLastError();
}

template <class OP, int D, int M, int C>
static hipError_t bwd_dispatch(const ScanProblem& p, const BwdPtrs& f, hipStream_t s) {
  if (f.eta) return bwd_dispatch2<OP, D, M, C, true>(p, f, s);
  return bwd_dispatch2<OP, D, M, C, false>(p, f, s);
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
  if (p.chunk != bwd_chunk_for(p.bf16, p.d, p.m, 0)) return hipErrorInvalidValue;
  if (p.chunk == 64) return p.bf16 ? bwd_dispatch<OpBF16, 64, 64, 64>(p, f, s) : bwd_dispatch<OpF32, 64, 64, 64>(p, f, s);
  return p.bf16 ? bwd_by_dims<OpBF16, 32>(p, f, s) : bwd_by_dims<OpF32, 32>(p, f, s);
}

}  // namespace gradlev
