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
//   * segments are joined by their aggregated writes A_k = sum eta g x^T
//     (agg_kernel, one pass before the main kernel); a workgroup starts from
//     W_0 - sum_{j<k} A_j, summed in its prologue.
// Chunk inputs are staged through registers two chunks ahead of the compute
// (about 3 us of loaded HBM latency has to be covered) into row-major LDS
// tiles; operands with k along the tile rows use the transposing LDS read.
#include "scan_common.hpp"

namespace gradlev {

// ---------------------------------------------------------------------------
// Main forward kernel.  NW = max(d, m)/16 waves.  Wave w < m/16 owns output
// rows i in [16w, 16w+16): it holds that slice of the state as accumulator
// tiles of W^T (rows j, cols i) and produces the matching columns of Y for
// every token of the chunk.
// ---------------------------------------------------------------------------
// RST (document resets, unit retention; exclusive reads, 64-token chunks):
// the chunk masks of scan_common.hpp.  Scores pair tokens of one document
// only; rows at or after the chunk's first reset read W_0 (a second state
// pass against W_0, in the chunks that hold a reset); the carry keeps the
// writes of the chunk's last document and restarts from W_0.  The state at
// the start of each such chunk is stored for the backward (cstate).
template <class OP, int D, int M, int C, bool INCL, bool ETAV, bool RST = false>
__global__ void __launch_bounds__(cmax(D, M) / 16 * 64, 128 / cmax(D, M))
fwd_main_kernel(const KArgs a) {
  typedef typename OP::elem E;
  typedef typename OP::frag F;
  constexpr int NW = cmax(D, M) / 16, NT = NW * 64;
  constexpr int TB = C / 16, JB = D / 16, IB = M / 16;
  constexpr bool SPLITV = ETAV && OP::kSplit == 2;
  __shared__ E Xs[C * D];                 // X[t][j]
  __shared__ E Gs[C * M];                 // G[t][i]
  // Scores -eta_s (x_t . x_s): built per wave in registers for bf16 tiles of up
  // to 64 tokens (no LDS round trip, no barrier); otherwise shared through LDS.
  constexpr bool RS = C <= 64 && OP::kSplit == 2;
  __shared__ E Pl[RS ? 1 : C * C];        // -eta_s (x_t . x_s) masked, [t][s]
  __shared__ E Vh[ETAV ? C * M : 1];      // -(eta G)[t][i] hi (per-token eta)
  __shared__ E Vl[SPLITV ? C * M : 1];    // -(eta G)[t][i] lo
  __shared__ __attribute__((aligned(16))) float et[C];
  static_assert(!RST || (C == 64 && !INCL), "resets: exclusive reads, 64-token chunks");
  __shared__ int red[1];
  __shared__ int didw[RST ? NW : 1][64];  // per wave: document index of each chunk position (reset chunks)

  int64_t bh, seg;
  if (!map_block(a.BH, a.nseg, bh, seg)) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, c = lane & 15, q = lane >> 4;
  const int64_t h = bh % a.H;
  const int64_t T = a.T;
  const int64_t t_begin = seg * a.seg_len;
  const int64_t t_end = t_begin + a.seg_len < T ? t_begin + a.seg_len : T;
  const rsrc_t X = make_rsrc(static_cast<const E*>(a.X) + bh * T * D, (uint32_t)(T * D * sizeof(E)));
  const rsrc_t G = make_rsrc(static_cast<const E*>(a.G) + bh * T * M, (uint32_t)(T * M * sizeof(E)));
  const rsrc_t Y = make_rsrc(a.out0 + bh * T * M, (uint32_t)(T * M * 4));
  // With resets: this sequence's chunk-start states (under 2 GiB, checked by the host).
  const int64_t nchs = (T + C - 1) / C;
  const rsrc_t Cst = make_rsrc(RST && a.cstate ? a.cstate + bh * nchs * M * D : nullptr,
                               RST && a.cstate ? (uint32_t)(nchs * M * D * 4) : 0u);

  // Register staging, two chunks ahead.
  Tile4<OP, C, D, NT> xa, xb;
  Tile4<OP, C, M, NT> ga, gb;
  EtaReg<ETAV> ea, eb;
  RstReg<RST> ra, rb;
  const rsrc_t Et = eta_rsrc(a.eta, bh, T);
  const rsrc_t Rrow = reset_rsrc(RST ? a.reset : nullptr, bh / a.H, T);
  auto fetch = [&](Tile4<OP, C, D, NT>& xr, Tile4<OP, C, M, NT>& gr, EtaReg<ETAV>& er, RstReg<RST>& rr,
                   int64_t t0) {
    const bool ok = t0 < t_end;
    er.load(Et, ok ? (uint32_t)(t0 * 4) : kOOB, tid, C);
    rr.load(Rrow, t0, ok, tid, C);
    xr.load(X, ok ? (uint32_t)(t0 * D * sizeof(E)) : kOOB, tid);
    gr.load(G, ok ? (uint32_t)(t0 * M * sizeof(E)) : kOOB, tid);
  };
  // With resets the segment starts from the state after the last document
  // start at or before t_begin: W_0 if that is t_begin itself, else W_0 minus
  // the (post-reset) aggregates from that document's segment on.
  fetch(xa, ga, ea, ra, t_begin);
  fetch(xb, gb, eb, rb, t_begin + C);
  int64_t j_first = 0;
  bool from_w0 = false;
  if constexpr (RST) {
    // The last document start at or before t_begin: the latest one the
    // aggregate pass found in an earlier segment, or t_begin itself.
    int64_t lr = -1;
    if (a.segreset) {
      // Lane j < seg reads segment j's record (one load each, in parallel);
      // the latest segment holding a document start has the latest one.
      const int v = lane < seg ? a.segreset[bh * a.nseg + lane] : -1;
      const uint64_t m = __ballot(v >= 0);
      if (m) lr = __builtin_amdgcn_readlane(v, 63 - __builtin_clzll(m));
      if (t_begin >= 1 && __builtin_amdgcn_raw_buffer_load_b8(Rrow, (int)t_begin, 0, 0) != 0) lr = t_begin;
    } else {
      lr = last_reset_in<NT>(Rrow, 0, t_begin, tid, red);
    }
    if (lr == t_begin) from_w0 = true;
    else if (lr > 0) j_first = lr / a.seg_len;
  }

  // State tiles: Ws[jb] holds W[i = 16w + c][j = 16jb + 4q + r] = W^T tile (rows j, cols i).
  // The segment starts from W_0 - sum_{j<seg} A_j (the aggregate pass's sums),
  // subtracted in segment order, four segments' loads in flight at a time.
  f32x4 Ws[JB];
  f32x4 W0r[RST ? JB : 1];  // with resets, this wave's rows of W_0 stay in registers
  if (w < IB) {
    const int64_t o = (int64_t)(16 * w + c) * D + 4 * q;
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) Ws[jb] = *reinterpret_cast<const f32x4*>(a.W0 + h * M * D + o + 16 * jb);
    if constexpr (RST)
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) W0r[jb] = Ws[jb];
    const float* ag = a.aggA + bh * a.nseg * M * D + o;
    for (int64_t j0 = j_first; !from_w0 && j0 < seg; j0 += 4) {
      f32x4 v[4][JB];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int jb = 0; jb < JB; ++jb)
          v[u][jb] = j0 + u < seg ? *reinterpret_cast<const f32x4*>(ag + (j0 + u) * M * D + 16 * jb) : zero4();
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int jb = 0; jb < JB; ++jb)
          if (j0 + u < seg) Ws[jb] -= v[u][jb];
    }
  }
  if constexpr (!RS)
    for (int i = tid; i < C * C; i += NT) Pl[i] = (E)0.f;

  // Saved-state block of the chunk ends: index and end of the current block
  // (save_len is a whole number of chunks and so divides t_begin).
  int64_t save_idx = 0, save_next = -1;
  if (a.wend) {
    save_idx = t_begin / a.save_len;
    save_next = (save_idx + 1) * a.save_len;
  }
  auto chunk = [&](Tile4<OP, C, D, NT>& xr, Tile4<OP, C, M, NT>& gr, EtaReg<ETAV>& er, RstReg<RST>& rr,
                   int64_t t0) {
    // A step past the segment end (the second of a pair) sees zero tiles,
    // leaves the state unchanged and stores nothing.
    const bool live = t0 < t_end;
    const int nvalid = live ? (int)(t_end - t0 < C ? t_end - t0 : C) : 0;
    __syncthreads();
    er.stage(et, C, a.eta_scalar, nvalid, -1.f, tid);
    xr.store(Xs, tid);
    gr.store(Gs, tid);
    __syncthreads();
    // Reset masks of this chunk (fr = C, lr = -1 without a reset).
    const uint64_t dm = rr.mask();
    const int fr = first_flag(dm), lr = last_flag(dm);
    const bool has = RST && lr >= 0 && live;
    if (ETAV) gr.store_scaled(Vh, Vl, tid, et);  // read by the carry, after a barrier
    // The state at the start of a chunk holding a reset, kept for the
    // backward: stored transposed, [d][m], so that the backward's lanes read
    // it 16 bytes at a time, and before the next chunks' loads, so that
    // waiting for those does not wait for these stores as well.
    // Streamed like the outputs: no dirty lines left in the L2 at the end.
    if (RST && has && a.cstate && w < IB) {
      const uint32_t o = (uint32_t)(((t0 / C) * M * D + 16 * w + c) * 4);
#pragma unroll
      for (int jb = 0; jb < JB; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) buf_store1(Cst, o + (uint32_t)((16 * jb + 4 * q + r) * M * 4), Ws[jb][r]);
    }
    fetch(xr, gr, er, rr, t0 + 2 * C);
    // The chunk's compute, compiled with the reset masks (HAS) for the chunks
    // that hold a reset and without them for the others.
    auto compute = [&](auto hc) {
    constexpr bool HAS = decltype(hc)::value;
    // Each wave writes its own table (in-order LDS within a wave: no barrier).
    if constexpr (HAS) didw[w][lane] = __builtin_popcountll(lane == 63 ? dm : dm & ((2ull << lane) - 1));

    // Intra-chunk scores, lower-triangular tiles (tb >= sb) shared by all waves.
    if constexpr (!RS) {
#pragma unroll
      for (int idx = 0; idx < TB * (TB + 1) / 2; ++idx) {
        if (idx % NW != w) continue;
        int tb = 0;
        while ((tb + 1) * (tb + 2) / 2 <= idx) ++tb;
        const int sb = idx - tb * (tb + 1) / 2;
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < D / 32; ++kb)
          acc = OP::mma(acc, OP::load_n(Xs, D, 16 * sb, 32 * kb, lane), OP::load_n(Xs, D, 16 * tb, 32 * kb, lane));
        // acc[r] = x_s . x_t with s = 16sb + 4q + r, t = 16tb + c; et holds -eta.
        const int t = 16 * tb + c;
        const f32x4 es = *reinterpret_cast<const f32x4*>(et + 16 * sb + 4 * q);
        f32x4 v;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int s = 16 * sb + 4 * q + r;
          bool keep = sb < tb || (INCL ? (s <= t) : (s < t));
          if constexpr (HAS) keep = keep && didw[w][s] == didw[w][t];
          v[r] = keep ? acc[r] * es[r] : 0.f;
        }
        OP::store4(Pl + lds_off(t, 16 * sb + 4 * q, C), v);
      }
      __syncthreads();
    }
    if (w < IB) {
      // Y^T[i][t] for all t blocks at once (independent accumulator chains).
      f32x4 acc[TB];
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) acc[tb] = zero4();
#pragma unroll
      for (int kb = 0; kb < D / 32; ++kb) {
        F wh, wl;
        OP::split(cat(Ws[2 * kb], Ws[2 * kb + 1]), wh, wl);
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          F xf = OP::load_n(Xs, D, 16 * tb, 32 * kb, lane);
          if constexpr (HAS) xf = keep_row<OP>(xf, 16 * tb + c < fr);
          acc[tb] = mma_split_a<OP>(acc[tb], wh, wl, xf);
        }
      }
      if constexpr (HAS) {
        {
          // Rows of the documents that start in this chunk read W_0.
#pragma unroll
          for (int kb = 0; kb < D / 32; ++kb) {
            F wh, wl;
            OP::split(cat(W0r[2 * kb], W0r[2 * kb + 1]), wh, wl);
#pragma unroll
            for (int tb = 0; tb < TB; ++tb)
              acc[tb] = mma_split_a<OP>(acc[tb], wh, wl,
                                        keep_row<OP>(OP::load_n(Xs, D, 16 * tb, 32 * kb, lane), 16 * tb + c >= fr));
          }
        }
      }
#pragma unroll
      for (int kb = 0; kb < C / 32; ++kb) {
        const F gq = OP::load_t(Gs, M, 32 * kb, 16 * w, lane);  // G[s][i], k = s
#pragma unroll
        for (int tb = 2 * kb; tb < TB; ++tb) {
          F sq;  // row t of -eta_s (x_t . x_s), masked, over k = s in [32kb, 32kb + 32)
          if constexpr (RS) {
            // The tile with rows s, cols t is the operand contracted over s:
            // built here from the X row fragments the state term already read.
            f32x8 sv;
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
              const int sb = 2 * kb + hh;
              f32x4 st = zero4();
              if (sb <= tb) {
#pragma unroll
                for (int kj = 0; kj < D / 32; ++kj)
                  st = OP::mma(st, OP::load_n(Xs, D, 16 * sb, 32 * kj, lane), OP::load_n(Xs, D, 16 * tb, 32 * kj, lane));
                const f32x4 es = *reinterpret_cast<const f32x4*>(et + 16 * sb + 4 * q);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                  bool keep = sb < tb || (INCL ? (4 * q + r <= c) : (4 * q + r < c));
                  if constexpr (HAS) keep = keep && didw[w][16 * sb + 4 * q + r] == didw[w][16 * tb + c];
                  st[r] = keep ? st[r] * es[r] : 0.f;
                }
              }
#pragma unroll
              for (int r = 0; r < 4; ++r) sv[4 * hh + r] = st[r];
            }
            F lo;
            OP::split(sv, sq, lo);  // hi part only: the same rounding as a bf16 score tile
          } else {
            sq = OP::load_n(Pl, C, 16 * tb, 32 * kb, lane);
          }
          acc[tb] = OP::mma(acc[tb], gq, sq);
        }
      }
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        // acc[tb][r] = y_t[i] with i = 16w + 4q + r, t = 16tb + c (rows past T are dropped).
        const int t = 16 * tb + c;
        // A dead step's stores go past the resource's end (selecting the
        // resource itself instead made the compiler loop over its values).
        buf_store4(Y, live ? (uint32_t)(((t0 + t) * M + 16 * w + 4 * q) * 4) : kOOB, acc[tb]);
      }
    }
    // The eta-scaled V tiles were written by every wave; with register scores
    // no barrier has passed since (the shared-score path had one).
    if constexpr (RS && ETAV) __syncthreads();
    if (w < IB) {
      // With resets: a carry that restarts from W_0 with the last document's writes.
      if constexpr (HAS) {
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) Ws[jb] = W0r[jb];
      }
      const int klo = HAS ? lr : 0;  // writes before the last reset do not reach the next chunk
      // Carry to the next chunk (also after the last one, where it is unused).
      if constexpr (ETAV) {
        // W^T[j][i] += sum_t X[t][j] (-eta G)[t][i], eta folded into the split operand.
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
          F vh = OP::load_t(Vh, M, 32 * kb, 16 * w, lane);
          F vl = vh;
          if constexpr (SPLITV) vl = OP::load_t(Vl, M, 32 * kb, 16 * w, lane);
          if constexpr (HAS) {
            vh = mask_k<OP>(vh, 32 * kb, q, klo, C);
            vl = mask_k<OP>(vl, 32 * kb, q, klo, C);
          }
#pragma unroll
          for (int jb = 0; jb < JB; ++jb)
            Ws[jb] = mma_split_b<OP>(Ws[jb], OP::load_t(Xs, D, 32 * kb, 16 * jb, lane), vh, vl);
        }
      } else {
        // Exact products G^T X, scaled once by the scalar eta.
        f32x4 dw[JB];
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) dw[jb] = zero4();
#pragma unroll
        for (int kb = 0; kb < C / 32; ++kb) {
          F gq = OP::load_t(Gs, M, 32 * kb, 16 * w, lane);
          if constexpr (HAS) gq = mask_k<OP>(gq, 32 * kb, q, klo, C);
#pragma unroll
          for (int jb = 0; jb < JB; ++jb) dw[jb] = OP::mma(dw[jb], OP::load_t(Xs, D, 32 * kb, 16 * jb, lane), gq);
        }
        const float e = a.eta_scalar;
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) Ws[jb] -= e * dw[jb];
      }
      // Saved for a backward: the fast weights after the last write of each
      // save_len-token block (and of the sequence), row-major [m][d]; lane
      // (c, q) holds W[16w + c][16jb + 4q .. +3].  The blocks are whole
      // chunks, so the next boundary is tracked instead of divided for.
      const int64_t te = t0 + C < t_end ? t0 + C : t_end;
      if (a.wend && live && (te == save_next || te == T)) {
        float* o = a.wend + (bh * a.nsave + save_idx) * M * D + (int64_t)(16 * w + c) * D + 4 * q;
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) *reinterpret_cast<f32x4*>(o + 16 * jb) = Ws[jb];
      }
      if (live && te == save_next) {
        save_next += a.save_len;
        ++save_idx;
      }
    }
      };
    if (RST && has) compute(IntC<RST ? 1 : 0>{});
    else compute(IntC<0>{});
  };

  for (int64_t t0 = t_begin; t0 < t_end; t0 += 2 * C) {
    chunk(xa, ga, ea, ra, t0);
    chunk(xb, gb, eb, rb, t0 + C);
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
static constexpr int lds_bytes_fwd(int bf16, int d, int m, int C, int etav) {
  const int es = bf16 ? 2 : 4;
  const int v = etav ? (bf16 ? 2 : 1) * C * m : 0;
  return es * (C * d + C * m + C * C + v) + 4 * C;
}

int fwd_chunk_for(int bf16, int d, int m, int requested) {
  int C = (bf16 && requested == 128) ? 128 : 64;
  if (C == 128 && lds_bytes_fwd(bf16, d, m, 128, 0) > 160 * 1024) C = 64;
  return C;
}

// Workgroups per CU the forward's segmentation aims at: one.  With inputs
// streamed from HBM, half as many segments of twice the length measured
// faster at B=8, H=16, T=2048, d=m=64 (main kernel 40 -> 35 us, aggregate
// pass 19 -> 17 us): fewer concurrent streams, and a quarter less aggregate
// reading.
int fwd_wgs_per_cu(int bf16, int d, int m, int C) {
  (void)bf16;
  (void)d;
  (void)m;
  (void)C;
  return 1;
}

template <class OP, int D, int M, int C, bool ETAV>
static hipError_t fwd_dispatch2(const ScanProblem& p, const KArgs& k, bool resets, hipStream_t s) {
  constexpr int NT = cmax(D, M) / 16 * 64;
  const unsigned grid = (unsigned)seg_grid(k.BH, p.nseg);
  if (resets) {
    // Document resets at unit retention: exclusive 64 x 64 maps, 64-token chunks.
    if constexpr (D == 64 && M == 64 && C == 64) {
      if (p.inclusive) return hipErrorInvalidValue;
      if (p.nseg > 1) {
        timing_begin(GRADLEV_K_FWD_AGG, s);
        hipLaunchKernelGGL((agg_kernel<OP, D, M, C, kAggFwd, ETAV, true>), dim3(grid), dim3(NT), 0, s, k, p.nseg - 1);
        timing_end(GRADLEV_K_FWD_AGG, s);
      }
      timing_begin(GRADLEV_K_FWD_MAIN, s);
      hipLaunchKernelGGL((fwd_main_kernel<OP, D, M, C, false, ETAV, true>), dim3(grid), dim3(NT), 0, s, k);
      timing_end(GRADLEV_K_FWD_MAIN, s);
      return hipGetLastError();
    } else {
      return hipErrorInvalidValue;
    }
  }
  if (p.nseg > 1) {
    timing_begin(GRADLEV_K_FWD_AGG, s);
    hipLaunchKernelGGL((agg_kernel<OP, D, M, C, kAggFwd, ETAV>), dim3(grid), dim3(NT), 0, s, k, p.nseg - 1);
    timing_end(GRADLEV_K_FWD_AGG, s);
  }
  timing_begin(GRADLEV_K_FWD_MAIN, s);
  if (p.inclusive)
    hipLaunchKernelGGL((fwd_main_kernel<OP, D, M, C, true, ETAV>), dim3(grid), dim3(NT), 0, s, k);
  else
    hipLaunchKernelGGL((fwd_main_kernel<OP, D, M, C, false, ETAV>), dim3(grid), dim3(NT), 0, s, k);
  timing_end(GRADLEV_K_FWD_MAIN, s);
  return hipGetLastError();
}

template <class OP, int D, int M, int C>
static hipError_t fwd_dispatch(const ScanProblem& p, const KArgs& k, bool resets, hipStream_t s) {
  constexpr int bf = OP::kSplit == 2 ? 1 : 0;
  if (k.eta) {
    // The per-token split operands need two more tiles of LDS; where they do
    // not fit at this tile length the chunk drops to 64 (same segments).
    if constexpr (lds_bytes_fwd(bf, D, M, C, 1) <= 160 * 1024) return fwd_dispatch2<OP, D, M, C, true>(p, k, resets, s);
    else return fwd_dispatch2<OP, D, M, 64, true>(p, k, resets, s);
  }
  return fwd_dispatch2<OP, D, M, C, false>(p, k, resets, s);
}

template <class OP, int C>
static hipError_t fwd_by_dims(const ScanProblem& p, const KArgs& k, bool resets, hipStream_t s) {
  if (p.d == 64 && p.m == 64) return fwd_dispatch<OP, 64, 64, C>(p, k, resets, s);
  if (p.d == 64 && p.m == 128) return fwd_dispatch<OP, 64, 128, C>(p, k, resets, s);
  if (p.d == 128 && p.m == 64) return fwd_dispatch<OP, 128, 64, C>(p, k, resets, s);
  if (p.d == 128 && p.m == 128) return fwd_dispatch<OP, 128, 128, C>(p, k, resets, s);
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
  k.BH = p.B * p.H;
  k.H = p.H;
  k.T = p.T;
  k.seg_len = p.seg_len;
  k.nseg = p.nseg;
  k.out0 = f.Y;
  k.aggA = p.nseg > 1 ? f.agg : nullptr;
  k.aggB = nullptr;
  k.wend = f.wend;
  k.save_len = f.save_len;
  k.nsave = f.nsave;
  k.reset = f.reset;
  k.cstate = f.cstate;
  k.segreset = f.resets && p.nseg > 1 ? f.segreset : nullptr;  // written by the aggregate pass
  if (f.resets && p.chunk != 64) return hipErrorInvalidValue;
  if (p.bf16) {
    if (p.chunk == 128) return fwd_by_dims<OpBF16, 128>(p, k, f.resets, s);
    return fwd_by_dims<OpBF16, 64>(p, k, f.resets, s);
  }
  return fwd_by_dims<OpF32, 64>(p, k, f.resets, s);
}

}  // namespace gradlev
