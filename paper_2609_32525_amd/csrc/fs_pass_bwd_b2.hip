// Streaming pass: backward pass B of the untied variant and of LinearNO in one kernel, for
// token sets one wavefront covers (G <= 64). Each point tile is read once and both weight
// sets are handled in turn: the slice weights (W_s, b, tau: dw = F dU^T + ds; for LinearNO
// normalised over the points of each slot, with no per-point correction) give dfx, their dx
// contribution and dW_s, db, dtau partials; the deslice weights (W_d, b_d, tau_d: dw = dO z'^T)
// add their dx contribution and give dW_d, db_d, dtau_d partials. dx is written once.
// Kernel design and MFMA lane layouts are described at the top of fs_stream.h.

#include "fs_stream.h"

namespace fs {
namespace {

// The operand images and the da transpose buffers must fit the 160 KB of LDS, and the
// registers: every shape but dh = 64 with 64 slots (which keeps the two-kernel form).
constexpr bool bwd_b2_fits(bool, int D, int GS) { return D < 64 || GS < 64; }

// COLN: LinearNO's slice weights. Partials per workgroup as in k_bwd_b, the slice set into
// a.part and the deslice set into a.part_d.
template <bool BF, int D, int GS, int NS, int NP, int PB, bool COLN>
__global__ __launch_bounds__(64 * NS * NP) __attribute__((amdgpu_waves_per_eu(GS <= 32 && D <= 32 ? FS_WPE_BWD_B2_G32 : FS_WPE_BWD_B))) void k_bwd_b2(
    PassArgs a) {
  static_assert(NS == 1, "one wavefront covers the tile's slots");
  static_assert(PB == 2 || !BF, "bf16 contracts over 32 points");
  constexpr int GB = GS / 16, VB = D / 16, DB = D / 16, TP = 16 * PB;
  constexpr bool SPLIT = BF;
  using T = typename Store<BF>::T;
  using SOp = SlotOp<BF, D, GB>;
  using UOp = GOp<BF, GB, VB>;
  using XOp = GOp<BF, GB, DB>;
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int wave = threadIdx.x >> 6, wp = wave;
  const HeadCtx c = head_ctx<D>(a, 0, GS);
  const int64_t rs = (int64_t)a.H * D;
  const T* xb = (const T*)a.x + c.off;
  const T* fb = (const T*)a.fx + c.off;
  const T* gb_ = (const T*)a.dout + c.off;
  T* dxb = (T*)a.out + c.off;
  T* dfb = (T*)a.out2 + c.off;
  const float inv_tau = 1.0f / a.tau[c.h];
  const float inv_taud = 1.0f / a.taud[c.h];
  const float scd = kLog2e * inv_taud;
  const float* Wd = a.Wd + (a.ws_per_head ? (int64_t)c.h * D * a.G : 0);
  const float* bd = a.bd + (a.ws_per_head ? (int64_t)c.h * a.G : 0);
  const float* zm = a.zmix + (int64_t)c.bh * a.G * D;
  const float* dU = a.dU + (int64_t)c.bh * a.G * D;
  // slot-mean shifts (valid for per-point softmax weights only, so not for LinearNO's slice)
  const float* cen = a.cen + (int64_t)c.bh * (2 * D + 1);
  float bT[GB][4], bTd[GB][4], dsT[GB][4];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      // padding blocks (slots >= G) read the last real block and take masked logits, no ds
      bool real;
      const int sl = slot_block(c.g0 + 16 * gb, slot_lim(a), real) + 4 * j + r;
      const float bv = c.sc * c.bias[sl] - (COLN ? a.clse[(int64_t)c.bh * a.G + sl] : 0.f);
      const float bdv = scd * bd[sl];
      const float dv = a.ds[(int64_t)c.bh * a.G + sl] - (COLN ? 0.f : cen[2 * D]);
      bT[gb][r] = slot_mask(real, bv, kMaskedSlot);
      bTd[gb][r] = slot_mask(real, bdv, kMaskedSlot);
      dsT[gb][r] = slot_mask(real, dv, 0.f);
    }

  // operand images in LDS, shared by the point groups: W_s, W_d (logits), zmix and dU
  // (dw, shifted), dU (dfx), W_s^T / tau and W_d^T / tau_d (dx)
  constexpr int kS = lds_chunks<SOp>(), kU = lds_chunks<UOp>(), kX = lds_chunks<XOp>();
  __shared__ uint4 opl[4 * kS + kU + 2 * kX];
  if (wp == 0) {
    SOp t;
    load_slotop<BF, D, GB, true, SPLIT>(t, c.W, a.G, c.g0, slot_lim(a), c.sc, i, j);
    lds_put(t, opl, lane);
    load_slotop<BF, D, GB, true, SPLIT>(t, Wd, a.G, c.g0, slot_lim(a), scd, i, j);
    lds_put(t, opl + kS, lane);
    load_slotop<BF, D, GB, false, false>(t, zm, D, c.g0, slot_lim(a), 1.0f, i, j, cen);
    lds_put(t, opl + 2 * kS, lane);
    load_slotop<BF, D, GB, false, false>(t, dU, D, c.g0, slot_lim(a), 1.0f, i, j, COLN ? nullptr : cen + D);
    lds_put(t, opl + 3 * kS, lane);
    UOp u;
    load_gop<BF, GB, VB, false>(u, dU, D, c.g0, slot_lim(a), 1.0f, i, j);
    lds_put(u, opl + 4 * kS, lane);
    XOp x;
    load_gop<BF, GB, DB, true>(x, c.W, a.G, c.g0, slot_lim(a), inv_tau, i, j);
    lds_put(x, opl + 4 * kS + kU, lane);
    load_gop<BF, GB, DB, true>(x, Wd, a.G, c.g0, slot_lim(a), inv_taud, i, j);
    lds_put(x, opl + 4 * kS + kU + kX, lane);
  }
  __syncthreads();

  // parameter accumulators: [0] slice weights, [1] deslice weights
  f4 dW[2][DB][GB];
  float dbacc[2][GB][4];
  double dtacc[2] = {0.0, 0.0};
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
      for (int r = 0; r < 4; ++r) dbacc[q][gb][r] = 0.f;
#pragma unroll
      for (int d = 0; d < DB; ++d) dW[q][d][gb] = zero4();
    }

  // per-wave da transpose buffer: fp32 [TP points][GS + 1], bf16 [GS slots][36]
  constexpr int kDaWords = da_words<BF, GS, TP>();
  __shared__ __attribute__((aligned(16))) float dabuf[NP][kDaWords];
  float* myda = dabuf[wp];

  const int64_t pbeg = (int64_t)c.chunk * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int npts = pend > pbeg ? (int)(pend - pbeg) : 0;
  const int ntile = (npts + TP * NP - 1) / (TP * NP);
  const int rsb = (int)(rs * sizeof(T));
  const auto rx = rows_rsrc(xb + pbeg * rs, npts, (int)rs, D);
  const auto rf = rows_rsrc(fb + pbeg * rs, npts, (int)rs, D);
  const auto rg = rows_rsrc(gb_ + pbeg * rs, npts, (int)rs, D);
  const auto rdx = rows_rsrc(dxb + pbeg * rs, npts, (int)rs, D);
  const auto rdf = rows_rsrc(dfb + pbeg * rs, npts, (int)rs, D);
  const float* lss = COLN ? a.lse_d : a.lse_in + (int64_t)c.bh * a.N + pbeg;  // unread for COLN
  const auto rls = rows_rsrc(lss, npts, 1, 1);
  const auto rld = rows_rsrc(a.lse_d + (int64_t)c.bh * a.N + pbeg, npts, 1, 1);
  const int wpu = __builtin_amdgcn_readfirstlane(wp);

  struct Tile {
    RowOp<BF, D> xo[PB], go[PB], fo[PB];
    float ls[PB], ld[PB];
    KGather<BF, DB, PB> xk;  // bf16: X again, points on the k index, for dW
  };
  auto load_tile = [&](Tile& tt, int t) {
    const int tb = (t * NP + wpu) * TP;
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int so = (tb + 16 * pb) * rsb;
      load_row_buf<BF, D>(tt.xo[pb], rx, i * rsb, so, j);
      load_row_buf<BF, D>(tt.go[pb], rg, i * rsb, so, j);
      load_row_buf<BF, D>(tt.fo[pb], rf, i * rsb, so, j);
      const bool ok = tb + 16 * pb + i < npts;
      const float l = COLN ? 0.f : bld32(rls, 4 * i, 4 * (tb + 16 * pb));
      tt.ls[pb] = ok ? l : kMasked;
      const float ld = bld32(rld, 4 * i, 4 * (tb + 16 * pb));
      tt.ld[pb] = ok ? ld : kMasked;
    }
    // fp32 loads this copy where it is used instead: holding it for a tile's lifetime costs
    // the fp32 kernels an occupancy step
    if constexpr (BF) gather_k<BF, DB, PB>(tt.xk, rx, rsb, tb, i, j);
  };

  // dW[q] += X^T da over the tile's points (da goes through LDS to put points on the k index)
  auto acc_dW = [&](f4 (&dWq)[DB][GB], const f4 (&da)[GB][PB], const Tile& cur, int tp0) {
    if constexpr (!BF) {
      KGather<BF, DB, PB> XK;
      gather_k<BF, DB, PB>(XK, rx, rsb, tp0, i, j);
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r) myda[da_at<GS>(16 * pb + i, 16 * gb + 4 * j + r)] = da[gb][pb][r];
      wave_lds_sync();
#pragma unroll
      for (int pb = 0; pb < PB; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pl = 16 * pb + 4 * j + r;
          float xv[DB];
#pragma unroll
          for (int d = 0; d < DB; ++d) xv[d] = XK.v[pb][r][d];
#pragma unroll
          for (int gb = 0; gb < GB; ++gb) {
            const float bv = myda[da_at<GS>(pl, 16 * gb + i)];
#pragma unroll
            for (int d = 0; d < DB; ++d) dWq[d][gb] = mfma_f32(xv[d], bv, dWq[d][gb]);
          }
        }
      wave_lds_sync();
    } else {
      unsigned short* t16 = reinterpret_cast<unsigned short*>(myda);
      da_put_bf<GB, PB>(t16, da, i, j);
      wave_lds_sync();
      const bf8(&xa)[DB] = cur.xk.v;
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
        const bf8 bt = da_get_bf(t16, gb, i, j);
#pragma unroll
        for (int d = 0; d < DB; ++d) dWq[d][gb] = mfma_bf16(xa[d], bt, dWq[d][gb]);
      }
      wave_lds_sync();
    }
  };

  pipeline<(FS_PF_BWD_B), Tile>(ntile, load_tile, [&](Tile& cur, int t) {
    const int tp0 = (t * NP + wpu) * TP;
    f4 gx_[DB][PB], gf[VB][PB];
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
#pragma unroll
      for (int d = 0; d < DB; ++d) gx_[d][pb] = zero4();
    }
    // q = 0: slice weights; q = 1: deslice weights
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      // T-layout tiles: rows = slots g0 + 16 gb + 4 j + r, cols = points 16 pb + i
      f4 tl[GB][PB], w[GB][PB], dw[GB][PB];
      {
        SOp wop;
        lds_get(wop, opl + q * kS, lane);
#pragma unroll
        for (int gb = 0; gb < GB; ++gb)
#pragma unroll
          for (int pb = 0; pb < PB; ++pb) {
            const float(&bb)[4] = q == 0 ? bT[gb] : bTd[gb];
            f4 acc = f4{bb[0], bb[1], bb[2], bb[3]};
            acc = mm_slot_row<BF, D, GB, SPLIT>(wop, gb, cur.xo[pb], acc);
            const float l2 = q == 0 ? cur.ls[pb] : cur.ld[pb];
            f4 tt, ww;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              tt[r] = acc[r] - l2;
              ww[r] = __builtin_amdgcn_exp2f(tt[r]);
            }
            tl[gb][pb] = tt;
            w[gb][pb] = ww;
          }
      }
      {
        SOp op;
        lds_get(op, opl + (q == 0 ? 3 : 2) * kS, lane);
#pragma unroll
        for (int gb = 0; gb < GB; ++gb)
#pragma unroll
          for (int pb = 0; pb < PB; ++pb) {
            f4 g = q == 0 ? f4{dsT[gb][0], dsT[gb][1], dsT[gb][2], dsT[gb][3]} : zero4();
            g = mm_slot_row<BF, D, GB, false>(op, gb, q == 0 ? cur.fo[pb] : cur.go[pb], g);
            dw[gb][pb] = g;
          }
      }
      // per point: c = sum_g w dw and tb = sum_g w t (none for LinearNO's slice weights)
      float cc[PB], tb[PB];
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        float sum = 0.f, st = 0.f;
        if (!(COLN && q == 0)) {
#pragma unroll
          for (int gb = 0; gb < GB; ++gb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              sum += w[gb][pb][r] * dw[gb][pb][r];
              st += w[gb][pb][r] * tl[gb][pb][r];
            }
          sum = col4_sum(sum);
          st = col4_sum(st);
        }
        cc[pb] = sum;
        tb[pb] = st;
      }
      float dts = 0.f;
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float da = w[gb][pb][r] * (dw[gb][pb][r] - cc[pb]);
            dw[gb][pb][r] = da;
            dts += da * (tl[gb][pb][r] - tb[pb]);
            dbacc[q][gb][r] += da;
          }
      dtacc[q] += (double)dts;
      {
        XOp wg;
        lds_get(wg, opl + 4 * kS + kU + q * kX, lane);
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
#pragma unroll
          for (int d = 0; d < DB; ++d) gx_[d][pb] = mm_gop_tile<BF, GB, DB, PB>(wg, d, dw, pb, gx_[d][pb]);
      }
      if (q == 0) {  // dfx = w dU (slice weights)
        UOp ug;
        lds_get(ug, opl + 4 * kS, lane);
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
#pragma unroll
          for (int vb = 0; vb < VB; ++vb) gf[vb][pb] = mm_gop_tile<BF, GB, VB, PB>(ug, vb, w, pb, zero4());
      }
      acc_dW(dW[q], dw, cur, tp0);
    }
#pragma unroll
    for (int pb = 0; pb < PB; ++pb)
#pragma unroll
      for (int cb = 0; cb < VB; ++cb) {
        const int vo = i * rsb + (16 * cb + 4 * j) * (int)sizeof(T), so = (tp0 + 16 * pb) * rsb;
        bst_row4<BF>(rdf, gf[cb][pb], vo, so);
        bst_row4<BF>(rdx, gx_[cb][pb], vo, so);
      }
  });

  // ---- finish: reduce over lanes and point groups, write both partials ------------------
  __shared__ f4 red[NP > 1 ? NP - 1 : 1][DB][GB][64];
  __shared__ float redb[NP > 1 ? NP - 1 : 1][GB][4][16];
  __shared__ double dtw[2][NP];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    float dbv[GB][4];
#pragma unroll
    for (int gb = 0; gb < GB; ++gb)
#pragma unroll
      for (int r = 0; r < 4; ++r) dbv[gb][r] = row16_sum(dbacc[q][gb][r]);
    double dt = dtacc[q];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) dt += __shfl_xor(dt, off);
    if (lane == 0) dtw[q][wave] = dt;
    if (NP > 1 && wp > 0) {
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
        for (int d = 0; d < DB; ++d) red[wp - 1][d][gb][lane] = dW[q][d][gb];
        if (i == 0)
#pragma unroll
          for (int r = 0; r < 4; ++r) redb[wp - 1][gb][r][j] = dbv[gb][r];
      }
    }
    __syncthreads();
    const float it = q == 0 ? inv_tau : inv_taud;
    float* pp = (q == 0 ? a.part : a.part_d) +
                ((int64_t)c.bh * a.chunks + c.chunk) * ((int64_t)D * a.G + a.G + 2 * a.nblk);
    if (wp == 0) {
      for (int s = 0; s < NP - 1; ++s)
#pragma unroll
        for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
          for (int d = 0; d < DB; ++d) dW[q][d][gb] += red[s][d][gb][lane];
#pragma unroll
          for (int r = 0; r < 4; ++r) dbv[gb][r] += redb[s][gb][r][j];
        }
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
        for (int d = 0; d < DB; ++d)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (c.g0 + 16 * gb + i < a.G)
              pp[(int64_t)(16 * d + 4 * j + r) * a.G + c.g0 + 16 * gb + i] = dW[q][d][gb][r] * it;
        if (i == 0)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (c.g0 + 16 * gb + 4 * j + r < a.G)
              pp[(int64_t)D * a.G + c.g0 + 16 * gb + 4 * j + r] = dbv[gb][r] * it;
      }
    }
    if (threadIdx.x == 0) {
      double s = 0.0;
      for (int w = 0; w < NP; ++w) s += dtw[q][w];
      *reinterpret_cast<double*>(pp + (int64_t)D * a.G + a.G + 2 * c.blk) = -s * (double)kLn2 * (double)it;
    }
    __syncthreads();  // the exchange buffers are reused by the second weight set
  }
}

template <bool COLN>
struct Run_k_bwd_b2_ {
  template <bool BF, int D, int GS, int NS, int NP, int PB>
  struct R {
    static hipError_t run(const PassCfg& cfg, int BH, const PassArgs& a, hipStream_t st) {
      if constexpr (NS != 1 || !bwd_b2_fits(BF, D, GS)) {
        return hipErrorInvalidConfiguration;
      } else {
        dim3 grid(cfg.chunks * BH * cfg.nblk);
        hipLaunchKernelGGL((k_bwd_b2<BF, D, GS, NS, NP, PB, COLN>), grid, dim3(64 * NS * NP), 0, st, a);
        return hipGetLastError();
      }
    }
  };
};

}  // namespace

bool fused_untied_bwd_b(const Geom& g) {
  const PassCfg cfg = pick_cfg(g, PASS_BWD_B);
  return cfg.NS == 1 && bwd_b2_fits(g.bf16, g.D, cfg.GS);
}

hipError_t run_pass_bwd_b2(const Geom& g, const PassArgs& a, bool coln, hipStream_t st) {
  if (coln) return run_pass_tilings<PASS_BWD_B, Run_k_bwd_b2_<true>::R>(g, a, st);
  return run_pass_tilings<PASS_BWD_B, Run_k_bwd_b2_<false>::R>(g, a, st);
}

}  // namespace fs
