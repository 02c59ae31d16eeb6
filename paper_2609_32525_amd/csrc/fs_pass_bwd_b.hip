// Streaming pass: backward pass B (point gradients and parameter partials), and its
// slot-owned parameter half in the slot-blocked family (PM: the per-point correction c and
// the weighted logit mean tb come from the point-owned pass; dx and dfx are not written).
// Kernel design and MFMA lane layouts are described at the top of fs_stream.h.

#include "fs_stream.h"

// bf16: the point groups' end-of-kernel reduction in the LDS of the loop's exchange buffers
// (1) or in an allocation of its own (0). fp32 keeps its own: with the smaller LDS footprint
// two workgroups fit a compute unit, and the kernel compiled for that spilled (head width 32,
// G = 64: pass B 1035 -> 1165 us).
#ifndef FS_BWDB_LDS_ALIAS
#define FS_BWDB_LDS_ALIAS 1
#endif
// bf16 head width 32: dW_s's point-ordered x operand from the loaded rows through LDS (1), or
// a second, point-by-point load of x (0).
#ifndef FS_BWDB_XT
#define FS_BWDB_XT 1
#endif

namespace fs {
namespace {

// =======================================================================================
// Backward pass B: point gradients and parameter partials
// partial layout per workgroup: [D * G] dW_s (row-major (D, G)), [G] dbias, [2] fp64 dtau
// PB: 16-point blocks per tile (1 or 2; bf16 needs 2: its contraction over points has K=32).
// ROLE: 0 the tied path (one set of weights feeds the slice and the deslice); in the untied
// variant, 1 is the slice weights' part (dw = F dU^T + ds; writes dfx and dx) and 2 the
// deslice weights' part (dw = dO zmix^T; adds its dx contribution to the dx already written);
// 3 is LinearNO's slice part: weights k = 2^(a - clse_g) normalised over the points of each
// slot, dw = F dz^T + ds with ds_g = -z_g . dz_g, and da = k dw (the per-slot correction is
// ds itself, so there is no per-point one; nor are the slot-mean shifts valid).
// With at most two slot groups, the per-head operands live in LDS as register images shared
// by the workgroup's wavefronts and are read where they are used, which keeps the register
// count (and so the number of resident wavefronts) in line with the other passes.
// =======================================================================================
template <bool BF, int D, int GS, int NS, int NP, int PB, bool PM, int ROLE>
__global__ __launch_bounds__(64 * NS * NP) __attribute__((amdgpu_waves_per_eu(PM ? FS_WPE_BWD_PM : BF ? FS_WPE_BWD_B : FS_WPE_BWD_B_F32))) void k_bwd_b(
    PassArgs a) {
  static_assert(PB == 2 || !BF, "bf16 contracts over 32 points");
  static_assert(!PM || (GS == 64 && NS == 1), "the parameter pass owns one 64-slot block");
  constexpr bool USE_DOUT = ROLE == 0 || ROLE == 2, USE_FX = ROLE != 2;
  constexpr bool COLN = ROLE == 3;  // weights normalised over the points of each slot
  constexpr int GB = GS / 16, VB = D / 16, DB = D / 16, TP = 16 * PB;
  constexpr bool SPLIT = BF;
  using T = typename Store<BF>::T;
  using SOp = SlotOp<BF, D, GB>;
  using UOp = GOp<BF, GB, VB>;
  using XOp = GOp<BF, GB, DB>;
  // operands in LDS when at most two slot groups share a tile and the images fit in 64 KB
  constexpr bool OPL =
      NS <= 2 && (size_t)NS * 64 * (3 * sizeof(SOp) + sizeof(UOp) + sizeof(XOp)) <= 65536;
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int wave = threadIdx.x >> 6, ws = wave % NS, wp = wave / NS;
  const HeadCtx c = head_ctx<D>(a, ws, GS);
  const int64_t rs = (int64_t)a.H * D;
  const T* xb = (const T*)a.x + c.off;
  const T* fb = (const T*)a.fx + c.off;
  const T* gb_ = (const T*)a.dout + c.off;
  T* dxb = (T*)a.out + c.off;
  T* dfb = (T*)a.out2 + c.off;
  const float* lse = a.lse_in + (int64_t)c.bh * a.N;
  const float inv_tau = 1.0f / a.tau[c.h];
  const float* zm = a.zmix + (int64_t)c.bh * a.G * D;
  const float* dU = a.dU + (int64_t)c.bh * a.G * D;

  // dw enters only through da = w (dw - sum_g w dw), which is unchanged when one vector is
  // added to every token of zmix or dU, or one constant to every ds_g (the weights sum to
  // one). Subtracting the mass-weighted slot means first keeps the rounding of these
  // operands relative to what actually differs between slots.
  const float* cen = a.cen + (int64_t)c.bh * (2 * D + 1);
  float bT[GB][4], dsT[GB][4];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      // padding blocks (slots >= G) read the last real block and take a masked logit, no ds
      bool real;
      const int sl = slot_block(c.g0 + 16 * gb, slot_lim(a), real) + 4 * j + r;
      const float bv = c.sc * c.bias[sl] - (COLN ? a.clse[(int64_t)c.bh * a.G + sl] : 0.f);
      const float dv = ROLE == 2 ? 0.f : a.ds[(int64_t)c.bh * a.G + sl] - (COLN ? 0.f : cen[2 * D]);
      bT[gb][r] = slot_mask(real, bv, kMaskedSlot);
      dsT[gb][r] = slot_mask(real, dv, 0.f);
    }

  // operands: W_s (logits), zmix and dU (dw, contraction over v), dU (dfx) and W_s / tau (dx)
  constexpr int kOpChunks = OPL ? 3 * lds_chunks<SOp>() + lds_chunks<UOp>() + lds_chunks<XOp>() : 1;
  __shared__ uint4 opl[OPL ? NS : 1][kOpChunks];
  SOp wop_r, zvop_r, uvop_r;
  UOp ugop_r;
  XOp wgop_r;
  {
    SOp t0, t1, t2;
    UOp t3;
    XOp t4;
    if (!OPL || wp == 0) {
      load_slotop<BF, D, GB, true, SPLIT>(t0, c.W, a.G, c.g0, slot_lim(a), c.sc, i, j);
      load_slotop<BF, D, GB, false, false>(t1, zm, D, c.g0, slot_lim(a), 1.0f, i, j, cen);
      load_slotop<BF, D, GB, false, false>(t2, dU, D, c.g0, slot_lim(a), 1.0f, i, j, COLN ? nullptr : cen + D);
      load_gop<BF, GB, VB, false>(t3, dU, D, c.g0, slot_lim(a), 1.0f, i, j);
      load_gop<BF, GB, DB, true>(t4, c.W, a.G, c.g0, slot_lim(a), inv_tau, i, j);
    }
    if constexpr (OPL) {
      uint4* b = opl[ws];
      if (wp == 0) {
        lds_put(t0, b, lane);
        lds_put(t1, b + lds_chunks<SOp>(), lane);
        lds_put(t2, b + 2 * lds_chunks<SOp>(), lane);
        lds_put(t3, b + 3 * lds_chunks<SOp>(), lane);
        lds_put(t4, b + 3 * lds_chunks<SOp>() + lds_chunks<UOp>(), lane);
      }
      __syncthreads();
    } else {
      wop_r = t0;
      zvop_r = t1;
      uvop_r = t2;
      ugop_r = t3;
      wgop_r = t4;
    }
  }
  const uint4* opb = opl[OPL ? ws : 0];
  auto get_w = [&](SOp& o) { if constexpr (OPL) lds_get(o, opb, lane); else o = wop_r; };
  auto get_zv = [&](SOp& o) { if constexpr (OPL) lds_get(o, opb + lds_chunks<SOp>(), lane); else o = zvop_r; };
  auto get_uv = [&](SOp& o) { if constexpr (OPL) lds_get(o, opb + 2 * lds_chunks<SOp>(), lane); else o = uvop_r; };
  auto get_ug = [&](UOp& o) { if constexpr (OPL) lds_get(o, opb + 3 * lds_chunks<SOp>(), lane); else o = ugop_r; };
  auto get_wg = [&](XOp& o) {
    if constexpr (OPL) lds_get(o, opb + 3 * lds_chunks<SOp>() + lds_chunks<UOp>(), lane); else o = wgop_r;
  };

  f4 dW[DB][GB];
  float dbacc[GB][4];
  double dtacc = 0.0;
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
    for (int r = 0; r < 4; ++r) dbacc[gb][r] = 0.f;
#pragma unroll
    for (int d = 0; d < DB; ++d) dW[d][gb] = zero4();
  }

  __shared__ float cx[NS > 1 ? NP : 1][NS > 1 ? NS : 1][2][TP];
  // The dfx / dx exchange buffer (NS > 1) and the per-wave da transpose buffer are never live
  // at the same time (a workgroup barrier separates every exchange from the transposes of
  // the previous and the next tile), so they share one LDS allocation.
  // gx: [NP][NS][VB][PB][64] f4; da transpose: fp32 [TP points][GS + 1], bf16 [GS slots][36].
  // bf16 tiles also stage dx and dfx there for whole-segment stores (store_tile_staged)
  constexpr bool STAGE = FS_BWDB_STAGE && BF && PB == 2 && D == VB * 16;
  constexpr int kDaWords = STAGE && kStageBytes<BF, D> / 4 > da_words<BF, GS, TP>() ? kStageBytes<BF, D> / 4
                                                                                    : da_words<BF, GS, TP>();
  constexpr size_t kGxBytes = NS > 1 ? (size_t)NP * NS * VB * PB * 64 * sizeof(f4) : 0;
  constexpr size_t kDaBytes = (size_t)NS * NP * kDaWords * sizeof(float);
  // the end-of-kernel reduction over the point groups reuses the same allocation
  constexpr size_t kRedBytes = NP > 1 ? (size_t)(NP - 1) * NS * DB * GB * 64 * sizeof(f4) +
                                            (size_t)(NP - 1) * NS * GB * 4 * 16 * sizeof(float)
                                      : 0;
  constexpr size_t kSmem0 = kGxBytes > kDaBytes ? kGxBytes : kDaBytes;
  constexpr bool kAlias = FS_BWDB_LDS_ALIAS && BF;
  __shared__ __attribute__((aligned(16))) char smem[kAlias && kRedBytes > kSmem0 ? kRedBytes : kSmem0];
  f4* gx = reinterpret_cast<f4*>(smem);
  float* myda = reinterpret_cast<float*>(smem) + (size_t)wave * kDaWords;
  // XT: bf16 with head width 32 forms dW_s's point-ordered x operand from the row operand the
  // logits already loaded, through this wavefront's LDS rows, instead of loading x again
  constexpr bool XT = FS_BWDB_XT && BF && D == 32 && PB == 2;
  constexpr int kXP = 80;  // LDS row pitch
  __shared__ __attribute__((aligned(16))) char xts[XT ? NS * NP : 1][XT ? 32 * kXP : 16];

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
  const auto rl = rows_rsrc(lse + pbeg, npts, 1, 1);
  const auto rc = rows_rsrc(PM ? a.cpt + ((int64_t)c.bh * a.N + pbeg) * 4 : a.Ws, npts, 4, 4);
  const int wpu = __builtin_amdgcn_readfirstlane(wp);

  struct Tile {
    RowOp<BF, D> xo[PB], go[PB], fo[PB];
    float lse2[PB];
    float l1;  // lse_load (bf16 tiles of the fused pass)
    float ct[PM ? PB : 1][2];
    f4 dx0[ROLE == 2 ? DB : 1][PB];  // the dx already written (untied deslice part)
    KGather<BF, DB, PB> xk;          // X again, points on the k index, for dW_s
  };
  auto load_tile = [&](Tile& tt, int t) {
    const int tb = (t * NP + wpu) * TP;
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int so = (tb + 16 * pb) * rsb;
      load_row_buf<BF, D>(tt.xo[pb], rx, i * rsb, so, j);
      if constexpr (USE_DOUT) load_row_buf<BF, D>(tt.go[pb], rg, i * rsb, so, j);
      if constexpr (USE_FX) load_row_buf<BF, D>(tt.fo[pb], rf, i * rsb, so, j);
      if constexpr (ROLE == 2) {
        if (ws == 0) {
#pragma unroll
          for (int cb = 0; cb < DB; ++cb)
            tt.dx0[cb][pb] = bld_row4<BF>(rdx, i * rsb + (16 * cb + 4 * j) * (int)sizeof(T), so);
        }
      }
      if constexpr (PM && !COLN) {
        // (c, tb, lse2) of the point as the point-owned pass wrote them
        const f4 rec = bld128(rc, 16 * i, 16 * (tb + 16 * pb));
        tt.ct[pb][0] = rec[0];
        tt.ct[pb][1] = rec[1];
        tt.lse2[pb] = tb + 16 * pb + i < npts ? rec[2] : kMasked;
      } else if constexpr (COLN || PB == 1) {
        const float l = COLN ? 0.f : bld32(rl, 4 * i, 4 * (tb + 16 * pb));
        tt.lse2[pb] = tb + 16 * pb + i < npts ? l : kMasked;
      }
    }
    if constexpr (!PM && !COLN && PB == 2) tt.l1 = lse_load(rl, tb, i, j);
    if constexpr (!XT) gather_k<BF, DB, PB>(tt.xk, rx, rsb, tb, i, j);
  };
  // fp32 with 64-slot waves has the longest tiles to cover: one more tile in flight there
  constexpr int PF = NS >= FS_NS_NOPF ? 0 : (!BF && GS == 64 && NS == 1 ? FS_PF_BWD_B + 1 : FS_PF_BWD_B);
  pipeline<PF, Tile>(ntile, load_tile, [&](Tile& cur, int t) {
    const int tp0 = (t * NP + wpu) * TP;
    const RowOp<BF, D>(&xo)[PB] = cur.xo;
    const RowOp<BF, D>(&go)[PB] = cur.go;
    const RowOp<BF, D>(&fo)[PB] = cur.fo;
    if constexpr (!PM && !COLN && PB == 2) lse_pair(cur.lse2, cur.l1, tp0, npts, i);
    const float(&lse2)[PB] = cur.lse2;
    // T-layout tiles: rows = slots g0 + 16 gb + 4 j + r, cols = points 16 pb + i
    f4 tl[GB][PB], w[GB][PB], dw[GB][PB];
    {
      SOp wop;
      get_w(wop);
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
#pragma unroll
        for (int pb = 0; pb < PB; ++pb) {
          f4 acc = f4{bT[gb][0], bT[gb][1], bT[gb][2], bT[gb][3]};
          acc = mm_slot_row<BF, D, GB, SPLIT>(wop, gb, xo[pb], acc);
          f4 tt, ww;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            tt[r] = acc[r] - lse2[pb];
            ww[r] = __builtin_amdgcn_exp2f(tt[r]);
          }
          tl[gb][pb] = tt;
          w[gb][pb] = ww;
        }
    }
    {
      SOp zv, uv;
      get_zv(zv);
      get_uv(uv);
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
#pragma unroll
        for (int pb = 0; pb < PB; ++pb) {
          f4 g = f4{dsT[gb][0], dsT[gb][1], dsT[gb][2], dsT[gb][3]};
          if constexpr (USE_DOUT) g = mm_slot_row<BF, D, GB, false>(zv, gb, go[pb], g);
          if constexpr (USE_FX) g = mm_slot_row<BF, D, GB, false>(uv, gb, fo[pb], g);
          dw[gb][pb] = g;
        }
    }
    // per point (column of the tile): c = sum_g w dw, the softmax correction, and
    // tb = sum_g w t, the weighted mean of the shifted base-2 logits t = a2 - lse2
    float cc[PB], tb[PB];
    if constexpr (COLN) {
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        cc[pb] = 0.f;
        tb[pb] = 0.f;
      }
    } else if constexpr (PM) {
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        cc[pb] = cur.ct[pb][0];
        tb[pb] = cur.ct[pb][1];
      }
    } else {
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      float sum = 0.f, st = 0.f;
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          sum += w[gb][pb][r] * dw[gb][pb][r];
          st += w[gb][pb][r] * tl[gb][pb][r];
        }
      cc[pb] = col4_sum(sum);
      tb[pb] = col4_sum(st);
    }
    if constexpr (NS > 1) {
      if (j == 0) {
#pragma unroll
        for (int pb = 0; pb < PB; ++pb) {
          cx[wp][ws][0][16 * pb + i] = cc[pb];
          cx[wp][ws][1][16 * pb + i] = tb[pb];
        }
      }
      __syncthreads();
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        float sum = 0.f, st = 0.f;
        for (int s = 0; s < NS; ++s) {
          sum += cx[wp][s][0][16 * pb + i];
          st += cx[wp][s][1][16 * pb + i];
        }
        cc[pb] = sum;
        tb[pb] = st;
      }
    }
    }
    // da = w (dw - c); dbias partials; dtau partial (App. F.2): sum_g da a = sum_g da (a - k)
    // for any per-point k because sum_g da = 0; with k = lse + tb the first-order effect of
    // the rounding of c on the sum cancels (sum_g w (t - tb) = 0).
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
          dbacc[gb][r] += da;
        }
    dtacc += (double)dts;
    if constexpr (!PM) {
    // dfx = w dU, dx = da W_s^T / tau (contractions over this wave's slots)
    f4 gf[VB][PB], gx_[DB][PB];
    {
      UOp ug;
      XOp wg;
      get_ug(ug);
      get_wg(wg);
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
          gf[vb][pb] = ROLE == 2 ? zero4() : mm_gop_tile<BF, GB, VB, PB>(ug, vb, w, pb, zero4());
#pragma unroll
        for (int d = 0; d < DB; ++d) gx_[d][pb] = mm_gop_tile<BF, GB, DB, PB>(wg, d, dw, pb, zero4());
      }
    }
    if constexpr (NS > 1) {
      __syncthreads();  // every wave has read cx and finished the previous da transposes
#pragma unroll
      for (int half = ROLE == 2 ? 1 : 0; half < 2; ++half) {
        f4(*src)[PB] = half == 0 ? gf : gx_;
        if (ws > 0) {
#pragma unroll
          for (int cb = 0; cb < VB; ++cb)
#pragma unroll
            for (int pb = 0; pb < PB; ++pb)
              gx[(((size_t)wp * NS + ws) * VB + cb) * (64 * PB) + pb * 64 + lane] = src[cb][pb];
        }
        __syncthreads();
        if (ws == 0) {
          for (int s = 1; s < NS; ++s)
#pragma unroll
            for (int cb = 0; cb < VB; ++cb)
#pragma unroll
              for (int pb = 0; pb < PB; ++pb)
                src[cb][pb] += gx[(((size_t)wp * NS + s) * VB + cb) * (64 * PB) + pb * 64 + lane];
        }
        __syncthreads();
      }
    }
    if (ws == 0) {
      if constexpr (STAGE) {
        // through this wavefront's da rows, which the transposes below overwrite afterwards
        char* sb = reinterpret_cast<char*>(myda);
        if constexpr (ROLE == 2) {
#pragma unroll
          for (int cb = 0; cb < DB; ++cb)
#pragma unroll
            for (int pb = 0; pb < PB; ++pb) gx_[cb][pb] += cur.dx0[cb][pb];
        } else {
          store_tile_staged<BF, D>(sb, gf, rdf, rsb, tp0, lane);
        }
        store_tile_staged<BF, D>(sb, gx_, rdx, rsb, tp0, lane);
      } else {
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
#pragma unroll
          for (int cb = 0; cb < VB; ++cb) {
            const int vo = i * rsb + (16 * cb + 4 * j) * (int)sizeof(T), so = (tp0 + 16 * pb) * rsb;
            if constexpr (ROLE == 2) {
              bst_row4<BF>(rdx, gx_[cb][pb] + cur.dx0[cb][pb], vo, so);
            } else {
              bst_row4<BF>(rdf, gf[cb][pb], vo, so);
              bst_row4<BF>(rdx, gx_[cb][pb], vo, so);
            }
          }
      }
    }
    }
    // dW_s += X^T da over the tile's points: da goes through LDS to put points on the k index.
    if constexpr (XT) {
      char* xt = xts[wave];
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
        *reinterpret_cast<bf8*>(xt + (16 * pb + i) * kXP + 16 * j) = xo[pb].v[0];
      wave_lds_sync();
#pragma unroll
      for (int d = 0; d < DB; ++d) {
        bf8 bt;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          bt[e] = *reinterpret_cast<const __bf16*>(xt + (16 * (e / 4) + 4 * j + (e % 4)) * kXP +
                                                   (16 * d + i) * 2);
        cur.xk.v[d] = bt;
      }
    }
    const KGather<BF, DB, PB>& XK = cur.xk;
    if constexpr (!BF) {
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r) myda[da_at<GS>(16 * pb + i, 16 * gb + 4 * j + r)] = dw[gb][pb][r];
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
            for (int d = 0; d < DB; ++d) dW[d][gb] = mfma_f32(xv[d], bv, dW[d][gb]);
          }
        }
      wave_lds_sync();
    } else {
      unsigned short* t16 = reinterpret_cast<unsigned short*>(myda);
      da_put_bf<GB, PB>(t16, dw, i, j);
      wave_lds_sync();
      const bf8(&xa)[DB] = XK.v;
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
        const bf8 bt = da_get_bf(t16, gb, i, j);
#pragma unroll
        for (int d = 0; d < DB; ++d) dW[d][gb] = mfma_bf16(xa[d], bt, dW[d][gb]);
      }
      wave_lds_sync();
    }
  });

  // ---- finish: reduce over lanes / waves and write the partial ---------------------------
  float dbv[GB][4];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb)
#pragma unroll
    for (int r = 0; r < 4; ++r) dbv[gb][r] = row16_sum(dbacc[gb][r]);
  // dtau: fp64 sum over the wave, then over all waves of the workgroup in a fixed order
  double dt = dtacc;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) dt += __shfl_xor(dt, off);
  __shared__ double dtw[NS * NP];
  if (lane == 0) dtw[wave] = dt;

  float* pp = a.part + ((int64_t)c.bh * a.chunks + c.chunk) * ((int64_t)D * a.G + a.G + 2 * a.nblk);
  if constexpr (NP > 1) {
    constexpr int kRed = (NP - 1) * NS * DB * GB * 64, kRedb = (NP - 1) * NS * GB * 4 * 16;
    __shared__ f4 red_own[kAlias ? 1 : kRed];
    __shared__ float redb_own[kAlias ? 1 : kRedb];
    if constexpr (kAlias) __syncthreads();  // every wave is done with the loop's buffers
    f4* redp = kAlias ? reinterpret_cast<f4*>(smem) : red_own;
    float* redbp = kAlias ? reinterpret_cast<float*>(smem + (size_t)kRed * sizeof(f4)) : redb_own;
    auto& red = *reinterpret_cast<f4(*)[NP - 1][NS][DB][GB][64]>(redp);
    auto& redb = *reinterpret_cast<float(*)[NP - 1][NS][GB][4][16]>(redbp);
    if (wp > 0) {
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
        for (int d = 0; d < DB; ++d) red[wp - 1][ws][d][gb][lane] = dW[d][gb];
        if (i == 0)
#pragma unroll
          for (int r = 0; r < 4; ++r) redb[wp - 1][ws][gb][r][j] = dbv[gb][r];
      }
    }
    __syncthreads();
    if (wp == 0) {
      for (int q = 0; q < NP - 1; ++q)
#pragma unroll
        for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
          for (int d = 0; d < DB; ++d) dW[d][gb] += red[q][ws][d][gb][lane];
#pragma unroll
          for (int r = 0; r < 4; ++r) dbv[gb][r] += redb[q][ws][gb][r][j];
        }
    }
  } else {
    __syncthreads();
  }
  if (wp == 0) {
#pragma unroll
    for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (c.g0 + 16 * gb + i < a.G)
            pp[(int64_t)(16 * d + 4 * j + r) * a.G + c.g0 + 16 * gb + i] = dW[d][gb][r] * inv_tau;
      if (i == 0)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (c.g0 + 16 * gb + 4 * j + r < a.G)
            pp[(int64_t)D * a.G + c.g0 + 16 * gb + 4 * j + r] = dbv[gb][r] * inv_tau;
    }
  }
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int q = 0; q < NS * NP; ++q) s += dtw[q];
    // (D * G + G) is even, so this slot is 8-byte aligned
    *reinterpret_cast<double*>(pp + (int64_t)D * a.G + a.G + 2 * c.blk) =
        -s * (double)kLn2 * (double)inv_tau;
  }
}

template <bool PM, int ROLE>
struct Run_k_bwd_b_ {
  template <bool BF, int D, int GS, int NS, int NP, int PB>
  struct R {
    static hipError_t run(const PassCfg& cfg, int BH, const PassArgs& a, hipStream_t st) {
      // the parameter half of the blocked family is slot-owned: 64-slot blocks (head width up
      // to 32 for the roles other than 0)
      if constexpr (PM && (NS != 1 || GS != 64 || (ROLE != 0 && D > 32))) {
        return hipErrorInvalidConfiguration;
      } else {
        dim3 grid(cfg.chunks * BH * cfg.nblk);
        hipLaunchKernelGGL((k_bwd_b<BF, D, GS, NS, NP, PB, PM, ROLE>), grid, dim3(64 * NS * NP), 0,
                           st, a);
        return hipGetLastError();
      }
    }
  };
};

}  // namespace

hipError_t run_pass_bwd_b(const Geom& g, const PassArgs& a, hipStream_t st) {
  return run_pass_tilings<PASS_BWD_B, Run_k_bwd_b_<false, 0>::R>(g, a, st);
}

hipError_t run_pass_bwd_params(const Geom& g, const PassArgs& a, int role, hipStream_t st) {
  switch (role) {
    case 0: return run_pass_tilings<PASS_BWD_B, Run_k_bwd_b_<true, 0>::R>(g, a, st);
    case 1: return run_pass_tilings<PASS_BWD_B, Run_k_bwd_b_<true, 1>::R>(g, a, st);
    case 2: return run_pass_tilings<PASS_BWD_B, Run_k_bwd_b_<true, 2>::R>(g, a, st);
    case 3: return run_pass_tilings<PASS_BWD_B, Run_k_bwd_b_<true, 3>::R>(g, a, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t run_pass_bwd_b_untied(const Geom& g, const PassArgs& a, int role, hipStream_t st) {
  if (role == 1) return run_pass_tilings<PASS_BWD_B, Run_k_bwd_b_<false, 1>::R>(g, a, st);
  if (role == 2) return run_pass_tilings<PASS_BWD_B, Run_k_bwd_b_<false, 2>::R>(g, a, st);
  if (role == 3) return run_pass_tilings<PASS_BWD_B, Run_k_bwd_b_<false, 3>::R>(g, a, st);
  return hipErrorInvalidValue;
}

}  // namespace fs
