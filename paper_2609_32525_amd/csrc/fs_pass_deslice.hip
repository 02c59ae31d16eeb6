// Streaming pass: deslice (logits, w = exp2(a - lse), out = w zmix), and the deslice that
// computes the per-point softmax statistics itself (no lse input; optionally writes lse).
// Kernel design and MFMA lane layouts are described at the top of fs_stream.h.

#include "fs_stream.h"

// Output tiles staged through LDS for whole-segment 16-byte stores (1) or stored straight
// from the MFMA result layout, 4 values per lane (0).
// Block images of the point-owned deslice: a ring of four (4) or two buffers (2).
#ifndef FS_DESLICE_PT_RING
#define FS_DESLICE_PT_RING 4
#endif
#ifndef FS_DESLICE_STAGE
#define FS_DESLICE_STAGE 1
#endif


namespace fs {
namespace {

// =======================================================================================
// Deslice pass. ST: the normaliser of every point is computed here from the logits (max and
// sum over the slot groups, combined across the NS slot waves through LDS) instead of read.
// =======================================================================================
template <bool BF, int D, int GS, int NS, int NP, bool ST>
__global__ __launch_bounds__(64 * NS * NP) __attribute__((amdgpu_waves_per_eu(D <= 32 ? FS_WPE_DESLICE : 1))) void k_deslice(
    PassArgs a) {
  constexpr int GB = GS / 16, VB = D / 16;
  constexpr bool SPLIT = BF;
  using T = typename Store<BF>::T;
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int wave = threadIdx.x >> 6, ws = wave % NS, wp = wave / NS;
  const HeadCtx c = head_ctx<D>(a, ws, GS);
  const int64_t rs = (int64_t)a.H * D;
  const T* xb = (const T*)a.x + c.off;
  T* ob = (T*)a.out + c.off;
  const float* lse = (ST ? a.lse_out : a.lse_in) + (int64_t)c.bh * a.N;
  const bool want_lse = !ST || a.lse_out != nullptr;

  SlotOp<BF, D, GB> wop;
  load_slotop<BF, D, GB, true, SPLIT>(wop, c.W, a.G, c.g0, slot_lim(a), c.sc, i, j);
  float bT[GB][4];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb)
#pragma unroll
    for (int r = 0; r < 4; ++r) bT[gb][r] = slot_bias(c, a, c.g0 + 16 * gb, 4 * j + r);
  GOp<BF, GB, VB> zop;
  load_gop<BF, GB, VB, false>(zop, a.zmix + (int64_t)c.bh * a.G * D, D, c.g0, slot_lim(a), 1.0f, i, j);

  __shared__ f4 ox[NS > 1 ? NP : 1][NS > 1 ? NS : 1][VB][2][64];
  // output staging: one 32-point tile per point group (store_tile_staged)
  __shared__ __attribute__((aligned(16))) char ostage[FS_DESLICE_STAGE ? NP : 1][FS_DESLICE_STAGE ? kStageBytes<BF, D> : 16];
  constexpr int SX = ST && NS > 1;
  __shared__ float st_m[SX ? 2 : 1][SX ? NP : 1][SX ? NS : 1][32];
  __shared__ float st_l[SX ? 2 : 1][SX ? NP : 1][SX ? NS : 1][32];

  const int64_t pbeg = (int64_t)c.chunk * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int npts = pend > pbeg ? (int)(pend - pbeg) : 0;
  const int ntile = (npts + 32 * NP - 1) / (32 * NP);
  const int rsb = (int)(rs * sizeof(T));
  const auto rx = rows_rsrc(xb + pbeg * rs, npts, (int)rs, D);
  const auto ro = rows_rsrc(ob + pbeg * rs, npts, (int)rs, D);
  const auto rl = rows_rsrc(want_lse ? lse + pbeg : a.Ws, npts, 1, 1);
  const int wpu = __builtin_amdgcn_readfirstlane(wp);

  struct Tile {
    RowOp<BF, D> xo[2];
    float lse2[2];
  };
  auto load_tile = [&](Tile& tt, int t) {
    const int tb = (t * NP + wpu) * 32;
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      load_row_buf<BF, D>(tt.xo[pb], rx, i * rsb, (tb + 16 * pb) * rsb, j);
      if constexpr (!ST) {
        const float l = bld32(rl, 4 * i, 4 * (tb + 16 * pb));
        tt.lse2[pb] = tb + 16 * pb + i < npts ? l : kMasked;
      }
    }
  };
  auto body = [&](const RowOp<BF, D>* xo, [[maybe_unused]] const float* lse2, int t) {
    const int tb = (t * NP + wpu) * 32;
    f4 w[GB][2];
#pragma unroll
    for (int gb = 0; gb < GB; ++gb)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) {
        f4 acc = f4{bT[gb][0], bT[gb][1], bT[gb][2], bT[gb][3]};
        acc = mm_slot_row<BF, D, GB, SPLIT>(wop, gb, xo[pb], acc);
        if constexpr (!ST) {
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[r] = __builtin_amdgcn_exp2f(acc[r] - lse2[pb]);
        }
        w[gb][pb] = acc;
      }
    if constexpr (ST) {
      // T-layout: lane (i, j) holds slots 4 j + r of point 16 pb + i; reduce over gb and r in
      // the lane, over j across the four 16-lane rows, then over the slot waves
      float m[2], l[2];
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) {
        float mx = w[0][pb][0];
#pragma unroll
        for (int gb = 0; gb < GB; ++gb)
#pragma unroll
          for (int r = 0; r < 4; ++r) mx = vmax(mx, w[gb][pb][r]);
        m[pb] = col4_max(mx);
        float sum = 0.f;
#pragma unroll
        for (int gb = 0; gb < GB; ++gb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float e = __builtin_amdgcn_exp2f(w[gb][pb][r] - m[pb]);
            w[gb][pb][r] = e;
            sum += e;
          }
        l[pb] = col4_sum(sum);
      }
      float f[2], ls2[2];
      if constexpr (NS == 1) {
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
          f[pb] = __builtin_amdgcn_rcpf(l[pb]);
          ls2[pb] = m[pb] + __log2f(l[pb]);
        }
      } else {
        const int par = t & 1;
        if (j == 0) {
#pragma unroll
          for (int pb = 0; pb < 2; ++pb) {
            st_m[par][wp][ws][16 * pb + i] = m[pb];
            st_l[par][wp][ws][16 * pb + i] = l[pb];
          }
        }
        __syncthreads();
        // lane p < 32 combines the slot waves' statistics of point p; every lane then fetches
        // the combined values of its own points
        float Mp = st_m[par][wp][0][lane & 31];
#pragma unroll
        for (int s = 1; s < NS; ++s) Mp = vmax(Mp, st_m[par][wp][s][lane & 31]);
        float Lp = 0.f;
#pragma unroll
        for (int s = 0; s < NS; ++s)
          Lp += st_l[par][wp][s][lane & 31] * __builtin_amdgcn_exp2f(st_m[par][wp][s][lane & 31] - Mp);
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
          const float M = __shfl(Mp, 16 * pb + i);
          const float L = __shfl(Lp, 16 * pb + i);
          f[pb] = __builtin_amdgcn_exp2f(m[pb] - M) * __builtin_amdgcn_rcpf(L);
          ls2[pb] = M + __log2f(L);
        }
      }
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) {
#pragma unroll
        for (int gb = 0; gb < GB; ++gb) w[gb][pb] *= f[pb];
        if (want_lse && ws == 0 && j == 0) bst32(rl, ls2[pb], 4 * (16 * pb + i), 4 * tb);
      }
    }
    f4 o[VB][2];
    const TileB<BF, GB, 2> wt = tile_b<BF, GB, 2>(w);
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) o[vb][pb] = mm_gop_b<BF, GB, VB, 2>(zop, vb, wt, pb, zero4());

    if constexpr (NS > 1) {
      if (ws > 0) {
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
#pragma unroll
          for (int pb = 0; pb < 2; ++pb) ox[wp][ws][vb][pb][lane] = o[vb][pb];
      }
      __syncthreads();
      if (ws == 0) {
        for (int s = 1; s < NS; ++s)
#pragma unroll
          for (int vb = 0; vb < VB; ++vb)
#pragma unroll
            for (int pb = 0; pb < 2; ++pb) o[vb][pb] += ox[wp][s][vb][pb][lane];
      }
      __syncthreads();
    }
    if (ws == 0) {
      if constexpr (FS_DESLICE_STAGE) {
        store_tile_staged<BF, D>(ostage[wp], o, ro, rsb, tb, lane);
      } else {
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
          for (int vb = 0; vb < VB; ++vb)
            bst_row4<BF>(ro, o[vb][pb], i * rsb + (16 * vb + 4 * j) * (int)sizeof(T), (tb + 16 * pb) * rsb);
      }
    }
  };
  pipeline<(NS >= FS_NS_NOPF ? 0 : FS_PF_DESLICE), Tile>(
      ntile, load_tile, [&](Tile& cur, int t) { body(cur.xo, cur.lse2, t); });
}


// =======================================================================================
// Point-owned deslice of the slot-blocked family (G > 128): every wavefront owns a 32-point
// tile per step and sweeps all slot blocks, out += w z' per block, with no exchange between
// wavefronts. A block's operand images (W_s scaled by log2(e)/tau, split in two bf16 parts;
// z' as the contraction-over-slots operand; the scaled bias), in halves of 32 slots, are
// built by four of the workgroup's wavefronts into the free half of a double-buffered LDS
// area while the block before is computed (one part each; the loads go out before the
// block's arithmetic, the LDS writes after it). ST: the normaliser is computed in the same
// sweep, online: a running maximum per point, with the sum and the output accumulator
// rescaled whenever the maximum grows.
// =======================================================================================
template <bool BF, int D>
struct DesliceImages {
  static constexpr int GBH = 2, VB = D / 16;
  using SOp = SlotOp<BF, D, GBH>;
  using ZOp = GOp<BF, GBH, VB>;
  static constexpr int kW = lds_chunks<SOp>(), kZ = lds_chunks<ZOp>();
  // [W half 0][W half 1][z' half 0][z' half 1][64 scaled biases]
  static constexpr int kChunks = 2 * kW + 2 * kZ + 64 / 4;
};

template <bool BF, int D, int NW, bool ST>
__global__ __launch_bounds__(64 * NW) void k_deslice_pt(PassArgs a) {
  static_assert(NW >= 4, "four wavefronts build the image parts of a block");
  using IM = DesliceImages<BF, D>;
  using SOp = typename IM::SOp;
  using ZOp = typename IM::ZOp;
  constexpr int GBH = IM::GBH, VB = IM::VB;
  using T = typename Store<BF>::T;
  // block images: a ring of four (blocks built two ahead, a workgroup barrier after every
  // second block) or two (one ahead, a barrier after every block; head width 64, whose two
  // workgroups per compute unit would not fit four)
  constexpr int RING = FS_DESLICE_PT_RING == 4 && D <= 32 ? 4 : 2, LA = RING / 2;
  __shared__ uint4 img[RING][IM::kChunks];
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int wpu = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const HeadCtx c = head_ctx<D>(a, 0, 0);
  const int NB = (a.G + 63) / 64;
  const int64_t rs = (int64_t)a.H * D;
  const T* xb = (const T*)a.x + c.off;
  T* ob = (T*)a.out + c.off;
  const float* lse = (ST ? a.lse_out : a.lse_in) + (int64_t)c.bh * a.N;
  const bool want_lse = !ST || a.lse_out != nullptr;
  const float* zm = a.zmix + (int64_t)c.bh * a.G * D;

  const int64_t pbeg = (int64_t)c.chunk * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int npts = pend > pbeg ? (int)(pend - pbeg) : 0;
  const int nstep = (npts + 32 * NW - 1) / (32 * NW);
  const int rsb = (int)(rs * sizeof(T));
  const auto rx = rows_rsrc(xb + pbeg * rs, npts, (int)rs, D);
  const auto ro = rows_rsrc(ob + pbeg * rs, npts, (int)rs, D);
  const auto rl = rows_rsrc(want_lse ? lse + pbeg : a.Ws, npts, 1, 1);

  // this wavefront's part of a block image: W half (waves 0, 1), z' half (2, 3), bias (0)
  SOp wpart;
  ZOp zpart;
  float bpart = 0.f;
  auto build = [&](int blk) {
    const int g0 = 64 * blk;
    if (wpu < 2) load_slotop<BF, D, GBH, true, BF>(wpart, c.W, a.G, g0 + 32 * wpu, slot_lim(a), c.sc, i, j);
    else if (wpu < 4) load_gop<BF, GBH, VB, false>(zpart, zm, D, g0 + 32 * (wpu - 2), slot_lim(a), 1.0f, i, j);
    if (wpu == 0) bpart = slot_bias_at(c, a, g0 + lane);
  };
  auto put = [&](uint4* dst) {
    if (wpu < 2) lds_put(wpart, dst + wpu * IM::kW, lane);
    else if (wpu < 4) lds_put(zpart, dst + 2 * IM::kW + (wpu - 2) * IM::kZ, lane);
    if (wpu == 0) reinterpret_cast<float*>(dst + 2 * IM::kW + 2 * IM::kZ)[lane] = bpart;
  };

  if (nstep == 0) return;  // uniform over the workgroup
  const int nu = nstep * NB;  // block visits, u = step NB + blk
#pragma unroll
  for (int u = 0; u < LA; ++u)
    if (u < nu) {
      build(u % NB);
      put(img[u]);
    }
  __syncthreads();
  int u = 0;
  for (int step = 0; step < nstep; ++step) {
    const int tb = (step * NW + wpu) * 32;
    RowOp<BF, D> xo[2];
    float lse2[2] = {0.f, 0.f};
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      load_row_buf<BF, D>(xo[pb], rx, i * rsb, (tb + 16 * pb) * rsb, j);
      if constexpr (!ST) {
        const float l = bld32(rl, 4 * i, 4 * (tb + 16 * pb));
        lse2[pb] = tb + 16 * pb + i < npts ? l : kMasked;
      }
    }
    // lane (i, j): point 16 pb + i; o[vb][pb] holds its outputs 16 vb + 4 j + r
    f4 o[VB][2];
    float m[2] = {-INFINITY, -INFINITY}, l[2] = {0.f, 0.f};
#pragma unroll
    for (int vb = 0; vb < VB; ++vb) o[vb][0] = o[vb][1] = zero4();
    for (int blk = 0; blk < NB; ++blk) {
      const bool more = u + LA < nu;
      if (more) build(blk + LA < NB ? blk + LA : blk + LA - NB);
      const uint4* cbuf = img[u % RING];
      const float* bS = reinterpret_cast<const float*>(cbuf + 2 * IM::kW + 2 * IM::kZ);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        // T-layout logits: rows = slots 32 h + 16 gb + 4 j + r of the block, cols = points
        f4 w[GBH][2];
        {
          SOp wop;
          lds_get(wop, cbuf + h * IM::kW, lane);
#pragma unroll
          for (int gb = 0; gb < GBH; ++gb) {
            const f4 bT = *reinterpret_cast<const f4*>(bS + 32 * h + 16 * gb + 4 * j);
#pragma unroll
            for (int pb = 0; pb < 2; ++pb) w[gb][pb] = mm_slot_row<BF, D, GBH, BF>(wop, gb, xo[pb], bT);
          }
        }
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
          if constexpr (ST) {
            float bm = w[0][pb][0];
#pragma unroll
            for (int gb = 0; gb < GBH; ++gb)
#pragma unroll
              for (int r = 0; r < 4; ++r) bm = vmax(bm, w[gb][pb][r]);
            const float mn = vmax(m[pb], col4_max(bm));
            const float f = __builtin_amdgcn_exp2f(m[pb] - mn);
            m[pb] = mn;
            float sum = 0.f;
#pragma unroll
            for (int gb = 0; gb < GBH; ++gb)
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const float e = __builtin_amdgcn_exp2f(w[gb][pb][r] - mn);
                w[gb][pb][r] = e;
                sum += e;
              }
            l[pb] = l[pb] * f + col4_sum(sum);
#pragma unroll
            for (int vb = 0; vb < VB; ++vb) o[vb][pb] *= f;
          } else {
#pragma unroll
            for (int gb = 0; gb < GBH; ++gb)
#pragma unroll
              for (int r = 0; r < 4; ++r) w[gb][pb][r] = __builtin_amdgcn_exp2f(w[gb][pb][r] - lse2[pb]);
          }
        }
        ZOp zop;
        lds_get(zop, cbuf + 2 * IM::kW + h * IM::kZ, lane);
        const TileB<BF, GBH, 2> wt = tile_b<BF, GBH, 2>(w);
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
#pragma unroll
          for (int pb = 0; pb < 2; ++pb) o[vb][pb] = mm_gop_b<BF, GBH, VB, 2>(zop, vb, wt, pb, o[vb][pb]);
      }
      if (more) put(img[(u + LA) % RING]);
      // with the ring of four the buffer written here held block u - 2, which every
      // wavefront finished before the barrier after block u - 1 (u even) or u - 2 (u odd)
      if (RING == 2 || (u & 1)) __syncthreads();
      ++u;
    }
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      if constexpr (ST) {
        const float inv = __builtin_amdgcn_rcpf(l[pb]);
#pragma unroll
        for (int vb = 0; vb < VB; ++vb) o[vb][pb] *= inv;
        if (want_lse && j == 0) bst32(rl, m[pb] + __log2f(l[pb]), 4 * i, 4 * (tb + 16 * pb));
      }
#pragma unroll
      for (int vb = 0; vb < VB; ++vb)
        bst_row4<BF>(ro, o[vb][pb], i * rsb + (16 * vb + 4 * j) * (int)sizeof(T), (tb + 16 * pb) * rsb);
    }
  }
}

template <bool ST>
struct Run_k_deslice_ {
  template <bool BF, int D, int GS, int NS, int NP, int PB>
  struct R {
    static hipError_t run(const PassCfg& cfg, int BH, const PassArgs& a, hipStream_t st) {
      dim3 grid(cfg.chunks * BH * cfg.nblk);
      hipLaunchKernelGGL((k_deslice<BF, D, GS, NS, NP, ST>), grid, dim3(64 * NS * NP), 0, st, a);
      return hipGetLastError();
    }
  };
};

}  // namespace

namespace {
template <bool ST>
hipError_t run_deslice_pt(const Geom& g, const PassArgs& a, hipStream_t st) {
  // the point-owned chunking with this kernel's wavefront count: each workgroup sweeps its
  // chunk in steps of 32 nw points
  const int nw = deslice_pt_waves(g);
  const PassCfg cfg = pick_cfg(g, PASS_POINT, nw);
  if (cfg.NP != nw) return hipErrorInvalidConfiguration;
  const dim3 grid(cfg.chunks * g.BH()), block(64 * nw);
#define FS_DPT(BF_, D_, NW_)                                                              \
  {                                                                                       \
    hipLaunchKernelGGL((k_deslice_pt<BF_, D_, NW_, ST>), grid, block, 0, st, a);          \
    return hipGetLastError();                                                             \
  }
  if (g.bf16 && g.D == 16) FS_DPT(true, 16, FS_DESLICE_PT_WAVES)
  if (g.bf16 && g.D == 32) FS_DPT(true, 32, FS_DESLICE_PT_WAVES)
  if (g.bf16 && g.D == 64) FS_DPT(true, 64, FS_POINT_WAVES_WIDE)
  if (!g.bf16 && g.D == 16) FS_DPT(false, 16, FS_DESLICE_PT_WAVES)
  if (!g.bf16 && g.D == 32) FS_DPT(false, 32, FS_DESLICE_PT_WAVES)
#undef FS_DPT
  return hipErrorInvalidConfiguration;
}
}  // namespace

hipError_t run_pass_deslice(const Geom& g, const PassArgs& a, hipStream_t st) {
  // the slot-blocked family: point-owned, slot blocks streamed (with the normaliser computed
  // online when none is given); a carries the point-owned passes' chunking
  if (deslice_point_owned(g))
    return a.lse_in == nullptr ? run_deslice_pt<true>(g, a, st) : run_deslice_pt<false>(g, a, st);
  if (a.lse_in == nullptr) return run_pass_tilings<PASS_DESLICE, Run_k_deslice_<true>::R>(g, a, st);
  return run_pass_tilings<PASS_DESLICE, Run_k_deslice_<false>::R>(g, a, st);
}

}  // namespace fs
