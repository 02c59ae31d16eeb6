// Streaming pass: backward pass A (dzmix partials = w^T dout), and the slot-owned slice of
// the slot-blocked family (U partials = w^T fx and s partials = sum w, with the per-point
// softmax statistics from the statistics pass).
// Kernel design and MFMA lane layouts are described at the top of fs_stream.h.

#include "fs_stream.h"

// bf16 head width 32: backward pass A (and the slot-owned slice) load dout / fx as rows and
// form the point-ordered operand through LDS (1), or gather it point by point (0).
#ifndef FS_BWDA_T
#define FS_BWDA_T 1
#endif

namespace fs {
namespace {

// =======================================================================================
// Backward pass A: dzmix = w^T dout (partials per workgroup). SL: the same contraction with
// fx in place of dout, plus the weight sums s (the slot-owned slice).
// =======================================================================================
template <bool BF, int D, int GS, int NS, int NP, bool SL>
__global__ __launch_bounds__(64 * NS * NP) __attribute__((amdgpu_waves_per_eu(D > 32 ? 1 : FS_WPE_BWD_A))) void k_bwd_a(
    PassArgs a) {
  constexpr int GB = GS / 16, VB = D / 16;
  constexpr bool SPLIT = BF;
  using T = typename Store<BF>::T;
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int wave = threadIdx.x >> 6, ws = wave % NS, wp = wave / NS;
  const HeadCtx c = head_ctx<D>(a, ws, GS);
  const int64_t rs = (int64_t)a.H * D;
  const T* xb = (const T*)a.x + c.off;
  const T* db = (const T*)(SL ? a.fx : a.dout) + c.off;
  const float* lse = a.lse_in + (int64_t)c.bh * a.N;

  SlotOp<BF, D, GB> wop;
  load_slotop<BF, D, GB, true, SPLIT>(wop, c.W, a.G, c.g0, slot_lim(a), c.sc, i, j);
  float bS[GB];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) bS[gb] = slot_bias(c, a, c.g0 + 16 * gb, i);
  f4 Z[GB][VB];
  float sacc[GB];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) {
    sacc[gb] = 0.f;
#pragma unroll
    for (int vb = 0; vb < VB; ++vb) Z[gb][vb] = zero4();
  }

  const int64_t pbeg = (int64_t)c.chunk * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int npts = pend > pbeg ? (int)(pend - pbeg) : 0;
  const int ntile = (npts + 32 * NP - 1) / (32 * NP);
  const int rsb = (int)(rs * sizeof(T));
  const auto rx = rows_rsrc(xb + pbeg * rs, npts, (int)rs, D);
  const auto rg = rows_rsrc(db + pbeg * rs, npts, (int)rs, D);
  const auto rl = rows_rsrc(lse + pbeg, npts, 1, 1);
  const int wpu = __builtin_amdgcn_readfirstlane(wp);

  // TR: bf16 dout (or fx) tiles arrive as rows, 16 bytes per lane like x, and are turned into
  // the point-ordered k-operand through this wavefront's LDS rows; lse arrives one value per
  // point and is spread over the lanes by shuffles.
  constexpr bool TR = FS_BWDA_T && BF && D == 32 && NS == 1;
  constexpr int kTP = 80;  // LDS row pitch (64 bytes of a head row + 16)
  __shared__ __attribute__((aligned(16))) char trs[TR ? NP : 1][TR ? 32 * kTP : 16];
  struct Tile {
    RowOp<BF, D> xo[2];
    float lse2[2][4];
    PtGather<BF, VB> g;
    uint4 grow[TR ? 2 : 1];
    float l1;  // TR: lse of point 16 (j % 2) + i of the tile
  };
  auto load_tile = [&](Tile& tt, int t) {
    const int tb = (t * NP + wpu) * 32;
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      load_row_buf<BF, D>(tt.xo[pb], rx, i * rsb, (tb + 16 * pb) * rsb, j);
      if constexpr (TR) {
        tt.grow[pb] = bld128u(rg, i * rsb + 16 * j, (tb + 16 * pb) * rsb);
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float l = bld32(rl, 4 * (4 * j + r), 4 * (tb + 16 * pb));
          tt.lse2[pb][r] = tb + 16 * pb + 4 * j + r < npts ? l : kMasked;
        }
      }
    }
    if constexpr (TR) {
      // the tile's 32 normalisers in one load, spread over the lanes by shuffles
      const int p = 16 * (j & 1) + i;
      const float l = bld32(rl, 4 * p, 4 * tb);
      tt.l1 = tb + p < npts ? l : kMasked;
    } else {
      gather_points_buf<BF, VB>(tt.g, rg, rsb, tb * rsb, i, j);
    }
  };
  pipeline<(NS >= FS_NS_NOPF ? 0 : FS_PF_BWD_A), Tile>(ntile, load_tile, [&](Tile& cur, int t) {
    const RowOp<BF, D>* xo = cur.xo;
    if constexpr (TR) {
      char* tr = trs[wp];
      wave_lds_sync();
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
        *reinterpret_cast<uint4*>(tr + (16 * pb + i) * kTP + 16 * j) = cur.grow[pb];
      wave_lds_sync();
#pragma unroll
      for (int cb = 0; cb < VB; ++cb) {
        bf8 bt;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          bt[e] = *reinterpret_cast<const __bf16*>(tr + (16 * (e / 4) + 4 * j + (e % 4)) * kTP +
                                                   (16 * cb + i) * 2);
        cur.g.v[cb] = bt;
      }
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) cur.lse2[pb][r] = __shfl(cur.l1, 16 * pb + 4 * j + r);
    }
    const float(*lse2)[4] = cur.lse2;
    f4 w[2][GB];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
        f4 acc = mm_row_slot<BF, D, GB, SPLIT>(xo[pb], wop, gb, splat4(bS[gb]));
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] = __builtin_amdgcn_exp2f(acc[r] - lse2[pb][r]);
        w[pb][gb] = acc;
      }
    if constexpr (SL) {
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
        float sum = 0.f;
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r) sum += w[pb][gb][r];
        sacc[gb] += sum;
      }
    }
    mm_points<BF, GB, VB>(Z, w, cur.g);
  });
  if constexpr (SL) {
#pragma unroll
    for (int gb = 0; gb < GB; ++gb) sacc[gb] = col4_sum(sacc[gb]);
  }

  float* pZ = a.part + ((int64_t)c.bh * a.chunks + c.chunk) * a.G * D;
  if constexpr (NP > 1) {
    __shared__ f4 red[NP - 1][NS][GB][VB][64];
    __shared__ float reds[SL ? NP - 1 : 1][NS][GB][16];
    if (wp > 0) {
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
        for (int vb = 0; vb < VB; ++vb) red[wp - 1][ws][gb][vb][lane] = Z[gb][vb];
        if (SL && j == 0) reds[SL ? wp - 1 : 0][ws][gb][i] = sacc[gb];
      }
    }
    __syncthreads();
    if (wp == 0) {
      for (int q = 0; q < NP - 1; ++q)
#pragma unroll
        for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
          for (int vb = 0; vb < VB; ++vb) Z[gb][vb] += red[q][ws][gb][vb][lane];
          if constexpr (SL) sacc[gb] += reds[q][ws][gb][i];
        }
    }
  }
  if (wp == 0) {
#pragma unroll
    for (int gb = 0; gb < GB; ++gb)
#pragma unroll
      for (int vb = 0; vb < VB; ++vb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int g = c.g0 + 16 * gb + 4 * j + r;
          if (g < a.G) pZ[(int64_t)g * D + 16 * vb + i] = Z[gb][vb][r];
        }
    if constexpr (SL) {
      float* pS = a.part2 + ((int64_t)c.bh * a.chunks + c.chunk) * a.G;
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
        if (j == 0 && c.g0 + 16 * gb + i < a.G) pS[c.g0 + 16 * gb + i] = sacc[gb];
    }
  }
}

template <bool SL>
struct Run_k_bwd_a_ {
  template <bool BF, int D, int GS, int NS, int NP, int PB>
  struct R {
    static hipError_t run(const PassCfg& cfg, int BH, const PassArgs& a, hipStream_t st) {
      if constexpr (SL && NS != 1) {  // the slice of the blocked family is slot-owned
        return hipErrorInvalidConfiguration;
      } else {
        dim3 grid(cfg.chunks * BH * cfg.nblk);
        hipLaunchKernelGGL((k_bwd_a<BF, D, GS, NS, NP, SL>), grid, dim3(64 * NS * NP), 0, st, a);
        return hipGetLastError();
      }
    }
  };
};

}  // namespace

hipError_t run_pass_bwd_a(const Geom& g, const PassArgs& a, hipStream_t st) {
  return run_pass_tilings<PASS_BWD_A, Run_k_bwd_a_<false>::R>(g, a, st);
}

hipError_t run_pass_slice_blk(const Geom& g, const PassArgs& a, hipStream_t st) {
  return run_pass_tilings<PASS_SLICE, Run_k_bwd_a_<true>::R>(g, a, st);
}

}  // namespace fs
