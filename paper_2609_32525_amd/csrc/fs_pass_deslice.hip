// Streaming pass: deslice (logits, w = exp2(a - lse), out = w zmix).
// Kernel design and MFMA lane layouts are described at the top of fs_stream.h.

#include "fs_stream.h"

namespace fs {
namespace {

// =======================================================================================
// Deslice pass
// =======================================================================================
template <bool BF, int D, int GS, int NS, int NP>
__global__ __launch_bounds__(64 * NS * NP) __attribute__((amdgpu_waves_per_eu(FS_WPE_DESLICE))) void k_deslice(
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
  const float* lse = a.lse_in + (int64_t)c.bh * a.N;

  SlotOp<BF, D, GB> wop;
  load_slotop<BF, D, GB, true, SPLIT>(wop, c.W, a.G, c.g0, c.sc, i, j);
  float bT[GB][4];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb)
#pragma unroll
    for (int r = 0; r < 4; ++r) bT[gb][r] = c.sc * c.bias[c.g0 + 16 * gb + 4 * j + r];
  GOp<BF, GB, VB> zop;
  load_gop<BF, GB, VB, false>(zop, a.zmix + (int64_t)c.bh * a.G * D, D, c.g0, 1.0f, i, j);

  __shared__ f4 ox[NS > 1 ? NP : 1][NS > 1 ? NS : 1][VB][2][64];

  const int64_t pbeg = (int64_t)c.chunk * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int npts = pend > pbeg ? (int)(pend - pbeg) : 0;
  const int ntile = (npts + 32 * NP - 1) / (32 * NP);
  const int rsb = (int)(rs * sizeof(T));
  const auto rx = rows_rsrc(xb + pbeg * rs, npts, (int)rs, D);
  const auto ro = rows_rsrc(ob + pbeg * rs, npts, (int)rs, D);
  const auto rl = rows_rsrc(lse + pbeg, npts, 1, 1);
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
      const float l = bld32(rl, 4 * i, 4 * (tb + 16 * pb));
      tt.lse2[pb] = tb + 16 * pb + i < npts ? l : kMasked;
    }
  };
  pipeline<(NS >= FS_NS_NOPF ? 0 : FS_PF_DESLICE), Tile>(ntile, load_tile, [&](Tile& cur, int t) {
    const int tb = (t * NP + wpu) * 32;
    const RowOp<BF, D>* xo = cur.xo;
    const float* lse2 = cur.lse2;
    f4 w[GB][2];
#pragma unroll
    for (int gb = 0; gb < GB; ++gb)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) {
        f4 acc = f4{bT[gb][0], bT[gb][1], bT[gb][2], bT[gb][3]};
        acc = mm_slot_row<BF, D, GB, SPLIT>(wop, gb, xo[pb], acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] = __builtin_amdgcn_exp2f(acc[r] - lse2[pb]);
        w[gb][pb] = acc;
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
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
          bst_row4<BF>(ro, o[vb][pb], i * rsb + (16 * vb + 4 * j) * (int)sizeof(T), (tb + 16 * pb) * rsb);
    }
  });
}

template <bool BF, int D, int GS, int NS, int NP, int PB>
struct Run_k_deslice {
  static hipError_t run(const PassCfg& cfg, int BH, const PassArgs& a, hipStream_t st) {
    dim3 grid(cfg.chunks * BH * cfg.nblk);
    hipLaunchKernelGGL((k_deslice<BF, D, GS, NS, NP>), grid, dim3(64 * NS * NP), 0, st, a);
    return hipGetLastError();
  }
};

}  // namespace

hipError_t run_pass_deslice(const Geom& g, const PassArgs& a, hipStream_t st) {
  return run_pass_tilings<PASS_DESLICE, Run_k_deslice>(g, a, st);
}

}  // namespace fs
