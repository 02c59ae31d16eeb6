// Streaming pass: slice (logits, per-point softmax, U += w^T F, s += sum w, lse), and the
// statistics pass of the slot-blocked family (the same softmax statistics, lse only).
// Kernel design and MFMA lane layouts are described at the top of fs_stream.h.

#include "fs_stream.h"

// bf16 head width 32, one slot wave per tile: the slice loads fx as rows and forms the
// point-ordered operand through LDS when it writes no normaliser (1: the forward-only slice;
// 2: always), or gathers it point by point (0). Measured at N = 2^24 (no normaliser) 2%
// faster, and at N = 2^20 with the normaliser written 6% slower.
#ifndef FS_SLICE_T
#define FS_SLICE_T 1
#endif

namespace fs {
namespace {

// =======================================================================================
// Slice pass
// =======================================================================================
// ST: statistics only (lse), no token accumulation. TRX: fx through LDS (above).
template <bool BF, int D, int GS, int NS, int NP, bool ST, bool TRX>
__global__ __launch_bounds__(64 * NS * NP) __attribute__((amdgpu_waves_per_eu(FS_WPE_SLICE))) void k_slice(
    PassArgs a) {
  constexpr int GB = GS / 16, VB = D / 16;
  constexpr bool SPLIT = BF;
  using T = typename Store<BF>::T;
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int wave = threadIdx.x >> 6, ws = wave % NS, wp = wave / NS;
  const HeadCtx c = head_ctx<D>(a, ws, GS);
  const int64_t rs = (int64_t)a.H * D;
  const T* xb = (const T*)a.x + c.off;
  const T* fb = (const T*)a.fx + c.off;

  SlotOp<BF, D, GB> wop;
  load_slotop<BF, D, GB, true, SPLIT>(wop, c.W, a.G, c.g0, slot_lim(a), c.sc, i, j);
  float bS[GB];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) bS[gb] = slot_bias(c, a, c.g0 + 16 * gb, i);

  f4 U[GB][VB];
  float sacc[GB];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) {
    sacc[gb] = 0.f;
#pragma unroll
    for (int vb = 0; vb < VB; ++vb) U[gb][vb] = zero4();
  }

  __shared__ float st_m[NS > 1 ? 2 : 1][NP][NS][32];
  __shared__ float st_l[NS > 1 ? 2 : 1][NP][NS][32];

  const int rsb = (int)(rs * sizeof(T));
  const bool want_lse = a.lse_out != nullptr;
  const int wpu = __builtin_amdgcn_readfirstlane(wp);
  // this chunk's sub-chunks: c.chunk, c.chunk + chunks, ... (one unless the stream is long)
  for (int64_t sub = c.chunk; sub < a.nsub; sub += a.chunks) {
  const int64_t pbeg = sub * a.sub_pts;
  const int64_t pend = min(a.N, pbeg + a.sub_pts);
  const int npts = pend > pbeg ? (int)(pend - pbeg) : 0;
  const int ntile = (npts + 32 * NP - 1) / (32 * NP);
  const auto rx = rows_rsrc(xb + pbeg * rs, npts, (int)rs, D);
  const auto rf = rows_rsrc(fb + pbeg * rs, npts, (int)rs, D);
  const auto rl = rows_rsrc(want_lse ? a.lse_out + (int64_t)c.bh * a.N + pbeg : a.Ws, npts, 1, 1);

  // TR: bf16 fx tiles (head width 32) arrive as rows, 16 bytes per lane, and become the
  // point-ordered k-operand of U += w^T fx through this wavefront's LDS rows
  constexpr bool TR = TRX && BF && D == 32 && !ST && NS == 1;
  constexpr int kTP = 80;  // LDS row pitch (64 bytes of a head row + 16)
  __shared__ __attribute__((aligned(16))) char trs[TR ? NP : 1][TR ? 32 * kTP : 16];
  struct Tile {
    RowOp<BF, D> xo[2];
    PtGather<BF, ST ? 1 : VB> f;
    uint4 frow[TR ? 2 : 1];
  };
  auto load_tile = [&](Tile& tt, int t) {
    const int tbo = (t * NP + wpu) * 32 * rsb;
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) load_row_buf<BF, D>(tt.xo[pb], rx, i * rsb, tbo + 16 * pb * rsb, j);
    if constexpr (TR) {
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) tt.frow[pb] = bld128u(rf, i * rsb + 16 * j, tbo + 16 * pb * rsb);
    } else if constexpr (!ST) {
      gather_points_buf<BF, VB>(tt.f, rf, rsb, tbo, i, j);
    }
  };
  pipeline<(NS >= FS_NS_NOPF ? 0 : FS_PF_SLICE), Tile>(ntile, load_tile, [&](Tile& cur, int t) {
    const int tb = (t * NP + wpu) * 32;
    const RowOp<BF, D>* xo = cur.xo;
    // S-layout logits: rows = points 16 pb + 4 j + r, cols = slots g0 + 16 gb + i
    f4 w[2][GB];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
        w[pb][gb] = mm_row_slot<BF, D, GB, SPLIT>(xo[pb], wop, gb, splat4(bS[gb]));

    // per point (row): max over the slots, then the sum of 2^(a - max); the eight rows of a
    // lane are reduced across the 16 slot lanes together
    float m[2][4], l[2][4];
    {
      float mx[8];
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float v = w[pb][0][r];
#pragma unroll
          for (int gb = 1; gb < GB; ++gb) v = vmax(v, w[pb][gb][r]);
          mx[4 * pb + r] = v;
        }
      row16_max_n(mx);
      float sm[8];
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          m[pb][r] = mx[4 * pb + r];
          float sum = 0.f;
#pragma unroll
          for (int gb = 0; gb < GB; ++gb) {
            const float e = __builtin_amdgcn_exp2f(w[pb][gb][r] - m[pb][r]);
            w[pb][gb][r] = e;
            sum += e;
          }
          sm[4 * pb + r] = sum;
        }
      row16_sum_n(sm);
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) l[pb][r] = sm[4 * pb + r];
    }

    // the lse store: lane i < 8 of row group j writes point 16 (i / 4) + 4 j + i % 4 (every
    // lane of a group holds the group's statistics), one store for the tile's 32 points
    auto pick = [i](float a0, float a1, float a2, float a3, float b0, float b1, float b2, float b3) {
      const bool o = i & 1, t = i & 2;
      const float va = t ? (o ? a3 : a2) : (o ? a1 : a0), vb = t ? (o ? b3 : b2) : (o ? b1 : b0);
      return (i & 4) ? vb : va;
    };
    float f[2][4], lse2[2][4], lse_st;
    if constexpr (NS == 1) {
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) f[pb][r] = __builtin_amdgcn_rcpf(l[pb][r]);
      lse_st = pick(m[0][0], m[0][1], m[0][2], m[0][3], m[1][0], m[1][1], m[1][2], m[1][3]) +
               __log2f(pick(l[0][0], l[0][1], l[0][2], l[0][3], l[1][0], l[1][1], l[1][2], l[1][3]));
    } else {
      const int par = t & 1;
      if (i == 0) {
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            st_m[par][wp][ws][16 * pb + 4 * j + r] = m[pb][r];
            st_l[par][wp][ws][16 * pb + 4 * j + r] = l[pb][r];
          }
      }
      __syncthreads();
      // lane p < 32 combines the slot groups' statistics of point p, then every lane fetches
      // the combined values of its own rows
      float Mp = st_m[par][wp][0][lane & 31];
#pragma unroll
      for (int s = 1; s < NS; ++s) Mp = vmax(Mp, st_m[par][wp][s][lane & 31]);
      float Lp = 0.f;
#pragma unroll
      for (int s = 0; s < NS; ++s)
        Lp += st_l[par][wp][s][lane & 31] * __builtin_amdgcn_exp2f(st_m[par][wp][s][lane & 31] - Mp);
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int q = 16 * pb + 4 * j + r;
          const float M = __shfl(Mp, q);
          const float L = __shfl(Lp, q);
          f[pb][r] = __builtin_amdgcn_exp2f(m[pb][r] - M) * __builtin_amdgcn_rcpf(L);
          lse2[pb][r] = M + __log2f(L);
        }
      lse_st = pick(lse2[0][0], lse2[0][1], lse2[0][2], lse2[0][3], lse2[1][0], lse2[1][1], lse2[1][2], lse2[1][3]);
    }

#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int q = 16 * pb + 4 * j + r;
        const float fr = tb + q < npts ? f[pb][r] : 0.f;
#pragma unroll
        for (int gb = 0; gb < GB; ++gb) w[pb][gb][r] *= fr;
      }
    if (want_lse && ws == 0 && i < 8) bst32(rl, lse_st, 4 * (16 * (i >> 2) + 4 * j + (i & 3)), 4 * tb);
    if constexpr (ST) return;
#pragma unroll
    for (int gb = 0; gb < GB; ++gb) {
      float sum = 0.f;
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) sum += w[pb][gb][r];
      sacc[gb] += sum;
    }
    if constexpr (TR) {
      char* tr = trs[wp];
      wave_lds_sync();
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
        *reinterpret_cast<uint4*>(tr + (16 * pb + i) * kTP + 16 * j) = cur.frow[pb];
      wave_lds_sync();
#pragma unroll
      for (int cb = 0; cb < VB; ++cb) {
        bf8 bt;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          bt[e] = *reinterpret_cast<const __bf16*>(tr + (16 * (e / 4) + 4 * j + (e % 4)) * kTP +
                                                   (16 * cb + i) * 2);
        cur.f.v[cb] = bt;
      }
    }
    if constexpr (!ST) mm_points<BF, GB, VB>(U, w, cur.f);
  });
  }
  if constexpr (ST) return;

  // ---- combine the NP point groups and write this workgroup's partials --------------------
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) sacc[gb] = col4_sum(sacc[gb]);
  float* pU = a.part + ((int64_t)c.bh * a.chunks + c.chunk) * a.G * D;
  float* pS = a.part2 + ((int64_t)c.bh * a.chunks + c.chunk) * a.G;
  if constexpr (NP > 1) {
    __shared__ f4 red[NP - 1][NS][GB][VB][64];
    __shared__ float reds[NP - 1][NS][GB][16];
    if (wp > 0) {
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
        for (int vb = 0; vb < VB; ++vb) red[wp - 1][ws][gb][vb][lane] = U[gb][vb];
        if (j == 0) reds[wp - 1][ws][gb][i] = sacc[gb];
      }
    }
    __syncthreads();
    if (wp == 0) {
      for (int q = 0; q < NP - 1; ++q)
#pragma unroll
        for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
          for (int vb = 0; vb < VB; ++vb) U[gb][vb] += red[q][ws][gb][vb][lane];
          sacc[gb] += reds[q][ws][gb][i];
        }
    }
  }
  if (wp == 0) {
#pragma unroll
    for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
      for (int vb = 0; vb < VB; ++vb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int g = c.g0 + 16 * gb + 4 * j + r;
          if (g < a.G) pU[(int64_t)g * D + 16 * vb + i] = U[gb][vb][r];
        }
      if (j == 0 && c.g0 + 16 * gb + i < a.G) pS[c.g0 + 16 * gb + i] = sacc[gb];
    }
  }
}

template <bool ST>
struct Run_k_slice_ {
  template <bool BF, int D, int GS, int NS, int NP, int PB>
  struct R {
    static hipError_t run(const PassCfg& cfg, int BH, const PassArgs& a, hipStream_t st) {
      dim3 grid(cfg.chunks * BH * cfg.nblk);
      constexpr bool kCanTR = FS_SLICE_T > 0 && BF && D == 32 && NS == 1 && !ST;
      if (kCanTR && (FS_SLICE_T == 2 || a.lse_out == nullptr))
        hipLaunchKernelGGL((k_slice<BF, D, GS, NS, NP, ST, kCanTR>), grid, dim3(64 * NS * NP), 0, st, a);
      else
        hipLaunchKernelGGL((k_slice<BF, D, GS, NS, NP, ST, false>), grid, dim3(64 * NS * NP), 0, st, a);
      return hipGetLastError();
    }
  };
};

}  // namespace

hipError_t run_pass_slice(const Geom& g, const PassArgs& a, hipStream_t st) {
  return run_pass_tilings<PASS_SLICE, Run_k_slice_<false>::R>(g, a, st);
}

hipError_t run_pass_stats(const Geom& g, const PassArgs& a, hipStream_t st) {
  return run_pass_tilings<PASS_STATS, Run_k_slice_<true>::R>(g, a, st);
}

}  // namespace fs
