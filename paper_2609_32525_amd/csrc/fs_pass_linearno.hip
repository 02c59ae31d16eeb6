// Streaming pass of the LinearNO variant: slice weights normalised by a softmax over the
// points of each slot, k[:, g] = softmax_n(a[:, g]), so z_g = sum_n k[n, g] fx[n] (App. E;
// the Untied-LN row of the Sec. 2 ablation suite). One pass over the points: every wavefront
// keeps, per slot it owns, a running maximum of the base-2 logits, the sum of 2^(a - max) and
// the numerators sum 2^(a - max) fx, rescaling both when the maximum grows; the wavefronts
// of a workgroup and then the workgroups (chunks) are merged the same way in a fixed order.
// Kernel design and MFMA lane layouts are described at the top of fs_stream.h.

#include <type_traits>

#include "fs_stream.h"

namespace fs {
namespace {

// 2^(m - M) for M >= m, exact 1 where they are equal (both -inf included: no points yet).
__device__ __forceinline__ float rescale(float m, float M) {
  return m == M ? 1.0f : __builtin_amdgcn_exp2f(m - M);
}

// Partials per (sample, head, chunk): U [G][D] into part, then [G] maxima and [G] sums into
// part2 (2 G floats).
template <bool BF, int D, int GS, int NS, int NP>
__global__ __launch_bounds__(64 * NS * NP) void k_slice_col(PassArgs a) {
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

  // U rows are slots 16 gb + 4 j + r (C layout); mrun, lrun belong to slot column 16 gb + i
  f4 U[GB][VB];
  float mrun[GB], lrun[GB];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) {
    mrun[gb] = -INFINITY;
    lrun[gb] = 0.f;
#pragma unroll
    for (int vb = 0; vb < VB; ++vb) U[gb][vb] = zero4();
  }

  const int64_t pbeg = (int64_t)c.chunk * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int npts = pend > pbeg ? (int)(pend - pbeg) : 0;
  const int ntile = (npts + 32 * NP - 1) / (32 * NP);
  const int rsb = (int)(rs * sizeof(T));
  const auto rx = rows_rsrc(xb + pbeg * rs, npts, (int)rs, D);
  const auto rf = rows_rsrc(fb + pbeg * rs, npts, (int)rs, D);
  const int wpu = __builtin_amdgcn_readfirstlane(wp);

  struct Tile {
    RowOp<BF, D> xo[2];
    PtGather<BF, VB> f;
  };
  auto load_tile = [&](Tile& tt, int t) {
    const int tbo = (t * NP + wpu) * 32 * rsb;
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) load_row_buf<BF, D>(tt.xo[pb], rx, i * rsb, tbo + 16 * pb * rsb, j);
    gather_points_buf<BF, VB>(tt.f, rf, rsb, tbo, i, j);
  };
  pipeline<(NS >= FS_NS_NOPF ? 0 : FS_PF_SLICE), Tile>(ntile, load_tile, [&](Tile& cur, int t) {
    const int tb = (t * NP + wpu) * 32;
    // S-layout logits: rows = points 16 pb + 4 j + r, cols = slots g0 + 16 gb + i
    f4 w[2][GB];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
        w[pb][gb] = mm_row_slot<BF, D, GB, SPLIT>(cur.xo[pb], wop, gb, splat4(bS[gb]));
    // padding rows (past the chunk's points) exist only in its last tile
    auto update = [&](auto ragged) {
      bool valid[2][4];
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) valid[pb][r] = !ragged.value || tb + 16 * pb + 4 * j + r < npts;
      bool moved = false;
      float fs[GB];
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
        float cm = -INFINITY;
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r) cm = valid[pb][r] ? vmax(cm, w[pb][gb][r]) : cm;
        cm = col4_max(cm);
        const float mnew = vmax(mrun[gb], cm);
        fs[gb] = rescale(mrun[gb], mnew);
        moved = moved || mnew != mrun[gb];
        mrun[gb] = mnew;
        float sum = 0.f;
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float e = valid[pb][r] ? __builtin_amdgcn_exp2f(w[pb][gb][r] - mnew) : 0.f;
            w[pb][gb][r] = e;
            sum += e;
          }
        lrun[gb] = lrun[gb] * fs[gb] + sum;
      }
      // the numerators follow only where some slot's maximum grew (rare once it settles)
      if (__any(moved)) {
#pragma unroll
        for (int gb = 0; gb < GB; ++gb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float fr = __shfl(fs[gb], 4 * j + r);  // the factor of slot row 4 j + r
#pragma unroll
            for (int vb = 0; vb < VB; ++vb) U[gb][vb][r] *= fr;
          }
      }
    };
    if (tb + 32 <= npts)
      update(std::false_type{});
    else
      update(std::true_type{});
    mm_points<BF, GB, VB>(U, w, cur.f);
  });

  // ---- merge the NP point groups (fixed order) and write the workgroup's partials --------
  float lsum[GB];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) lsum[gb] = col4_sum(lrun[gb]);
  float* pU = a.part + ((int64_t)c.bh * a.chunks + c.chunk) * a.G * D;
  float* pML = a.part2 + ((int64_t)c.bh * a.chunks + c.chunk) * 2 * a.G;
  if constexpr (NP > 1) {
    __shared__ f4 red[NP - 1][NS][GB][VB][64];
    __shared__ float redm[NP - 1][NS][GB][16], redl[NP - 1][NS][GB][16];
    if (wp > 0) {
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
#pragma unroll
        for (int vb = 0; vb < VB; ++vb) red[wp - 1][ws][gb][vb][lane] = U[gb][vb];
        if (j == 0) {
          redm[wp - 1][ws][gb][i] = mrun[gb];
          redl[wp - 1][ws][gb][i] = lsum[gb];
        }
      }
    }
    __syncthreads();
    if (wp == 0) {
      for (int q = 0; q < NP - 1; ++q)
#pragma unroll
        for (int gb = 0; gb < GB; ++gb) {
          const float mq = redm[q][ws][gb][i];
          const float M = vmax(mrun[gb], mq);
          const float f0 = rescale(mrun[gb], M), fq = rescale(mq, M);
          lsum[gb] = lsum[gb] * f0 + redl[q][ws][gb][i] * fq;
          mrun[gb] = M;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float f0r = __shfl(f0, 4 * j + r), fqr = __shfl(fq, 4 * j + r);
#pragma unroll
            for (int vb = 0; vb < VB; ++vb)
              U[gb][vb][r] = U[gb][vb][r] * f0r + red[q][ws][gb][vb][lane][r] * fqr;
          }
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
      if (j == 0 && c.g0 + 16 * gb + i < a.G) {
        pML[c.g0 + 16 * gb + i] = mrun[gb];
        pML[a.G + c.g0 + 16 * gb + i] = lsum[gb];
      }
    }
  }
}

template <bool BF, int D, int GS, int NS, int NP, int PB>
struct Run_k_slice_col {
  static hipError_t run(const PassCfg& cfg, int BH, const PassArgs& a, hipStream_t st) {
    dim3 grid(cfg.chunks * BH * cfg.nblk);
    hipLaunchKernelGGL((k_slice_col<BF, D, GS, NS, NP>), grid, dim3(64 * NS * NP), 0, st, a);
    return hipGetLastError();
  }
};

// Merge of the chunk partials of one (sample, head): per slot the largest maximum M, then
// l = sum_c l_c 2^(m_c - M) and z = sum_c U_c 2^(m_c - M) / l in chunk order; clse = M + log2 l
// (base 2). A slot with no points gets z = 0 and clse = -inf.
constexpr int kColThreads = 256;

__global__ __launch_bounds__(kColThreads) void k_reduce_col(const float* partU,
                                                            const float* partML, int chunks,
                                                            float* z, float* clse, int G,
                                                            int V) {
  const int bh = blockIdx.y;
  const int idx = blockIdx.x * kColThreads + threadIdx.x;
  if (idx >= G * V) return;
  const int g = idx / V;
  const float* ml = partML + (int64_t)bh * chunks * 2 * G;
  const float* pu = partU + (int64_t)bh * chunks * G * V + idx;
  float M = -INFINITY;
  for (int c = 0; c < chunks; ++c) M = vmax(M, ml[(int64_t)c * 2 * G + g]);
  float l = 0.f, u = 0.f;
#pragma unroll 4
  for (int c = 0; c < chunks; ++c) {
    const float f = rescale(ml[(int64_t)c * 2 * G + g], M);
    l += ml[(int64_t)c * 2 * G + G + g] * f;
    u += pu[(int64_t)c * G * V] * f;
  }
  z[(int64_t)bh * G * V + idx] = l > 0.f ? u / l : 0.f;
  if (idx % V == 0 && clse != nullptr) clse[(int64_t)bh * G + g] = l > 0.f ? M + __log2f(l) : -INFINITY;
}

__global__ __launch_bounds__(256) void k_fill(float* p, float v, int64_t n) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx < n) p[idx] = v;
}

}  // namespace

hipError_t launch_fill(float* p, float v, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, v, n);
  return hipGetLastError();
}

hipError_t run_pass_slice_col(const Geom& g, const PassArgs& a, hipStream_t st) {
  return run_pass_tilings<PASS_SLICE, Run_k_slice_col>(g, a, st);
}

hipError_t launch_reduce_col(const Geom& g, const float* partU, const float* partML, int chunks,
                             float* z, float* clse, hipStream_t st) {
  dim3 grid((g.G * g.V + kColThreads - 1) / kColThreads, g.BH());
  hipLaunchKernelGGL(k_reduce_col, grid, dim3(kColThreads), 0, st, partU, partML, chunks, z, clse,
                     g.G, g.V);
  return hipGetLastError();
}

}  // namespace fs
