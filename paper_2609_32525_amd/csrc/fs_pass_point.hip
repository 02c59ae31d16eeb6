// Point-owned pass of the slot-blocked backward (large G): for every point, with the slots
// streamed in blocks of 64,
//   c  = sum_g w dw          (the softmax correction; dw = dout zmix^T + F dU^T + ds)
//   tb = sum_g w t           (weighted mean of the shifted base-2 logits, for dtau)
//   dfx = sum_g w dU
//   dx  = sum_g w (dw - c) W_s[:, g] / tau = (P - c Q) / tau,
//         P = sum_g (w dw) W_s[:, g] / tau,  Q = sum_g w W_s[:, g] / tau
// The last identity lets dx be accumulated in the same sweep over the slot blocks, before c
// is known (paper: App. F.1, "G-blocked kernels": a point-owned backward kernel; here one
// sweep instead of two). The slot-owned parameter pass then reads (c, tb) per point.
// ROLE (as in the fused pass B): 0 tied; 1 the untied slice weights (dw = F dU^T + ds; dx and
// dfx written); 2 the untied deslice weights (dw = dout zmix^T, no ds; their dx part added to
// the dx role 1 wrote; no dfx); 3 LinearNO's slice weights (weights 2^(a - clse_g), already
// normalised over the points, so no per-point normaliser and no correction: c = 0, dx = P;
// dw = F dz^T + ds with no slot-mean shifts).
//
// The per-head operands (W_s, zmix, dU, bias, ds) are far too large at large G to stay in
// registers, so each block's MFMA operand images are built once per workgroup in LDS, double
// buffered: while the wavefronts compute block k from one buffer, each of them has already
// issued the global loads for its share of block k + 1 and writes it to the other buffer
// afterwards. Every wavefront owns one 32-point tile per step and reads the images it needs.
// dw uses the same centred operands as the fused pass B (zmix, dU and ds minus their
// mass-weighted slot means), so c is consistent with the parameter pass. bf16 storage rounds
// the B operands of P and Q in two bf16 parts (w dw and w vary over many orders of magnitude
// and P - c Q cancels).

#include "fs_stream.h"

namespace fs {
namespace {

constexpr int kHS = 32;  // slots per half block: operands are imaged per half (GB = 2)

// Image buffers of the point pass: a ring of four where LDS allows (4), or two (2).
#ifndef FS_POINT_RING
#define FS_POINT_RING 4
#endif

template <bool BF, int D>
struct PointImages {
  static constexpr int GBH = kHS / 16;
  static constexpr int VB = D / 16;
  using SOp = SlotOp<BF, D, GBH>;
  using UOp = GOp<BF, GBH, VB>;
  // bf16 dw operands use only the high part of a SlotOp
  static constexpr int kW = lds_chunks<SOp>();
  static constexpr int kZ = BF ? lds_chunks<SOp>() / 2 : lds_chunks<SOp>();
  static constexpr int kU = lds_chunks<UOp>();
  // per half: W (logits), zv, uv (dw), ug (dfx), wg (P, Q); then bias and ds of the block
  static constexpr int kHalf = kW + 2 * kZ + 2 * kU;
  static constexpr int kChunks = 2 * kHalf + 2 * 64 / 4;  // + bS[64], dsS[64] as uint4
  // stride of one block's image set, padded so that the point pass's workgroup copies it in
  // whole rounds
  static constexpr int kRound = 64 * FS_POINT_WAVES;
  static constexpr int kStride = (kChunks + kRound - 1) / kRound * kRound;
};

// The first nchunks 16-byte chunks of a per-lane operand (its register image), per lane.

template <class Op>
__device__ __forceinline__ void put_first(const Op& o, uint4* base, int lane, int nchunks) {
  const u32x4* src = reinterpret_cast<const u32x4*>(&o);
#pragma unroll
  for (int q = 0; q < nchunks; ++q) reinterpret_cast<u32x4*>(base)[q * 64 + lane] = src[q];
}
template <class Op>
__device__ __forceinline__ void get_first(Op& o, const uint4* base, int lane, int nchunks) {
  u32x4* dst = reinterpret_cast<u32x4*>(&o);
#pragma unroll
  for (int q = 0; q < nchunks; ++q) dst[q] = reinterpret_cast<const u32x4*>(base)[q * 64 + lane];
}

// Builds job q (q < 11) of slot block blk's image set for one (b, h) into `out` (global or
// LDS, same layout): jobs 0..9 are (half h = q / 5, kind q % 5) with kinds W (logits, scaled by
// log2(e)/tau), zv and uv (centred zmix and dU for dw), ug (dU for dfx), wg (W^T / tau for P
// and Q); job 10 is the block's scaled bias and centred ds. Called by a whole wavefront.
template <bool BF, int D, int ROLE>
__device__ __forceinline__ void build_job(int q, int blk, const HeadCtx& c, const PassArgs& a,
                                          uint4* out, int lane) {
  constexpr bool ZV = ROLE == 0 || ROLE == 2;  // dw has the dout zmix^T term
  constexpr bool UV = ROLE != 2;               // dw has the F dU^T term (and dfx is written)
  constexpr bool SHIFT = ROLE != 3;            // slot-mean shifts of the dw operands
  using IM = PointImages<BF, D>;
  using SOp = typename IM::SOp;
  using UOp = typename IM::UOp;
  constexpr int GBH = IM::GBH, VB = IM::VB, DB = D / 16;
  const int i = lane & 15, j = lane >> 4;
  const float inv_tau = 1.0f / a.tau[c.h];
  const float* zm = a.zmix + (int64_t)c.bh * a.G * D;
  const float* dU = a.dU + (int64_t)c.bh * a.G * D;
  const float* dsv = a.ds + (int64_t)c.bh * a.G;
  const float* cen = a.cen + (int64_t)c.bh * (2 * D + 1);
  const int g0 = blk * 64;
  if (q < 10) {
    const int h = q / 5, kind = q % 5, gh = g0 + kHS * h;
    uint4* hb = out + h * IM::kHalf;
    if (kind <= 2) {
      SOp o;
      if (kind == 1 && !ZV) return;  // images the role does not read
      if (kind == 2 && !UV) return;
      if (kind == 0) load_slotop<BF, D, GBH, true, BF>(o, c.W, a.G, gh, slot_lim(a), c.sc, i, j);
      if (kind == 1) load_slotop<BF, D, GBH, false, false>(o, zm, D, gh, slot_lim(a), 1.0f, i, j, cen);
      if (kind == 2)
        load_slotop<BF, D, GBH, false, false>(o, dU, D, gh, slot_lim(a), 1.0f, i, j,
                                              SHIFT ? cen + D : nullptr);
      if (kind == 0) put_first(o, hb, lane, IM::kW / 64);
      if (kind == 1) put_first(o, hb + IM::kW, lane, IM::kZ / 64);
      if (kind == 2) put_first(o, hb + IM::kW + IM::kZ, lane, IM::kZ / 64);
    } else {
      if (kind == 3 && !UV) return;
      UOp o;
      if (kind == 3) load_gop<BF, GBH, VB, false>(o, dU, D, gh, slot_lim(a), 1.0f, i, j);
      if (kind == 4) load_gop<BF, GBH, DB, true>(o, c.W, a.G, gh, slot_lim(a), inv_tau, i, j);
      put_first(o, hb + IM::kW + 2 * IM::kZ + (kind == 4 ? IM::kU : 0), lane, IM::kU / 64);
    }
  } else if (q == 10) {
    float* f = reinterpret_cast<float*>(out + 2 * IM::kHalf);
    const bool real = g0 + lane < a.G;  // padding slots: masked logit, no ds
    const int gl = min(g0 + lane, a.G - 1);
    const float dv = dsv[gl] - (SHIFT ? cen[2 * D] : 0.f);
    // LinearNO: the weights' per-slot normaliser over the points enters as a bias shift
    const float cl = ROLE == 3 ? a.clse[(int64_t)c.bh * a.G + gl] : 0.f;
    f[lane] = slot_bias_at(c, a, g0 + lane) - slot_mask(real, cl, 0.f);
    f[64 + lane] = ROLE == 2 ? 0.f : slot_mask(real, dv, 0.f);
  }
}

// Image sets of every slot block of every (b, h), [BH][ceil(G / 64)][kChunks] uint4: built once
// per backward so that the point-owned pass only copies them. grid ceil(G / 64) BH, 11
// wavefronts.
template <bool BF, int D, int ROLE>
__global__ __launch_bounds__(64 * 11) void k_point_images(PassArgs a, uint4* img) {
  using IM = PointImages<BF, D>;
  const int NB = (a.G + 63) / 64;
  const int blk = blockIdx.x % NB;
  const int bh = blockIdx.x / NB;
  HeadCtx c;
  c.bh = bh;
  c.b = bh / a.H;
  c.h = bh % a.H;
  c.sc = kLog2e / a.tau[c.h];
  c.W = a.Ws + (a.ws_per_head ? (int64_t)c.h * D * a.G : 0);
  c.bias = a.bias + (a.ws_per_head ? (int64_t)c.h * a.G : 0);
  build_job<BF, D, ROLE>(threadIdx.x >> 6, blk, c, a, img + ((int64_t)bh * NB + blk) * IM::kStride,
                         threadIdx.x & 63);
}

// A thread's share of one block's image set on its way from global memory to LDS: chunks
// t, t + NT, ... (compile-time recursion keeps every index constant). Held as native 4-lane
// vectors: as uint4 structs the array stayed in memory (the compiler placed it in LDS, and
// every load was waited for where it was issued).
template <int N>
struct Stage {
  u32x4 v[N];
};
template <int U, int N, int NT>
__device__ __forceinline__ void stage_load(Stage<N>& s, const uint4* src) {
  if constexpr (U < N) {
    s.v[U] = reinterpret_cast<const u32x4*>(src)[threadIdx.x + U * NT];
    stage_load<U + 1, N, NT>(s, src);
  }
}
template <int U, int N, int NT>
__device__ __forceinline__ void stage_put(const Stage<N>& s, uint4* dst) {
  if constexpr (U < N) {
    reinterpret_cast<u32x4*>(dst)[threadIdx.x + U * NT] = s.v[U];
    stage_put<U + 1, N, NT>(s, dst);
  }
}

// A T-layout tile over a half block's 32 slots as the B operand of contractions over slots,
// rounded in two bf16 parts for bf16 storage (hi + lo), converted once per tile.
template <bool BF, int GBH>
struct SplitB {
  const f4 (*t)[2];
  bf8 hi[GBH / 2][2], lo[GBH / 2][2];
};
template <bool BF, int GBH>
__device__ __forceinline__ SplitB<BF, GBH> split_b(const f4 (*t)[2]) {
  SplitB<BF, GBH> o;
  o.t = t;
  if constexpr (BF) {
#pragma unroll
    for (int q = 0; q < GBH / 2; ++q)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) split_bf8(t[2 * q][pb], t[2 * q + 1][pb], o.hi[q][pb], o.lo[q][pb]);
  }
  return o;
}
// acc += M^T (hi + lo): the contraction over the half block with the split operand.
template <bool BF, int GBH, int CB>
__device__ __forceinline__ f4 mm_split_b(const GOp<BF, GBH, CB>& o, int cb, const SplitB<BF, GBH>& s,
                                         int pb, f4 acc) {
  if constexpr (!BF) {
    return mm_gop_tile<false, GBH, CB, 2>(o, cb, s.t, pb, acc);
  } else {
#pragma unroll
    for (int q = 0; q < GBH / 2; ++q) {
      acc = mfma_bf16(o.v[q][cb], s.hi[q][pb], acc);
      acc = mfma_bf16(o.v[q][cb], s.lo[q][pb], acc);
    }
    return acc;
  }
}

template <bool BF, int D, int NW, int ROLE>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(D > 32 ? 1 : FS_POINT_WPE_MIN, D > 32 ? 1 : FS_POINT_WPE))) void k_point(
    PassArgs a) {
  constexpr bool ZV = ROLE == 0 || ROLE == 2;  // dw = dout zmix^T + ...
  constexpr bool UV = ROLE != 2;               // dw = ... + F dU^T; dfx = w dU
  constexpr bool COLN = ROLE == 3;             // no per-point normaliser or correction
  using IM = PointImages<BF, D>;
  using SOp = typename IM::SOp;
  using UOp = typename IM::UOp;
  constexpr int GBH = IM::GBH, VB = IM::VB, DB = D / 16;
  constexpr bool SPLIT = BF;
  using T = typename Store<BF>::T;
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int wave = threadIdx.x >> 6;
  const int wpu = __builtin_amdgcn_readfirstlane(wave);
  const HeadCtx c = head_ctx<D>(a, 0, 0);
  const int64_t rs = (int64_t)a.H * D;
  const T* xb = (const T*)a.x + c.off;
  const T* fb = (const T*)a.fx + c.off;
  const T* gb_ = (const T*)a.dout + c.off;
  T* dxb = (T*)a.out + c.off;
  T* dfb = (T*)a.out2 + c.off;
  const float* lse = a.lse_in + (int64_t)c.bh * a.N;
  const int NB = (a.G + 63) / 64;

  // image buffers: a ring of four where they fit in LDS (blocks staged two ahead, a workgroup
  // barrier after every second block), else two (one ahead, a barrier after every block)
  constexpr int RING = FS_POINT_RING == 4 && 4 * IM::kStride * 16 <= 160 * 1024 ? 4 : 2;
  constexpr int LA = RING / 2;
  __shared__ uint4 img[RING][IM::kStride];

  const int64_t pbeg = (int64_t)c.chunk * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int npts = pend > pbeg ? (int)(pend - pbeg) : 0;
  const int nstep = (npts + 32 * NW - 1) / (32 * NW);
  const int rsb = (int)(rs * sizeof(T));
  const auto rx = rows_rsrc(xb + pbeg * rs, npts, (int)rs, D);
  const auto rf = rows_rsrc(fb + pbeg * rs, npts, (int)rs, D);
  const auto rg = rows_rsrc(gb_ + pbeg * rs, npts, (int)rs, D);
  const auto rdx = rows_rsrc(dxb + pbeg * rs, npts, (int)rs, D);
  const auto rdf = rows_rsrc(dfb + pbeg * rs, npts, (int)rs, D);
  const auto rl = rows_rsrc(lse + pbeg, npts, 1, 1);
  const auto rc = rows_rsrc(a.cpt_out + ((int64_t)c.bh * a.N + pbeg) * 4, npts, 4, 4);

  // staging: thread t copies chunks t, t + 64 NW, ... of a block's image set
  static_assert(IM::kStride % (64 * NW) == 0, "image stride must be whole copy rounds");
  constexpr int kCopy = IM::kStride / (64 * NW);
  const uint4* himg = static_cast<const uint4*>(a.img) + (int64_t)c.bh * NB * IM::kStride;
  Stage<kCopy> stg;

  if (nstep == 0) return;  // uniform over the workgroup
  const int nu = nstep * NB;  // block visits of the workgroup, u = step NB + blk
#pragma unroll
  for (int u = 0; u < LA; ++u)
    if (u < nu) {
      stage_load<0, kCopy, 64 * NW>(stg, himg + (int64_t)u * IM::kStride);
      stage_put<0, kCopy, 64 * NW>(stg, img[u]);
    }
  __syncthreads();

  int u = 0;
  for (int step = 0; step < nstep; ++step) {
    const int tp0 = (step * NW + wpu) * 32;
    RowOp<BF, D> xo[2], go[2], fo[2];
    float lse2[2];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const int so = (tp0 + 16 * pb) * rsb;
      load_row_buf<BF, D>(xo[pb], rx, i * rsb, so, j);
      if constexpr (ZV) load_row_buf<BF, D>(go[pb], rg, i * rsb, so, j);
      if constexpr (UV) load_row_buf<BF, D>(fo[pb], rf, i * rsb, so, j);
      const float l = COLN ? 0.f : bld32(rl, 4 * i, 4 * (tp0 + 16 * pb));
      lse2[pb] = tp0 + 16 * pb + i < npts ? l : kMasked;
    }
    f4 gf[VB][2], P[DB][2], Q[DB][2];
    float csum[2] = {0.f, 0.f}, tsum[2] = {0.f, 0.f};
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
#pragma unroll
      for (int vb = 0; vb < VB; ++vb) gf[vb][pb] = zero4();
#pragma unroll
      for (int d = 0; d < DB; ++d) P[d][pb] = Q[d][pb] = zero4();
    }

    for (int blk = 0; blk < NB; ++blk) {
      // global loads of the next block's share (block 0 of the next step after the last),
      // in flight over this block's arithmetic; fp32 head width 32 has no registers to hold
      // them and loads them at the end of the block
      const bool more = u + LA < nu;
      const int nblk = blk + LA < NB ? blk + LA : blk + LA - NB;
      const uint4* next = himg + (int64_t)nblk * IM::kStride;
      constexpr bool kEarly = BF || D < 32;
      if (kEarly && more) stage_load<0, kCopy, 64 * NW>(stg, next);
      const uint4* cb = img[u % RING];
      const float* bS = reinterpret_cast<const float*>(cb + 2 * IM::kHalf);
#pragma unroll 1
      for (int h = 0; h < 2; ++h) {
        const uint4* hb = cb + h * IM::kHalf;
        // T-layout tiles: rows = slots 32 h + 16 gb + 4 j + r of the block, cols = points
        f4 w[GBH][2], dw[GBH][2];
        {
          SOp wop;
          lds_get(wop, hb, lane);
#pragma unroll
          for (int gb = 0; gb < GBH; ++gb) {
            const f4 bT = *reinterpret_cast<const f4*>(bS + kHS * h + 16 * gb + 4 * j);
#pragma unroll
            for (int pb = 0; pb < 2; ++pb) {
              f4 acc = mm_slot_row<BF, D, GBH, SPLIT>(wop, gb, xo[pb], bT);
              f4 ww;
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const float t = acc[r] - lse2[pb];
                ww[r] = __builtin_amdgcn_exp2f(t);
                tsum[pb] += ww[r] * t;
              }
              w[gb][pb] = ww;
            }
          }
        }
        {
          SOp zv, uv;
          if constexpr (BF) {  // only the high parts are imaged; the low parts are unused
            zv = SOp{};
            uv = SOp{};
          }
          if constexpr (ZV) get_first(zv, hb + IM::kW, lane, IM::kZ / 64);
          if constexpr (UV) get_first(uv, hb + IM::kW + IM::kZ, lane, IM::kZ / 64);
#pragma unroll
          for (int gb = 0; gb < GBH; ++gb) {
            const f4 dsT = *reinterpret_cast<const f4*>(bS + 64 + kHS * h + 16 * gb + 4 * j);
#pragma unroll
            for (int pb = 0; pb < 2; ++pb) {
              f4 g = dsT;
              if constexpr (ZV) g = mm_slot_row<BF, D, GBH, false>(zv, gb, go[pb], g);
              if constexpr (UV) g = mm_slot_row<BF, D, GBH, false>(uv, gb, fo[pb], g);
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                g[r] *= w[gb][pb][r];  // w dw
                csum[pb] += g[r];
              }
              dw[gb][pb] = g;
            }
          }
        }
        {
          UOp ug, wg;
          if constexpr (UV) lds_get(ug, hb + IM::kW + 2 * IM::kZ, lane);
          lds_get(wg, hb + IM::kW + 2 * IM::kZ + IM::kU, lane);
          const SplitB<BF, GBH> dws = split_b<BF, GBH>(dw);
#pragma unroll
          for (int pb = 0; pb < 2; ++pb) {
            if constexpr (UV) {
              const TileB<BF, GBH, 2> wt = tile_b<BF, GBH, 2>(w);
#pragma unroll
              for (int vb = 0; vb < VB; ++vb)
                gf[vb][pb] = mm_gop_b<BF, GBH, VB, 2>(ug, vb, wt, pb, gf[vb][pb]);
            }
#pragma unroll
            for (int d = 0; d < DB; ++d) P[d][pb] = mm_split_b<BF, GBH, DB>(wg, d, dws, pb, P[d][pb]);
            if constexpr (!COLN) {  // Q only for the correction c Q
              const SplitB<BF, GBH> ws = split_b<BF, GBH>(w);
#pragma unroll
              for (int d = 0; d < DB; ++d) Q[d][pb] = mm_split_b<BF, GBH, DB>(wg, d, ws, pb, Q[d][pb]);
            }
          }
        }
      }
      if (more) {
        if constexpr (!kEarly) stage_load<0, kCopy, 64 * NW>(stg, next);
        stage_put<0, kCopy, 64 * NW>(stg, img[(u + LA) % RING]);
      }
      // with the ring of four the buffer written here held block u - 2, which every
      // wavefront finished before the barrier after block u - 1 (u even) or u - 2 (u odd)
      if (RING == 2 || (u & 1)) __syncthreads();
      ++u;
    }

    // per point: c and tb over the four lane rows; dx = P - c Q; stores
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const float cc = COLN ? 0.f : col4_sum(csum[pb]);
      const float tb = COLN ? 0.f : col4_sum(tsum[pb]);
      const int so = (tp0 + 16 * pb) * rsb;
      if constexpr (UV) {
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
          bst_row4<BF>(rdf, gf[vb][pb], i * rsb + (16 * vb + 4 * j) * (int)sizeof(T), so);
      }
#pragma unroll
      for (int d = 0; d < DB; ++d) {
        const int vo = i * rsb + (16 * d + 4 * j) * (int)sizeof(T);
        f4 v;
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = COLN ? P[d][pb][r] : P[d][pb][r] - cc * Q[d][pb][r];
        if constexpr (ROLE == 2) v += bld_row4<BF>(rdx, vo, so);  // the slice weights' dx part
        bst_row4<BF>(rdx, v, vo, so);
      }
      // the parameter pass's per-point record: c, tb and the normaliser in one 16-byte load
      if (!COLN && j == pb) bst128(rc, f4{cc, tb, lse2[pb], 0.f}, 16 * i, 16 * (tp0 + 16 * pb));
      csum[pb] = tsum[pb] = 0.f;
    }
  }
}

// Wavefronts per workgroup of the in-LDS statistics pass (12 measured faster than 8 and 16).
#ifndef FS_STATS_WAVES
#define FS_STATS_WAVES 12
#endif

// Statistics pass of the slot-blocked family, point-owned: every wavefront takes a 32-point
// tile and sweeps all slots in blocks of 64, keeping per point a running maximum of the base-2
// logits and the sum of 2^(a - max), rescaled when the maximum grows; it writes
// lse2 = max + log2(sum). The projection's operand images for all slots (scaled by
// log2(e)/tau, bf16 hi + lo) and the scaled bias are built once per workgroup into LDS (up to
// 132 KB at G = 1024), so the sweep needs no exchange between wavefronts and no barrier.
template <bool BF, int D, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(NW / 4, NW / 4))) void k_stats_pt(
    PassArgs a) {
  using SOp = SlotOp<BF, D, 4>;
  using T = typename Store<BF>::T;
  constexpr int kB = lds_chunks<SOp>();  // one 64-slot block's image
  constexpr int kMaxBlk = 1024 / 64;
  __shared__ uint4 simg[kMaxBlk * kB + 1024 / 4];
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int wave = threadIdx.x >> 6;
  const int wpu = __builtin_amdgcn_readfirstlane(wave);
  const HeadCtx c = head_ctx<D>(a, 0, 0);
  const int NB = (a.G + 63) / 64;
  float* bS = reinterpret_cast<float*>(simg + kMaxBlk * kB);
  for (int blk = wave; blk < NB; blk += NW) {
    SOp o;
    load_slotop<BF, D, 4, true, BF>(o, c.W, a.G, 64 * blk, slot_lim(a), c.sc, i, j);
    lds_put(o, simg + blk * kB, lane);
  }
  for (int g = threadIdx.x; g < 64 * NB; g += 64 * NW) bS[g] = slot_bias_at(c, a, g);
  __syncthreads();

  const int64_t rs = (int64_t)a.H * D;
  const T* xb = (const T*)a.x + c.off;
  const int64_t pbeg = (int64_t)c.chunk * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int npts = pend > pbeg ? (int)(pend - pbeg) : 0;
  const int nstep = (npts + 32 * NW - 1) / (32 * NW);
  const int rsb = (int)(rs * sizeof(T));
  const auto rx = rows_rsrc(xb + pbeg * rs, npts, (int)rs, D);
  const auto rl = rows_rsrc(a.lse_out + (int64_t)c.bh * a.N + pbeg, npts, 1, 1);
  for (int step = 0; step < nstep; ++step) {
    const int tp0 = (step * NW + wpu) * 32;
    RowOp<BF, D> xo[2];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) load_row_buf<BF, D>(xo[pb], rx, i * rsb, (tp0 + 16 * pb) * rsb, j);
    // per lane: point 16 pb + i of the tile, slots 16 gb + 4 j + r of each block
    float m[2] = {-INFINITY, -INFINITY}, l[2] = {0.f, 0.f};
    for (int blk = 0; blk < NB; ++blk) {
      SOp wop;
      lds_get(wop, simg + blk * kB, lane);
      f4 t[4][2];
#pragma unroll
      for (int gb = 0; gb < 4; ++gb) {
        const f4 bT = *reinterpret_cast<const f4*>(bS + 64 * blk + 16 * gb + 4 * j);
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) t[gb][pb] = mm_slot_row<BF, D, 4, BF>(wop, gb, xo[pb], bT);
      }
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) {
        float bm = t[0][pb][0];
#pragma unroll
        for (int gb = 0; gb < 4; ++gb)
#pragma unroll
          for (int r = 0; r < 4; ++r) bm = vmax(bm, t[gb][pb][r]);
        const float mn = vmax(m[pb], col4_max(bm));
        float sum = 0.f;
#pragma unroll
        for (int gb = 0; gb < 4; ++gb)
#pragma unroll
          for (int r = 0; r < 4; ++r) sum += __builtin_amdgcn_exp2f(t[gb][pb][r] - mn);
        l[pb] = l[pb] * __builtin_amdgcn_exp2f(m[pb] - mn) + sum;
        m[pb] = mn;
      }
    }
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const float L = col4_sum(l[pb]);
      if (j == 0) bst32(rl, m[pb] + __log2f(L), 4 * i, 4 * (tp0 + 16 * pb));
    }
  }
}

// Statistics pass for head widths whose operand images of all slots do not fit in LDS
// (dh = 64: 256 KB at G = 1024): the same running maximum and rescaled sum per point, with the
// slot blocks' images (W_s split in two bf16 parts, scaled bias; built once per forward by
// k_stats_images) streamed through double-buffered LDS as in the point-owned pass.
template <bool BF, int D>
struct StatImages {
  using SOp = SlotOp<BF, D, 4>;
  static constexpr int kW = lds_chunks<SOp>();
  static constexpr int kChunks = kW + 64 / 4;  // + the block's 64 scaled biases
};
template <int NW>
constexpr int stat_stride(int chunks) {
  return (chunks + 64 * NW - 1) / (64 * NW) * (64 * NW);  // whole copy rounds
}

template <bool BF, int D, int NW>
__global__ __launch_bounds__(64) void k_stats_images(PassArgs a, uint4* img) {
  using SI = StatImages<BF, D>;
  constexpr int kStride = stat_stride<NW>(SI::kChunks);
  const int NB = (a.G + 63) / 64;
  const int blk = blockIdx.x % NB, bh = blockIdx.x / NB;
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  HeadCtx c;
  c.bh = bh;
  c.h = bh % a.H;
  c.sc = kLog2e / a.tau[c.h];
  c.W = a.Ws + (a.ws_per_head ? (int64_t)c.h * D * a.G : 0);
  c.bias = a.bias + (a.ws_per_head ? (int64_t)c.h * a.G : 0);
  uint4* out = img + ((int64_t)bh * NB + blk) * kStride;
  typename SI::SOp o;
  load_slotop<BF, D, 4, true, BF>(o, c.W, a.G, 64 * blk, slot_lim(a), c.sc, i, j);
  put_first(o, out, lane, SI::kW / 64);
  reinterpret_cast<float*>(out + SI::kW)[lane] = slot_bias_at(c, a, 64 * blk + lane);
}

template <bool BF, int D, int NW>
__global__ __launch_bounds__(64 * NW) void k_stats_stream(PassArgs a, const uint4* img) {
  using SI = StatImages<BF, D>;
  using SOp = typename SI::SOp;
  using T = typename Store<BF>::T;
  constexpr int kStride = stat_stride<NW>(SI::kChunks);
  constexpr int kCopy = kStride / (64 * NW);
  __shared__ uint4 simg[2][kStride];
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int wpu = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const HeadCtx c = head_ctx<D>(a, 0, 0);
  const int NB = (a.G + 63) / 64;
  const uint4* himg = img + (int64_t)c.bh * NB * kStride;

  const int64_t rs = (int64_t)a.H * D;
  const T* xb = (const T*)a.x + c.off;
  const int64_t pbeg = (int64_t)c.chunk * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int npts = pend > pbeg ? (int)(pend - pbeg) : 0;
  const int nstep = (npts + 32 * NW - 1) / (32 * NW);
  const int rsb = (int)(rs * sizeof(T));
  const auto rx = rows_rsrc(xb + pbeg * rs, npts, (int)rs, D);
  const auto rl = rows_rsrc(a.lse_out + (int64_t)c.bh * a.N + pbeg, npts, 1, 1);

  Stage<kCopy> stg;
  if (nstep == 0) return;  // uniform over the workgroup
  stage_load<0, kCopy, 64 * NW>(stg, himg);
  stage_put<0, kCopy, 64 * NW>(stg, simg[0]);
  __syncthreads();
  int kbuf = 0;
  for (int step = 0; step < nstep; ++step) {
    const int tp0 = (step * NW + wpu) * 32;
    RowOp<BF, D> xo[2];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) load_row_buf<BF, D>(xo[pb], rx, i * rsb, (tp0 + 16 * pb) * rsb, j);
    float m[2] = {-INFINITY, -INFINITY}, l[2] = {0.f, 0.f};
    for (int blk = 0; blk < NB; ++blk) {
      const bool more = blk + 1 < NB || step + 1 < nstep;
      if (more)
        stage_load<0, kCopy, 64 * NW>(stg, himg + (int64_t)(blk + 1 < NB ? blk + 1 : 0) * kStride);
      const uint4* cb = simg[kbuf];
      const float* bS = reinterpret_cast<const float*>(cb + SI::kW);
      SOp wop;
      lds_get(wop, cb, lane);
      f4 t[4][2];
#pragma unroll
      for (int gb = 0; gb < 4; ++gb) {
        const f4 bT = *reinterpret_cast<const f4*>(bS + 16 * gb + 4 * j);
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) t[gb][pb] = mm_slot_row<BF, D, 4, BF>(wop, gb, xo[pb], bT);
      }
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) {
        float bm = t[0][pb][0];
#pragma unroll
        for (int gb = 0; gb < 4; ++gb)
#pragma unroll
          for (int r = 0; r < 4; ++r) bm = vmax(bm, t[gb][pb][r]);
        const float mn = vmax(m[pb], col4_max(bm));
        float sum = 0.f;
#pragma unroll
        for (int gb = 0; gb < 4; ++gb)
#pragma unroll
          for (int r = 0; r < 4; ++r) sum += __builtin_amdgcn_exp2f(t[gb][pb][r] - mn);
        l[pb] = l[pb] * __builtin_amdgcn_exp2f(m[pb] - mn) + sum;
        m[pb] = mn;
      }
      if (more) stage_put<0, kCopy, 64 * NW>(stg, simg[kbuf ^ 1]);
      __syncthreads();
      kbuf ^= 1;
    }
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const float L = col4_sum(l[pb]);
      if (j == 0) bst32(rl, m[pb] + __log2f(L), 4 * i, 4 * (tp0 + 16 * pb));
    }
  }
}

}  // namespace

size_t stat_image_bytes(const Geom& g) {
  if (g.D != 64 || !g.bf16) return 0;  // the in-LDS statistics pass builds its own
  const int ch = stat_stride<FS_POINT_WAVES_WIDE>(StatImages<true, 64>::kChunks);
  return (size_t)g.BH() * ((g.G + 63) / 64) * ch * 16;
}

hipError_t run_pass_stats_stream(const Geom& g, const PassArgs& a, void* img, hipStream_t st) {
  const PassCfg cfg = pick_cfg(g, PASS_POINT);
  if (g.D != 64 || !g.bf16 || cfg.NP != FS_POINT_WAVES_WIDE) return hipErrorInvalidConfiguration;
  uint4* im = static_cast<uint4*>(img);
  const dim3 igrid(((g.G + 63) / 64) * g.BH()), grid(cfg.chunks * g.BH());
  hipLaunchKernelGGL((k_stats_images<true, 64, FS_POINT_WAVES_WIDE>), igrid, dim3(64), 0, st, a, im);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_stats_stream<true, 64, FS_POINT_WAVES_WIDE>), grid,
                     dim3(64 * FS_POINT_WAVES_WIDE), 0, st, a, im);
  return hipGetLastError();
}

size_t point_image_bytes(const Geom& g) {
  if (g.D > 64 || (g.D == 64 && !g.bf16)) return 0;
  const int ch = g.bf16 ? (g.D == 16 ? PointImages<true, 16>::kStride
                           : g.D == 32 ? PointImages<true, 32>::kStride : PointImages<true, 64>::kStride)
                        : (g.D == 16 ? PointImages<false, 16>::kStride : PointImages<false, 32>::kStride);
  return (size_t)g.BH() * ((g.G + 63) / 64) * ch * 16;
}

hipError_t run_pass_stats_pt(const Geom& g, const PassArgs& a, hipStream_t st) {
  // the point-owned passes' chunking; each workgroup sweeps its chunk in steps of 32 NW points
  const PassCfg cfg = pick_cfg(g, PASS_POINT);
  if (cfg.NP != FS_POINT_WAVES || g.D > 32 || g.G > 1024) return hipErrorInvalidConfiguration;
  const dim3 grid(cfg.chunks * g.BH()), block(64 * FS_STATS_WAVES);
#define FS_STATS(BF_, D_)                                                              \
  {                                                                                    \
    hipLaunchKernelGGL((k_stats_pt<BF_, D_, FS_STATS_WAVES>), grid, block, 0, st, a);  \
    return hipGetLastError();                                                          \
  }
  if (g.bf16 && g.D == 16) FS_STATS(true, 16)
  if (g.bf16 && g.D == 32) FS_STATS(true, 32)
  if (!g.bf16 && g.D == 16) FS_STATS(false, 16)
  if (!g.bf16 && g.D == 32) FS_STATS(false, 32)
#undef FS_STATS
  return hipErrorInvalidConfiguration;
}

namespace {
template <int ROLE>
hipError_t run_point_role(const Geom& g, const PassArgs& a, hipStream_t st) {
  const PassCfg cfg = pick_cfg(g, PASS_POINT);
  const int nw = g.D > 32 ? FS_POINT_WAVES_WIDE : FS_POINT_WAVES;
  if (cfg.NP != nw || g.D > 64 || (g.D > 32 && ROLE != 0)) return hipErrorInvalidConfiguration;
  uint4* img = static_cast<uint4*>(const_cast<void*>(a.img));
  const dim3 igrid(((g.G + 63) / 64) * g.BH()), iblock(64 * 11);
  const dim3 grid(cfg.chunks * g.BH()), block(64 * nw);
#define FS_POINT(BF_, D_, NW_)                                                             \
  {                                                                                        \
    hipLaunchKernelGGL((k_point_images<BF_, D_, ROLE>), igrid, iblock, 0, st, a, img);     \
    hipError_t e = hipGetLastError();                                                      \
    if (e != hipSuccess) return e;                                                         \
    hipLaunchKernelGGL((k_point<BF_, D_, NW_, ROLE>), grid, block, 0, st, a);              \
    return hipGetLastError();                                                              \
  }
  if (g.bf16 && g.D == 16) FS_POINT(true, 16, FS_POINT_WAVES)
  if (g.bf16 && g.D == 32) FS_POINT(true, 32, FS_POINT_WAVES)
  if (!g.bf16 && g.D == 16) FS_POINT(false, 16, FS_POINT_WAVES)
  if (!g.bf16 && g.D == 32) FS_POINT(false, 32, FS_POINT_WAVES)
  if constexpr (ROLE == 0) {  // head width 64: bf16 and the tied path only
    if (g.bf16 && g.D == 64) FS_POINT(true, 64, FS_POINT_WAVES_WIDE)
  }
#undef FS_POINT
  return hipErrorInvalidConfiguration;
}
}  // namespace

hipError_t run_pass_point(const Geom& g, const PassArgs& a, int role, hipStream_t st) {
  switch (role) {
    case 0: return run_point_role<0>(g, a, st);
    case 1: return run_point_role<1>(g, a, st);
    case 2: return run_point_role<2>(g, a, st);
    case 3: return run_point_role<3>(g, a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fs
