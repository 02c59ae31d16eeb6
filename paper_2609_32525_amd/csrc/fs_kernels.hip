// HIP kernels of the fused slice -> token mix -> deslice path for gfx950 (CDNA4).
//
// Streaming passes over the points (the hot path):
//   k_slice    logits -> per-point softmax over the slices -> U += w^T F, s += sum w, lse
//   k_deslice  logits -> w = exp(a - lse) -> out = w zmix
//   k_bwd_a    logits -> w -> dzmix += w^T dout
//   k_bwd_b    logits -> w -> dw = dout zmix^T + F dU^T + ds -> da = w (dw - sum_g w dw)
//              -> dx = da W_s^T / tau, dfx = w dU, and partials of dW_s, dbias, dtau
// (paper: Sec. 2 "The Transolver layer"; App. F.1 "Kernel design"; App. F.2 "Temperature
// gradients"; the backward is the exact derivative of the forward.)
//
// Design: a wavefront owns GS consecutive slots and a 32-point tile (two
// 16-point MFMA blocks); NS = G / GS wavefronts share one point tile and exchange per-point
// softmax statistics through LDS, so the slice weights never leave registers and no N x G
// tensor is ever written. The logits are an MFMA contraction over the head width; the
// token contractions are MFMAs over slots (deslice, dx, dfx) or over points (slice, dzmix,
// dW_s). fp32 storage uses v_mfma_f32_16x16x4_f32; bf16 storage uses
// v_mfma_f32_16x16x32_bf16 with the slice projection split into a high and a low bf16 part
// so the logits keep about 16 mantissa bits. The softmax works in base 2: the host-side
// constant log2(e)/tau is folded into W_s and the bias once per head.
//
// MFMA lane layouts used throughout (lane = 16 * j + i, 0 <= i < 16, 0 <= j < 4):
//   A operand A[m][k]: lane supplies m = i and a k-set that depends on j only;
//   B operand B[k][n]: lane supplies n = i and the same k-set;
//   C/D tile C[m][n]: lane holds rows m = 4 j + r (r = 0..3) of column n = i.
// The k-set is the same function of j for A and B, so any consistent assignment of the
// contraction index to (j, register) is a valid product; the code picks assignments that
// make global loads contiguous per lane.
//
// No atomics anywhere; all cross-workgroup sums are fixed-order reductions of partials.

#include <hip/hip_runtime.h>

#include "fs_internal.h"

namespace fs {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kMasked = 1.0e30f;  // base-2 lse of padding points: exp2(a - kMasked) == 0

__device__ __forceinline__ f4 mfma_f32(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f4 mfma_bf16(bf8 a, bf8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float bf_to_f(unsigned short h) {
  return __uint_as_float(((unsigned)h) << 16);
}
__device__ __forceinline__ unsigned short f_to_bf(float f) {
  return __builtin_bit_cast(unsigned short, (__bf16)f);  // round to nearest even
}
__device__ __forceinline__ f4 zero4() { return f4{0.f, 0.f, 0.f, 0.f}; }
__device__ __forceinline__ f4 splat4(float v) { return f4{v, v, v, v}; }

// Cross-lane reductions over the 16 lanes of a row (DPP: xor 1, xor 2, half-mirror, mirror).
// Every lane of the row ends with the same bitwise result (each step adds commuted pairs).
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  v = fmaxf(v, dpp<0x140>(v));
  return v;
}
__device__ __forceinline__ float row16_sum(float v) {
  v = v + dpp<0xB1>(v);
  v = v + dpp<0x4E>(v);
  v = v + dpp<0x141>(v);
  v = v + dpp<0x140>(v);
  return v;
}
// Sum over the four 16-lane rows (lanes i, i+16, i+32, i+48): identical result in all four.
__device__ __forceinline__ float col4_sum(float v) {
  v = v + __shfl_xor(v, 16);
  v = v + __shfl_xor(v, 32);
  return v;
}

// Orders LDS traffic between lanes of one wavefront (no s_barrier needed within a wave).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <bool BF>
struct Store;
template <>
struct Store<false> {
  using T = float;
};
template <>
struct Store<true> {
  using T = unsigned short;
};

template <bool BF>
__device__ __forceinline__ float ld1(const typename Store<BF>::T* p) {
  if constexpr (BF)
    return bf_to_f(*p);
  else
    return *p;
}

// ---------------------------------------------------------------------------------------
// Row operand of a 16-point block: lane (j, i) holds a contiguous segment of the row of
// point i. fp32: K = D/4 values, MFMA step kk uses column j*K + kk. bf16: one bf8 per K=32
// step; step kk holds columns kbase(j, kk) .. +7 (D = 16 pads rows j >= 2 with zeros).
// ---------------------------------------------------------------------------------------
template <bool BF, int D>
struct RowOp;
template <int D>
struct RowOp<false, D> {
  static constexpr int K = D / 4;
  float v[K];
};
template <int D>
struct RowOp<true, D> {
  static constexpr int K = (D + 31) / 32;
  bf8 v[K];
};

template <int D>
__device__ __forceinline__ int kbase_bf(int j, int kk) {
  return D == 64 ? 16 * j + 8 * kk : 8 * j;
}
// Column of K-slot (j, kk, e) of a bf16 row operand; -1 if it is padding.
template <int D>
__device__ __forceinline__ int kcol_bf(int j, int kk, int e) {
  if (D == 16 && j >= 2) return -1;
  return kbase_bf<D>(j, kk) + e;
}
// Column of K-slot (j, kk) of an fp32 row operand.
template <int D>
__device__ __forceinline__ int kcol_f(int j, int kk) {
  return j * (D / 4) + kk;
}

template <bool BF, int D>
__device__ __forceinline__ void load_row(RowOp<BF, D>& o, const typename Store<BF>::T* row,
                                         bool valid, int j) {
  if constexpr (!BF) {
    constexpr int K = D / 4;
    if (valid) {
      const float4* src = reinterpret_cast<const float4*>(row + j * K);
#pragma unroll
      for (int q = 0; q < K / 4; ++q) {
        float4 t = src[q];
        o.v[4 * q + 0] = t.x;
        o.v[4 * q + 1] = t.y;
        o.v[4 * q + 2] = t.z;
        o.v[4 * q + 3] = t.w;
      }
    } else {
#pragma unroll
      for (int q = 0; q < K; ++q) o.v[q] = 0.f;
    }
  } else {
    constexpr int K = (D + 31) / 32;
#pragma unroll
    for (int kk = 0; kk < K; ++kk) {
      if (valid && !(D == 16 && j >= 2)) {
        uint4 t = *reinterpret_cast<const uint4*>(row + kbase_bf<D>(j, kk));
        o.v[kk] = __builtin_bit_cast(bf8, t);
      } else {
        o.v[kk] = __builtin_bit_cast(bf8, uint4{0u, 0u, 0u, 0u});
      }
    }
  }
}

// ---------------------------------------------------------------------------------------
// Slot-range operand of a [rows = slots][cols = k] matrix for a contraction over k with the
// slot on the MFMA M (or N) index: lane (j, i) holds M(g0 + 16 gb + i, kcol(j, kk)).
// Used for the scaled slice projection (M(g, d) = W_s[d][g] * sc, W stored (D, G)) and for
// zmix / dU in dw (M(g, v) = Z[g][v], stored (G, V)). bf16 keeps a high and a low part.
// ---------------------------------------------------------------------------------------
template <bool BF, int D, int GB>
struct SlotOp;
template <int D, int GB>
struct SlotOp<false, D, GB> {
  float v[GB][D / 4];
};
template <int D, int GB>
struct SlotOp<true, D, GB> {
  static constexpr int K = (D + 31) / 32;
  bf8 hi[GB][K];
  bf8 lo[GB][K];
};

// TRANSPOSED = true: element (g, k) read from src[k * ld + g] (W_s (D,G)); else
// src[g * ld + k] - cen[k] (cen nullable: a per-column shift removed before rounding).
template <bool BF, int D, int GB, bool TRANSPOSED, bool SPLIT>
__device__ __forceinline__ void load_slotop(SlotOp<BF, D, GB>& o, const float* src, int ld,
                                            int g0, float sc, int i, int j,
                                            const float* cen = nullptr) {
  auto M = [&](int g, int k) -> float {
    if (TRANSPOSED) return sc * src[(int64_t)k * ld + g];
    return sc * (src[(int64_t)g * ld + k] - (cen != nullptr ? cen[k] : 0.f));
  };
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) {
    const int g = g0 + 16 * gb + i;
    if constexpr (!BF) {
#pragma unroll
      for (int kk = 0; kk < D / 4; ++kk) o.v[gb][kk] = M(g, kcol_f<D>(j, kk));
    } else {
#pragma unroll
      for (int kk = 0; kk < SlotOp<true, D, GB>::K; ++kk) {
        bf8 hi, lo;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int k = kcol_bf<D>(j, kk, e);
          float val = 0.f;
          if (k >= 0) val = M(g, k);
          const __bf16 h = (__bf16)val;
          hi[e] = h;
          lo[e] = SPLIT ? (__bf16)(val - (float)h) : (__bf16)0.f;
        }
        o.hi[gb][kk] = hi;
        o.lo[gb][kk] = lo;
      }
    }
  }
}

// acc += (slot operand) x (row operand)^T : T-layout tile (rows = slots, cols = points).
template <bool BF, int D, int GB, bool SPLIT>
__device__ __forceinline__ f4 mm_slot_row(const SlotOp<BF, D, GB>& s, int gb,
                                          const RowOp<BF, D>& r, f4 acc) {
  if constexpr (!BF) {
#pragma unroll
    for (int kk = 0; kk < D / 4; ++kk) acc = mfma_f32(s.v[gb][kk], r.v[kk], acc);
  } else {
#pragma unroll
    for (int kk = 0; kk < RowOp<true, D>::K; ++kk) {
      acc = mfma_bf16(s.hi[gb][kk], r.v[kk], acc);
      if constexpr (SPLIT) acc = mfma_bf16(s.lo[gb][kk], r.v[kk], acc);
    }
  }
  return acc;
}
// acc += (row operand) x (slot operand)^T : S-layout tile (rows = points, cols = slots).
template <bool BF, int D, int GB, bool SPLIT>
__device__ __forceinline__ f4 mm_row_slot(const RowOp<BF, D>& r, const SlotOp<BF, D, GB>& s,
                                          int gb, f4 acc) {
  if constexpr (!BF) {
#pragma unroll
    for (int kk = 0; kk < D / 4; ++kk) acc = mfma_f32(r.v[kk], s.v[gb][kk], acc);
  } else {
#pragma unroll
    for (int kk = 0; kk < RowOp<true, D>::K; ++kk) {
      acc = mfma_bf16(r.v[kk], s.hi[gb][kk], acc);
      if constexpr (SPLIT) acc = mfma_bf16(r.v[kk], s.lo[gb][kk], acc);
    }
  }
  return acc;
}

// ---------------------------------------------------------------------------------------
// Operand for a contraction over slots whose output rows are columns c of a slot-major
// matrix M(g, c): lane (j, i) supplies M(g, 16 cb + i) for g in its k-set.
//   fp32: k-set of (gb, r) is g0 + 16 gb + 4 j + r (one MFMA per (gb, r)).
//   bf16: k-set of pair q, element e: g0 + 32 q + 16 (e / 4) + 4 j + (e % 4).
// These k-sets coincide with the rows a T-layout tile holds, so the tile is the B operand.
// ---------------------------------------------------------------------------------------
template <bool BF, int GB, int CB>
struct GOp;
template <int GB, int CB>
struct GOp<false, GB, CB> {
  float v[GB][4][CB];
};
template <int GB, int CB>
struct GOp<true, GB, CB> {
  bf8 v[GB / 2][CB];
};

// TRANSPOSED = true: M(g, c) = src[c * ld + g] * sc, else src[g * ld + c] * sc.
template <bool BF, int GB, int CB, bool TRANSPOSED>
__device__ __forceinline__ void load_gop(GOp<BF, GB, CB>& o, const float* src, int ld, int g0,
                                         float sc, int i, int j) {
  auto M = [&](int g, int c) -> float {
    return sc * (TRANSPOSED ? src[(int64_t)c * ld + g] : src[(int64_t)g * ld + c]);
  };
  if constexpr (!BF) {
#pragma unroll
    for (int gb = 0; gb < GB; ++gb)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) o.v[gb][r][cb] = M(g0 + 16 * gb + 4 * j + r, 16 * cb + i);
  } else {
#pragma unroll
    for (int q = 0; q < GB / 2; ++q)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        bf8 t;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          t[e] = (__bf16)M(g0 + 32 * q + 16 * (e / 4) + 4 * j + (e % 4), 16 * cb + i);
        o.v[q][cb] = t;
      }
  }
}

// out[cb] (+)= M^T-contraction with a T-layout tile column block pb: rows c, cols points.
template <bool BF, int GB, int CB, int PB = 2>
__device__ __forceinline__ f4 mm_gop_tile(const GOp<BF, GB, CB>& o, int cb, const f4 (*t)[PB],
                                          int pb, f4 acc) {
  if constexpr (!BF) {
#pragma unroll
    for (int gb = 0; gb < GB; ++gb)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc = mfma_f32(o.v[gb][r][cb], t[gb][pb][r], acc);
  } else {
#pragma unroll
    for (int q = 0; q < GB / 2; ++q) {
      bf8 bt;
#pragma unroll
      for (int e = 0; e < 8; ++e) bt[e] = (__bf16)t[2 * q + e / 4][pb][e % 4];
      acc = mfma_bf16(o.v[q][cb], bt, acc);
    }
  }
  return acc;
}

// Operand rows of a point-major matrix P (row stride rs) for a contraction over the 32 points
// of a tile: lane (j, i) holds P(p, 16 cb + i) for the points of its k-set.
//   fp32: point 16 pb + 4 j + r for MFMA (pb, r);  bf16: point 16 (e / 4) + 4 j + (e % 4).
// Gathered separately from the MFMAs so that the next tile's loads can be issued early.
template <bool BF, int CB>
struct PtGather;
template <int CB>
struct PtGather<false, CB> {
  float v[2][4][CB];
};
template <int CB>
struct PtGather<true, CB> {
  bf8 v[CB];
};

template <bool BF, int CB>
__device__ __forceinline__ void gather_points(PtGather<BF, CB>& g,
                                              const typename Store<BF>::T* base, int64_t rs,
                                              int64_t p0, int64_t pend, int i, int j) {
  if constexpr (!BF) {
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t p = p0 + 16 * pb + 4 * j + r;
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) g.v[pb][r][cb] = p < pend ? base[p * rs + 16 * cb + i] : 0.f;
      }
  } else {
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      bf8 bt;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t p = p0 + 16 * (e / 4) + 4 * j + (e % 4);
        unsigned short h = 0;
        if (p < pend) h = base[p * rs + 16 * cb + i];
        bt[e] = __builtin_bit_cast(__bf16, h);
      }
      g.v[cb] = bt;
    }
  }
}

// acc[gb][cb] += (S-layout tile column gb)^T-contraction over the 32 points with the gathered
// rows: out(g, c) += sum_p w(p, g) P(p, 16 cb + i).
template <bool BF, int GB, int CB>
__device__ __forceinline__ void mm_points(f4 (*acc)[CB], const f4 (*w)[GB],
                                          const PtGather<BF, CB>& g) {
  if constexpr (!BF) {
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int gb = 0; gb < GB; ++gb) acc[gb][cb] = mfma_f32(w[pb][gb][r], g.v[pb][r][cb], acc[gb][cb]);
  } else {
    bf8 at[GB];
#pragma unroll
    for (int gb = 0; gb < GB; ++gb)
#pragma unroll
      for (int e = 0; e < 8; ++e) at[gb][e] = (__bf16)w[e / 4][gb][e % 4];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) acc[gb][cb] = mfma_bf16(at[gb], g.v[cb], acc[gb][cb]);
  }
}

// Register image of a per-wavefront operand in LDS: 16-byte chunk q of lane l at
// base[q * 64 + l], so every lane reads its own chunk and no two lanes share a bank group.
template <class Op>
__device__ __forceinline__ void lds_put(const Op& o, uint4* base, int lane) {
  static_assert(sizeof(Op) % 16 == 0, "operand image must be whole 16-byte chunks");
  const uint4* src = reinterpret_cast<const uint4*>(&o);
#pragma unroll
  for (int q = 0; q < (int)(sizeof(Op) / 16); ++q) base[q * 64 + lane] = src[q];
}
template <class Op>
__device__ __forceinline__ void lds_get(Op& o, const uint4* base, int lane) {
  uint4* dst = reinterpret_cast<uint4*>(&o);
#pragma unroll
  for (int q = 0; q < (int)(sizeof(Op) / 16); ++q) dst[q] = base[q * 64 + lane];
}
template <class Op>
constexpr int lds_chunks() {
  return (int)(sizeof(Op) / 16) * 64;
}

// ---------------------------------------------------------------------------------------
// Kernel arguments
// ---------------------------------------------------------------------------------------
struct PassArgs {
  const void* x;
  const void* fx;    // slice: F; bwd: F
  const void* dout;  // bwd
  void* out;         // deslice: O; bwd_b: dx
  void* out2;        // bwd_b: dfx
  const float* Ws;
  const float* bias;
  const float* tau;
  const float* zmix;  // deslice, bwd_b
  const float* dU;    // bwd_b
  const float* ds;    // bwd_b
  const float* cen;   // bwd_b: per (b,h) [V] slot-mean of zmix, [V] of dU, [1] of ds
  const float* lse_in;
  float* lse_out;
  float* part;   // slice: U partials; bwd_a: dzmix partials; bwd_b: parameter partials
  float* part2;  // slice: s partials
  int64_t N;
  int H, G;
  int ws_per_head;
  int chunks;
  int64_t chunk_pts;
};

struct HeadCtx {
  int bh, b, h, g0;
  float sc;  // log2(e) / tau_h
  const float* W;
  const float* bias;
  int64_t off;  // element offset of point 0 of this (b, h) in the (B, N, H, D) layout
};

template <int D>
__device__ __forceinline__ HeadCtx head_ctx(const PassArgs& a, int ws, int GS) {
  HeadCtx c;
  c.bh = blockIdx.y;
  c.b = c.bh / a.H;
  c.h = c.bh % a.H;
  c.g0 = ws * GS;
  c.sc = kLog2e / a.tau[c.h];
  c.W = a.Ws + (a.ws_per_head ? (int64_t)c.h * D * a.G : 0);
  c.bias = a.bias + (a.ws_per_head ? (int64_t)c.h * a.G : 0);
  c.off = ((int64_t)c.b * a.N * a.H + c.h) * D;
  return c;
}

// =======================================================================================
// Slice pass
// =======================================================================================
template <bool BF, int D, int GS, int NS, int NP>
__global__ __launch_bounds__(64 * NS * NP) void k_slice(PassArgs a) {
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
  load_slotop<BF, D, GB, true, SPLIT>(wop, c.W, a.G, c.g0, c.sc, i, j);
  float bS[GB];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) bS[gb] = c.sc * c.bias[c.g0 + 16 * gb + i];

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

  const int64_t pbeg = (int64_t)blockIdx.x * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int ntile = pend > pbeg ? (int)((pend - pbeg + 32 * NP - 1) / (32 * NP)) : 0;

  // software pipeline: the next tile's rows are loaded before the current tile is computed
  struct Tile {
    RowOp<BF, D> xo[2];
    PtGather<BF, VB> f;
  };
  auto load_tile = [&](Tile& tt, int t) {
    const int64_t p0 = pbeg + (int64_t)(t * NP + wp) * 32;
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const int64_t p = p0 + 16 * pb + i;
      load_row<BF, D>(tt.xo[pb], xb + p * rs, p < pend, j);
    }
    gather_points<BF, VB>(tt.f, fb, rs, p0, pend, i, j);
  };
  Tile cur;
  if (ntile > 0) load_tile(cur, 0);
  for (int t = 0; t < ntile; ++t) {
    const int64_t p0 = pbeg + (int64_t)(t * NP + wp) * 32;
    Tile nxt;
    if (t + 1 < ntile) load_tile(nxt, t + 1);
    const RowOp<BF, D>* xo = cur.xo;
    // S-layout logits: rows = points 16 pb + 4 j + r, cols = slots g0 + 16 gb + i
    f4 w[2][GB];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
        w[pb][gb] = mm_row_slot<BF, D, GB, SPLIT>(xo[pb], wop, gb, splat4(bS[gb]));

    float m[2][4], l[2][4];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float mx = w[pb][0][r];
#pragma unroll
        for (int gb = 1; gb < GB; ++gb) mx = fmaxf(mx, w[pb][gb][r]);
        m[pb][r] = row16_max(mx);
        float sum = 0.f;
#pragma unroll
        for (int gb = 0; gb < GB; ++gb) {
          const float e = __builtin_amdgcn_exp2f(w[pb][gb][r] - m[pb][r]);
          w[pb][gb][r] = e;
          sum += e;
        }
        l[pb][r] = row16_sum(sum);
      }

    float f[2][4], lse2[2][4];
    if constexpr (NS == 1) {
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          f[pb][r] = 1.0f / l[pb][r];
          lse2[pb][r] = m[pb][r] + __log2f(l[pb][r]);
        }
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
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int q = 16 * pb + 4 * j + r;
          float M = st_m[par][wp][0][q];
#pragma unroll
          for (int s = 1; s < NS; ++s) M = fmaxf(M, st_m[par][wp][s][q]);
          float L = 0.f;
#pragma unroll
          for (int s = 0; s < NS; ++s)
            L += st_l[par][wp][s][q] * __builtin_amdgcn_exp2f(st_m[par][wp][s][q] - M);
          f[pb][r] = __builtin_amdgcn_exp2f(m[pb][r] - M) / L;
          lse2[pb][r] = M + __log2f(L);
        }
    }

#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t p = p0 + 16 * pb + 4 * j + r;
        const float fr = p < pend ? f[pb][r] : 0.f;
#pragma unroll
        for (int gb = 0; gb < GB; ++gb) w[pb][gb][r] *= fr;
        if (a.lse_out != nullptr && ws == 0 && i == 0 && p < pend)
          a.lse_out[(int64_t)c.bh * a.N + p] = lse2[pb][r];
      }
#pragma unroll
    for (int gb = 0; gb < GB; ++gb) {
      float sum = 0.f;
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) sum += w[pb][gb][r];
      sacc[gb] += sum;
    }
    mm_points<BF, GB, VB>(U, w, cur.f);
    cur = nxt;
  }

  // ---- combine the NP point groups and write this workgroup's partials --------------------
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) sacc[gb] = col4_sum(sacc[gb]);
  float* pU = a.part + ((int64_t)c.bh * a.chunks + blockIdx.x) * a.G * D;
  float* pS = a.part2 + ((int64_t)c.bh * a.chunks + blockIdx.x) * a.G;
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
        for (int r = 0; r < 4; ++r)
          pU[(int64_t)(c.g0 + 16 * gb + 4 * j + r) * D + 16 * vb + i] = U[gb][vb][r];
      if (j == 0) pS[c.g0 + 16 * gb + i] = sacc[gb];
    }
  }
}

// =======================================================================================
// Deslice pass
// =======================================================================================
template <bool BF, int D, int GS, int NS, int NP>
__global__ __launch_bounds__(64 * NS * NP) void k_deslice(PassArgs a) {
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

  const int64_t pbeg = (int64_t)blockIdx.x * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int ntile = pend > pbeg ? (int)((pend - pbeg + 32 * NP - 1) / (32 * NP)) : 0;

  // software pipeline: the next tile's rows are loaded before the current tile is computed
  struct Tile {
    RowOp<BF, D> xo[2];
    float lse2[2];
  };
  auto load_tile = [&](Tile& tt, int t) {
    const int64_t p0 = pbeg + (int64_t)(t * NP + wp) * 32;
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const int64_t p = p0 + 16 * pb + i;
      load_row<BF, D>(tt.xo[pb], xb + p * rs, p < pend, j);
      tt.lse2[pb] = p < pend ? lse[p] : kMasked;
    }
  };
  Tile cur;
  if (ntile > 0) load_tile(cur, 0);
  for (int t = 0; t < ntile; ++t) {
    const int64_t p0 = pbeg + (int64_t)(t * NP + wp) * 32;
    Tile nxt;
    if (t + 1 < ntile) load_tile(nxt, t + 1);
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
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) o[vb][pb] = mm_gop_tile<BF, GB, VB>(zop, vb, w, pb, zero4());

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
      for (int pb = 0; pb < 2; ++pb) {
        const int64_t p = p0 + 16 * pb + i;
        if (p < pend) {
#pragma unroll
          for (int vb = 0; vb < VB; ++vb) {
            T* dst = ob + p * rs + 16 * vb + 4 * j;
            if constexpr (!BF) {
              *reinterpret_cast<float4*>(dst) =
                  float4{o[vb][pb][0], o[vb][pb][1], o[vb][pb][2], o[vb][pb][3]};
            } else {
              const unsigned lo = f_to_bf(o[vb][pb][0]) | ((unsigned)f_to_bf(o[vb][pb][1]) << 16);
              const unsigned hi = f_to_bf(o[vb][pb][2]) | ((unsigned)f_to_bf(o[vb][pb][3]) << 16);
              *reinterpret_cast<uint2*>(dst) = uint2{lo, hi};
            }
          }
        }
      }
    }
    cur = nxt;
  }
}

// =======================================================================================
// Backward pass A: dzmix = w^T dout (partials per workgroup)
// =======================================================================================
template <bool BF, int D, int GS, int NS, int NP>
__global__ __launch_bounds__(64 * NS * NP) void k_bwd_a(PassArgs a) {
  constexpr int GB = GS / 16, VB = D / 16;
  constexpr bool SPLIT = BF;
  using T = typename Store<BF>::T;
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int wave = threadIdx.x >> 6, ws = wave % NS, wp = wave / NS;
  const HeadCtx c = head_ctx<D>(a, ws, GS);
  const int64_t rs = (int64_t)a.H * D;
  const T* xb = (const T*)a.x + c.off;
  const T* db = (const T*)a.dout + c.off;
  const float* lse = a.lse_in + (int64_t)c.bh * a.N;

  SlotOp<BF, D, GB> wop;
  load_slotop<BF, D, GB, true, SPLIT>(wop, c.W, a.G, c.g0, c.sc, i, j);
  float bS[GB];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) bS[gb] = c.sc * c.bias[c.g0 + 16 * gb + i];
  f4 Z[GB][VB];
#pragma unroll
  for (int gb = 0; gb < GB; ++gb)
#pragma unroll
    for (int vb = 0; vb < VB; ++vb) Z[gb][vb] = zero4();

  const int64_t pbeg = (int64_t)blockIdx.x * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int ntile = pend > pbeg ? (int)((pend - pbeg + 32 * NP - 1) / (32 * NP)) : 0;

  // software pipeline: the next tile's rows are loaded before the current tile is computed
  struct Tile {
    RowOp<BF, D> xo[2];
    float lse2[2][4];
    PtGather<BF, VB> g;
  };
  auto load_tile = [&](Tile& tt, int t) {
    const int64_t p0 = pbeg + (int64_t)(t * NP + wp) * 32;
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const int64_t p = p0 + 16 * pb + i;
      load_row<BF, D>(tt.xo[pb], xb + p * rs, p < pend, j);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t q = p0 + 16 * pb + 4 * j + r;
        tt.lse2[pb][r] = q < pend ? lse[q] : kMasked;
      }
    }
    gather_points<BF, VB>(tt.g, db, rs, p0, pend, i, j);
  };
  Tile cur;
  if (ntile > 0) load_tile(cur, 0);
  for (int t = 0; t < ntile; ++t) {
    Tile nxt;
    if (t + 1 < ntile) load_tile(nxt, t + 1);
    const RowOp<BF, D>* xo = cur.xo;
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
    mm_points<BF, GB, VB>(Z, w, cur.g);
    cur = nxt;
  }

  float* pZ = a.part + ((int64_t)c.bh * a.chunks + blockIdx.x) * a.G * D;
  if constexpr (NP > 1) {
    __shared__ f4 red[NP - 1][NS][GB][VB][64];
    if (wp > 0) {
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
#pragma unroll
        for (int vb = 0; vb < VB; ++vb) red[wp - 1][ws][gb][vb][lane] = Z[gb][vb];
    }
    __syncthreads();
    if (wp == 0) {
      for (int q = 0; q < NP - 1; ++q)
#pragma unroll
        for (int gb = 0; gb < GB; ++gb)
#pragma unroll
          for (int vb = 0; vb < VB; ++vb) Z[gb][vb] += red[q][ws][gb][vb][lane];
    }
  }
  if (wp == 0) {
#pragma unroll
    for (int gb = 0; gb < GB; ++gb)
#pragma unroll
      for (int vb = 0; vb < VB; ++vb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          pZ[(int64_t)(c.g0 + 16 * gb + 4 * j + r) * D + 16 * vb + i] = Z[gb][vb][r];
  }
}

// =======================================================================================
// Backward pass B: point gradients and parameter partials
// partial layout per workgroup: [D * G] dW_s (row-major (D, G)), [G] dbias, [2] fp64 dtau
// PB: 16-point blocks per tile (1 or 2; bf16 needs 2: its contraction over points has K=32).
// With at most two slot groups, the per-head operands live in LDS as register images shared
// by the workgroup's wavefronts and are read where they are used, which keeps the register
// count (and so the number of resident wavefronts) in line with the other passes.
// =======================================================================================
template <bool BF, int D, int GS, int NS, int NP, int PB>
__global__ __launch_bounds__(64 * NS * NP) void k_bwd_b(PassArgs a) {
  static_assert(PB == 2 || !BF, "bf16 contracts over 32 points");
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
      bT[gb][r] = c.sc * c.bias[c.g0 + 16 * gb + 4 * j + r];
      dsT[gb][r] = a.ds[(int64_t)c.bh * a.G + c.g0 + 16 * gb + 4 * j + r] - cen[2 * D];
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
      load_slotop<BF, D, GB, true, SPLIT>(t0, c.W, a.G, c.g0, c.sc, i, j);
      load_slotop<BF, D, GB, false, false>(t1, zm, D, c.g0, 1.0f, i, j, cen);
      load_slotop<BF, D, GB, false, false>(t2, dU, D, c.g0, 1.0f, i, j, cen + D);
      load_gop<BF, GB, VB, false>(t3, dU, D, c.g0, 1.0f, i, j);
      load_gop<BF, GB, DB, true>(t4, c.W, a.G, c.g0, inv_tau, i, j);
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
  // gx: [NP][NS][VB][PB][64] f4; da transpose: fp32 [TP points][GS + 1], bf16 [GS slots][40].
  constexpr int kDaWords = BF ? (GS * 40 + 1) / 2 : TP * (GS + 1);
  constexpr size_t kGxBytes = NS > 1 ? (size_t)NP * NS * VB * PB * 64 * sizeof(f4) : 0;
  constexpr size_t kDaBytes = (size_t)NS * NP * kDaWords * sizeof(float);
  __shared__ __attribute__((aligned(16))) char smem[kGxBytes > kDaBytes ? kGxBytes : kDaBytes];
  f4* gx = reinterpret_cast<f4*>(smem);
  float* myda = reinterpret_cast<float*>(smem) + (size_t)wave * kDaWords;

  const int64_t pbeg = (int64_t)blockIdx.x * a.chunk_pts;
  const int64_t pend = min(a.N, pbeg + a.chunk_pts);
  const int ntile = pend > pbeg ? (int)((pend - pbeg + TP * NP - 1) / (TP * NP)) : 0;

  for (int t = 0; t < ntile; ++t) {
    const int64_t p0 = pbeg + (int64_t)(t * NP + wp) * TP;
    RowOp<BF, D> xo[PB], go[PB], fo[PB];
    float lse2[PB];
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int64_t p = p0 + 16 * pb + i;
      const bool ok = p < pend;
      load_row<BF, D>(xo[pb], xb + p * rs, ok, j);
      load_row<BF, D>(go[pb], gb_ + p * rs, ok, j);
      load_row<BF, D>(fo[pb], fb + p * rs, ok, j);
      lse2[pb] = ok ? lse[p] : kMasked;
    }
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
          g = mm_slot_row<BF, D, GB, false>(zv, gb, go[pb], g);
          g = mm_slot_row<BF, D, GB, false>(uv, gb, fo[pb], g);
          dw[gb][pb] = g;
        }
    }
    // per point (column of the tile): c = sum_g w dw, the softmax correction, and
    // tb = sum_g w t, the weighted mean of the shifted base-2 logits t = a2 - lse2
    float cc[PB], tb[PB];
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
        for (int vb = 0; vb < VB; ++vb) gf[vb][pb] = mm_gop_tile<BF, GB, VB, PB>(ug, vb, w, pb, zero4());
#pragma unroll
        for (int d = 0; d < DB; ++d) gx_[d][pb] = mm_gop_tile<BF, GB, DB, PB>(wg, d, dw, pb, zero4());
      }
    }
    if constexpr (NS > 1) {
      __syncthreads();  // every wave has read cx and finished the previous da transposes
#pragma unroll
      for (int half = 0; half < 2; ++half) {
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
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        const int64_t p = p0 + 16 * pb + i;
        if (p < pend) {
#pragma unroll
          for (int cb = 0; cb < VB; ++cb) {
            T* d1 = dfb + p * rs + 16 * cb + 4 * j;
            T* d2 = dxb + p * rs + 16 * cb + 4 * j;
            if constexpr (!BF) {
              *reinterpret_cast<float4*>(d1) =
                  float4{gf[cb][pb][0], gf[cb][pb][1], gf[cb][pb][2], gf[cb][pb][3]};
              *reinterpret_cast<float4*>(d2) =
                  float4{gx_[cb][pb][0], gx_[cb][pb][1], gx_[cb][pb][2], gx_[cb][pb][3]};
            } else {
              *reinterpret_cast<uint2*>(d1) =
                  uint2{f_to_bf(gf[cb][pb][0]) | ((unsigned)f_to_bf(gf[cb][pb][1]) << 16),
                        f_to_bf(gf[cb][pb][2]) | ((unsigned)f_to_bf(gf[cb][pb][3]) << 16)};
              *reinterpret_cast<uint2*>(d2) =
                  uint2{f_to_bf(gx_[cb][pb][0]) | ((unsigned)f_to_bf(gx_[cb][pb][1]) << 16),
                        f_to_bf(gx_[cb][pb][2]) | ((unsigned)f_to_bf(gx_[cb][pb][3]) << 16)};
            }
          }
        }
      }
    }
    // dW_s += X^T da over the tile's points: da goes through LDS to put points on the k index.
    if constexpr (!BF) {
      // myda[p * (GS + 1) + gl]
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r) myda[(16 * pb + i) * (GS + 1) + 16 * gb + 4 * j + r] = dw[gb][pb][r];
      wave_lds_sync();
#pragma unroll
      for (int pb = 0; pb < PB; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pl = 16 * pb + 4 * j + r;
          const int64_t p = p0 + pl;
          float xv[DB];
#pragma unroll
          for (int d = 0; d < DB; ++d) xv[d] = p < pend ? xb[p * rs + 16 * d + i] : 0.f;
#pragma unroll
          for (int gb = 0; gb < GB; ++gb) {
            const float bv = myda[pl * (GS + 1) + 16 * gb + i];
#pragma unroll
            for (int d = 0; d < DB; ++d) dW[d][gb] = mfma_f32(xv[d], bv, dW[d][gb]);
          }
        }
      wave_lds_sync();
    } else {
      unsigned short* t16 = reinterpret_cast<unsigned short*>(myda);  // [GS][40]
#pragma unroll
      for (int gb = 0; gb < GB; ++gb)
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r) t16[(16 * gb + 4 * j + r) * 40 + 16 * pb + i] = f_to_bf(dw[gb][pb][r]);
      wave_lds_sync();
      bf8 xa[DB];
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int64_t p = p0 + 16 * (e / 4) + 4 * j + (e % 4);
          unsigned short h = 0;
          if (p < pend) h = xb[p * rs + 16 * d + i];
          xa[d][e] = __builtin_bit_cast(__bf16, h);
        }
#pragma unroll
      for (int gb = 0; gb < GB; ++gb) {
        const uint2 lo = *reinterpret_cast<const uint2*>(t16 + (16 * gb + i) * 40 + 4 * j);
        const uint2 hi = *reinterpret_cast<const uint2*>(t16 + (16 * gb + i) * 40 + 16 + 4 * j);
        const bf8 bt = __builtin_bit_cast(bf8, uint4{lo.x, lo.y, hi.x, hi.y});
#pragma unroll
        for (int d = 0; d < DB; ++d) dW[d][gb] = mfma_bf16(xa[d], bt, dW[d][gb]);
      }
      wave_lds_sync();
    }
  }

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

  float* pp = a.part + ((int64_t)c.bh * a.chunks + blockIdx.x) * ((int64_t)D * a.G + a.G + 2);
  if constexpr (NP > 1) {
    __shared__ f4 red[NP - 1][NS][DB][GB][64];
    __shared__ float redb[NP - 1][NS][GB][4][16];
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
          pp[(int64_t)(16 * d + 4 * j + r) * a.G + c.g0 + 16 * gb + i] = dW[d][gb][r] * inv_tau;
      if (i == 0)
#pragma unroll
        for (int r = 0; r < 4; ++r) pp[(int64_t)D * a.G + c.g0 + 16 * gb + 4 * j + r] = dbv[gb][r] * inv_tau;
    }
  }
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int q = 0; q < NS * NP; ++q) s += dtw[q];
    // (D * G + G) is even, so this slot is 8-byte aligned
    *reinterpret_cast<double*>(pp + (int64_t)D * a.G + a.G) = -s * (double)kLn2 * (double)inv_tau;
  }
}

// =======================================================================================
// Dispatch over the compile-time tiling
// =======================================================================================
#define FS_DISPATCH_KERNEL(KNAME, ...)                                                      \
  template <bool BF, int D, int GS, int NS, int NP, int PB>                                \
  hipError_t run_##KNAME(const PassCfg& cfg, int BH, const PassArgs& a, hipStream_t st) {  \
    dim3 grid(cfg.chunks, BH);                                                             \
    hipLaunchKernelGGL((KNAME<__VA_ARGS__>), grid, dim3(64 * NS * NP), 0, st, a);          \
    return hipGetLastError();                                                              \
  }
FS_DISPATCH_KERNEL(k_slice, BF, D, GS, NS, NP)
FS_DISPATCH_KERNEL(k_deslice, BF, D, GS, NS, NP)
FS_DISPATCH_KERNEL(k_bwd_a, BF, D, GS, NS, NP)
FS_DISPATCH_KERNEL(k_bwd_b, BF, D, GS, NS, NP, PB)

// Supported (GS, NS, NP, PB) tilings; pick_cfg in fs_api.cpp chooses among exactly these.
// PB = 1 (16-point tiles) exists for the fp32 backward pass B only.
#define FS_TILINGS(X, BF, D)                                                              \
  X(BF, D, 16, 1, 4, 2) X(BF, D, 32, 1, 4, 2) X(BF, D, 64, 1, 4, 2) X(BF, D, 64, 2, 2, 2) \
  X(BF, D, 64, 4, 1, 2) X(BF, D, 64, 8, 1, 2) X(BF, D, 64, 16, 1, 2)                     \
  X(BF, D, 16, 1, 4, 1) X(BF, D, 32, 1, 4, 1) X(BF, D, 64, 1, 4, 1)

template <int PASS, bool BF, int D>
hipError_t run_tiled(const PassCfg& cfg, int BH, const PassArgs& a, hipStream_t st) {
#define FS_CASE(BF_, D_, GS_, NS_, NP_, PB_)                                                   \
  if (cfg.GS == GS_ && cfg.NS == NS_ && cfg.NP == NP_ && cfg.PB == PB_) {                      \
    if constexpr (!(BF_ && GS_ < 32) && (PB_ == 2 || (!BF_ && PASS == PASS_BWD_B))) {          \
      if constexpr (PASS == PASS_SLICE) return run_k_slice<BF_, D_, GS_, NS_, NP_, PB_>(cfg, BH, a, st);     \
      if constexpr (PASS == PASS_DESLICE) return run_k_deslice<BF_, D_, GS_, NS_, NP_, PB_>(cfg, BH, a, st); \
      if constexpr (PASS == PASS_BWD_A) return run_k_bwd_a<BF_, D_, GS_, NS_, NP_, PB_>(cfg, BH, a, st);     \
      if constexpr (PASS == PASS_BWD_B) return run_k_bwd_b<BF_, D_, GS_, NS_, NP_, PB_>(cfg, BH, a, st);     \
    }                                                                                          \
  }
  FS_TILINGS(FS_CASE, BF, D)
#undef FS_CASE
  return hipErrorInvalidConfiguration;
}

template <int PASS>
hipError_t run_pass_impl(const Geom& g, const PassArgs& a, hipStream_t st) {
  const PassCfg cfg = pick_cfg(g, (Pass)PASS);
  const int BH = g.BH();
  if (g.bf16) {
    if (g.D == 16) return run_tiled<PASS, true, 16>(cfg, BH, a, st);
    if (g.D == 32) return run_tiled<PASS, true, 32>(cfg, BH, a, st);
    if (g.D == 64) return run_tiled<PASS, true, 64>(cfg, BH, a, st);
  } else {
    if (g.D == 16) return run_tiled<PASS, false, 16>(cfg, BH, a, st);
    if (g.D == 32) return run_tiled<PASS, false, 32>(cfg, BH, a, st);
    if (g.D == 64) return run_tiled<PASS, false, 64>(cfg, BH, a, st);
  }
  return hipErrorInvalidConfiguration;
}

// Launch one streaming pass, bracketed by the caller's measurement events if requested.
template <int PASS>
hipError_t run_pass(const Geom& g, const PassArgs& a, hipStream_t st) {
  const PassEvents& ev = pass_events();
  if (ev.before[PASS] != nullptr) {
    hipError_t e = hipEventRecord(ev.before[PASS], st);
    if (e != hipSuccess) return e;
  }
  hipError_t e = run_pass_impl<PASS>(g, a, st);
  if (e == hipSuccess && ev.after[PASS] != nullptr) e = hipEventRecord(ev.after[PASS], st);
  return e;
}

PassArgs base_args(const Geom& g, Pass p) {
  PassArgs a{};
  const PassCfg cfg = pick_cfg(g, p);
  a.N = g.N;
  a.H = g.H;
  a.G = g.G;
  a.ws_per_head = g.ws_per_head ? 1 : 0;
  a.chunks = cfg.chunks;
  a.chunk_pts = cfg.chunk_pts;
  return a;
}

inline hipError_t first_err(hipError_t a, hipError_t b) { return a != hipSuccess ? a : b; }

}  // namespace

// =======================================================================================
// Launchers
// =======================================================================================
hipError_t launch_slice(const Geom& g, const void* x, const void* fx, const float* Ws,
                        const float* bias, const float* tau, float* z, float* s, float* lse,
                        float* partU, float* partS, hipStream_t st) {
  PassArgs a = base_args(g, PASS_SLICE);
  a.x = x;
  a.fx = fx;
  a.Ws = Ws;
  a.bias = bias;
  a.tau = tau;
  a.lse_out = lse;
  a.part = partU;
  a.part2 = partS;
  hipError_t e = run_pass<PASS_SLICE>(g, a, st);
  if (e != hipSuccess) return e;
  return launch_reduce_tokens(g, partU, partS, a.chunks, z, s, st);
}

hipError_t launch_deslice(const Geom& g, const void* x, const float* Ws, const float* bias,
                          const float* tau, const float* zmix, const float* lse, void* out,
                          hipStream_t st) {
  PassArgs a = base_args(g, PASS_DESLICE);
  a.x = x;
  a.Ws = Ws;
  a.bias = bias;
  a.tau = tau;
  a.zmix = zmix;
  a.lse_in = lse;
  a.out = out;
  return run_pass<PASS_DESLICE>(g, a, st);
}

hipError_t launch_bwd(const Geom& g, const MixArgs& m, const void* x, const void* fx,
                      const float* Ws, const float* bias, const float* tau, const float* z,
                      const float* s, const float* zmix, const float* attn, const float* lse,
                      const void* dout, void* dx, void* dfx, float* dWs, float* dbias,
                      float* dtau, float* dmix, float* dzm_out, char* ws, hipStream_t st) {
  const BwdWs L = bwd_ws_layout(g, m.kind);
  float* partDZ = reinterpret_cast<float*>(ws + L.partDZ);
  float* dzm = dzm_out != nullptr ? dzm_out : reinterpret_cast<float*>(ws + L.dzm);
  float* dz = reinterpret_cast<float*>(ws + L.dz);
  float* dU = reinterpret_cast<float*>(ws + L.dU);
  float* dsv = reinterpret_cast<float*>(ws + L.ds);
  float* partP = reinterpret_cast<float*>(ws + L.partP);
  float* partM = reinterpret_cast<float*>(ws + L.partM);
  // pass A: dzmix = w^T dout
  PassArgs a = base_args(g, PASS_BWD_A);
  a.x = x;
  a.dout = dout;
  a.Ws = Ws;
  a.bias = bias;
  a.tau = tau;
  a.lse_in = lse;
  a.part = partDZ;
  hipError_t e = run_pass<PASS_BWD_A>(g, a, st);
  if (e != hipSuccess) return e;
  e = launch_reduce_rows(g, partDZ, dzm, a.chunks, (int64_t)g.G * g.V, st);
  if (e != hipSuccess) return e;
  // mix backward: dz, dU, ds, the slot-mean shifts (+ parameter gradients)
  float* cen = reinterpret_cast<float*>(ws + L.cen);
  e = launch_mix_bwd(g, m, z, s, zmix, attn, dzm, dz, dU, dsv, cen,
                     reinterpret_cast<float*>(ws + L.scr), partM, dmix, st);
  if (e != hipSuccess) return e;
  // pass B
  PassArgs b = base_args(g, PASS_BWD_B);
  b.x = x;
  b.fx = fx;
  b.dout = dout;
  b.out = dx;
  b.out2 = dfx;
  b.Ws = Ws;
  b.bias = bias;
  b.tau = tau;
  b.zmix = zmix;
  b.dU = dU;
  b.ds = dsv;
  b.cen = cen;
  b.lse_in = lse;
  b.part = partP;
  e = run_pass<PASS_BWD_B>(g, b, st);
  if (e != hipSuccess) return e;
  e = launch_reduce_params(g, partP, dWs, dbias, dtau, b.chunks, st);
  return e;
}

}  // namespace fs
