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
// so the logits keep about 16 mantissa bits. The softmax works in base 2: each workgroup
// folds log2(e)/tau_h into W_s and the bias as it loads them.
//
// MFMA lane layouts used throughout (lane = 16 * j + i, 0 <= i < 16, 0 <= j < 4):
//   A operand A[m][k]: lane supplies m = i and a k-set that depends on j only;
//   B operand B[k][n]: lane supplies n = i and the same k-set;
//   C/D tile C[m][n]: lane holds rows m = 4 j + r (r = 0..3) of column n = i.
// The k-set is the same function of j for A and B, so any consistent assignment of the
// contraction index to (j, register) is a valid product; the code picks assignments that
// make global loads contiguous per lane.
//
// This header holds what the four passes share (one translation unit per pass includes it):
// MFMA wrappers and operand layouts, cross-lane reductions, the per-(sample, head) context,
// and the dispatch over the compile-time tilings.
#pragma once

#include <hip/hip_runtime.h>

#include "fs_internal.h"

namespace fs {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kMasked = 1.0e30f;  // base-2 lse of padding points: exp2(a - kMasked) == 0
// Base-2 logit of a padding slot (slot counts that are not a whole number of 16-slot tiles per
// wave are padded up): its weight exp2(kMaskedSlot - m) is exactly 0 and, being finite, it
// leaves every product with a zero weight or gradient at zero.
constexpr float kMaskedSlot = -1.0e30f;

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
// 16 bytes as a native vector: copies of HIP's uint4 struct are memcpys, which can keep the
// array they read or write in memory instead of registers
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef float fl2 __attribute__((ext_vector_type(2)));
typedef __bf16 bfl2 __attribute__((ext_vector_type(2)));
// Two floats rounded to bf16 (nearest even) in one 32-bit word, the first in the low half.
__device__ __forceinline__ unsigned bf_pair(float a, float b) {
  return __builtin_bit_cast(unsigned, __builtin_convertvector(fl2{a, b}, bfl2));
}
// The 8 values a[0..3], b[0..3] as one bf16 MFMA operand (element e from a for e < 4).
__device__ __forceinline__ bf8 to_bf8(const f4& a, const f4& b) {
  return __builtin_bit_cast(bf8, uint4{bf_pair(a[0], a[1]), bf_pair(a[2], a[3]), bf_pair(b[0], b[1]),
                                       bf_pair(b[2], b[3])});
}
// The same 8 values in two bf16 parts, hi = RN(v) and lo = RN(v - hi), whose sum keeps about
// 16 significant bits. Each pair's rounded high parts are read back from their packed word (a
// shift and a mask) instead of being converted one by one.
__device__ __forceinline__ void split_bf8(const f4& a, const f4& b, bf8& hi, bf8& lo) {
  const float v[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  unsigned h[4], l[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    h[k] = bf_pair(v[2 * k], v[2 * k + 1]);
    const float h0 = __uint_as_float(h[k] << 16), h1 = __uint_as_float(h[k] & 0xffff0000u);
    l[k] = bf_pair(v[2 * k] - h0, v[2 * k + 1] - h1);
  }
  hi = __builtin_bit_cast(bf8, uint4{h[0], h[1], h[2], h[3]});
  lo = __builtin_bit_cast(bf8, uint4{l[0], l[1], l[2], l[3]});
}
__device__ __forceinline__ f4 zero4() { return f4{0.f, 0.f, 0.f, 0.f}; }
__device__ __forceinline__ f4 splat4(float v) { return f4{v, v, v, v}; }

// Cross-lane reductions over the 16 lanes of a row (DPP: xor 1, xor 2, half-mirror, mirror).
// Every lane of the row ends with the same bitwise result (each step adds commuted pairs).
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  // every lane's source lies in its own row for these patterns, so no lane keeps an old value
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}
// IEEE maximum (v_maximum3_f32): unlike fmaxf it needs no canonicalising of its inputs.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float row16_max(float v) {
  v = vmax(v, dpp<0xB1>(v));
  v = vmax(v, dpp<0x4E>(v));
  v = vmax(v, dpp<0x141>(v));
  v = vmax(v, dpp<0x140>(v));
  return v;
}
__device__ __forceinline__ float row16_sum(float v) {
  v = v + dpp<0xB1>(v);
  v = v + dpp<0x4E>(v);
  v = v + dpp<0x141>(v);
  v = v + dpp<0x140>(v);
  return v;
}
// The same reductions over several independent values at once, one butterfly step for all of
// them before the next: consecutive DPP reads of a just-written register need wait states,
// which the other values' steps fill.
template <int N>
__device__ __forceinline__ void row16_max_n(float (&v)[N]) {
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = vmax(v[k], dpp<0xB1>(v[k]));
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = vmax(v[k], dpp<0x4E>(v[k]));
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = vmax(v[k], dpp<0x141>(v[k]));
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = vmax(v[k], dpp<0x140>(v[k]));
}
template <int N>
__device__ __forceinline__ void row16_sum_n(float (&v)[N]) {
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = v[k] + dpp<0xB1>(v[k]);
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = v[k] + dpp<0x4E>(v[k]);
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = v[k] + dpp<0x141>(v[k]);
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = v[k] + dpp<0x140>(v[k]);
}
// Sum over the four 16-lane rows (lanes i, i+16, i+32, i+48): identical result in all four.
// VALU lane swaps instead of LDS permutes: the 32-lane swap pairs row r with row r ^ 2, the
// 16-lane swap then pairs odd rows with even ones; each pair is added in the same order in
// both of its rows.
__device__ __forceinline__ float col4_sum(float v) {
  const unsigned u = __float_as_uint(v);
  const auto h = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const float s = __uint_as_float(h[0]) + __uint_as_float(h[1]);
  const unsigned us = __float_as_uint(s);
  const auto q = __builtin_amdgcn_permlane16_swap(us, us, false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}
// Maximum over the four 16-lane rows, by the same two lane swaps.
__device__ __forceinline__ float col4_max(float v) {
  const unsigned u = __float_as_uint(v);
  const auto h = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const float s = vmax(__uint_as_float(h[0]), __uint_as_float(h[1]));
  const unsigned us = __float_as_uint(s);
  const auto q = __builtin_amdgcn_permlane16_swap(us, us, false, false);
  return vmax(__uint_as_float(q[0]), __uint_as_float(q[1]));
}

// Orders LDS traffic between lanes of one wavefront (no s_barrier needed within a wave).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---- da transposes through a wavefront's LDS rows (dW_s = X^T da needs the points on the
// MFMA k index, da comes out of the logits product with the slots there). The LDS serves 32
// banks of 4 bytes; 4-byte accesses go 32 lanes a pass, 8-byte ones 16.
//  bf16: one row per slot, its 32 points in 36 halves (18 words), so the 16 rows that one
//        8-byte read pass touches start on 16 distinct even banks (no pass meets a bank
//        twice);
//  fp32: one row per point, GS + 1 words: two lanes share a bank in each pass. The layouts
//        without that (the slot index XORed with the point's low bits) cost the fp32 kernels
//        an address register per row offset, and spills where the registers are tight.
constexpr int kDaPitchBf = 36;
template <bool BF, int GS, int TP>
constexpr int da_words() {
  return BF ? GS * kDaPitchBf / 2 : TP * (GS + 1);
}
template <int GS>
__device__ __forceinline__ int da_at(int p, int g) {
  return p * (GS + 1) + g;
}
// da tile (T layout: slot 16 gb + 4 j + r, point 16 pb + i) into the bf16 rows
template <int GB, int PB>
__device__ __forceinline__ void da_put_bf(unsigned short* t16, const f4 (&da)[GB][PB], int i, int j) {
#pragma unroll
  for (int gb = 0; gb < GB; ++gb)
#pragma unroll
    for (int pb = 0; pb < PB; ++pb)
#pragma unroll
      for (int r = 0; r < 4; ++r) t16[(16 * gb + 4 * j + r) * kDaPitchBf + 16 * pb + i] = f_to_bf(da[gb][pb][r]);
}
// the B operand of slot block gb: slot 16 gb + i, points 4 j .. 4 j + 3 and 16 + 4 j .. + 3
__device__ __forceinline__ bf8 da_get_bf(const unsigned short* t16, int gb, int i, int j) {
  const unsigned short* row = t16 + (16 * gb + i) * kDaPitchBf;
  const uint2 lo = *reinterpret_cast<const uint2*>(row + 4 * j);
  const uint2 hi = *reinterpret_cast<const uint2*>(row + 16 + 4 * j);
  return __builtin_bit_cast(bf8, uint4{lo.x, lo.y, hi.x, hi.y});
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

// ---------------------------------------------------------------------------------------
// Raw buffer access to the point rows of one workgroup's (b, h, chunk): byte offsets are
// 32-bit and relative to the chunk's first point; a tile's base goes in the scalar offset,
// the lane's part in the vector offset. The record count ends at the last valid point's
// final column of this head, so the hardware returns zero for loads past the chunk and
// drops stores there: ragged tails need no branches or exec-mask juggling.
// ---------------------------------------------------------------------------------------
constexpr int kRsrcWord3 = 0x00020000;  // gfx9 raw buffer descriptor, dword data format

template <class T>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const T* first_row, int npts,
                                                            int rs, int cols) {
  const int bytes = npts > 0 ? (int)(((int64_t)(npts - 1) * rs + cols) * (int64_t)sizeof(T)) : 0;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(first_row), (short)0, bytes, kRsrcWord3);
}
__device__ __forceinline__ f4 bld128(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ uint4 bld128u(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ float bld32(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}
__device__ __forceinline__ unsigned short bld16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(unsigned short, __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0));
}
// A store of more than 64 bits reads its data registers after it issues; an instruction that
// overwrites them right behind it corrupted the first dword of some lanes under heavy memory
// traffic (seen with the accumulator-read that followed a 128-bit store). The no-op below
// takes the data as an input, so the registers stay live up to it, and it supplies the wait
// states before anything may reuse them.
__device__ __forceinline__ void bst128(__amdgpu_buffer_rsrc_t r, f4 v, int voff, int soff) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(r, 0, 0, 0)), v), r, voff, soff, 0);
  asm volatile("s_nop 1" ::"v"(v));
}
__device__ __forceinline__ void bst64(__amdgpu_buffer_rsrc_t r, uint2 v, int voff, int soff) {
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(r, 0, 0, 0)), v), r, voff, soff, 0);
}
__device__ __forceinline__ void bst32(__amdgpu_buffer_rsrc_t r, float v, int voff, int soff) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), r, voff, soff, 0);
}
// Four values of one row in the storage dtype, at byte offset voff + soff.
template <bool BF>
__device__ __forceinline__ void bst_row4(__amdgpu_buffer_rsrc_t r, f4 v, int voff, int soff) {
  if constexpr (!BF) {
    bst128(r, v, voff, soff);
  } else {
    const unsigned lo = f_to_bf(v[0]) | ((unsigned)f_to_bf(v[1]) << 16);
    const unsigned hi = f_to_bf(v[2]) | ((unsigned)f_to_bf(v[3]) << 16);
    bst64(r, uint2{lo, hi}, voff, soff);
  }
}

// A wavefront's 32-point output tile o[vb][pb] (point 16 pb + i, columns 16 vb + 4 j .. + 3)
// stored through its LDS rows sb (32 rows of D values, kStageBytes<BF, D>) so that every lane
// stores 16 contiguous bytes and each store instruction writes whole D-value row segments.
// The rows' 16-byte chunks are XOR-swizzled by row, so that neither the chunk writes (8 lanes
// a pass, eight rows of one chunk column) nor the row reads (8 lanes a pass, whole rows) meet
// an LDS bank twice. bf16 lanes hold 8 bytes of a chunk: lanes of rows j and j ^ 1 first trade
// halves (one lane swap per dword: odd rows of the first operand with even rows of the
// second), pairing blocks (vb, vb + 1) of one point or, with one 16-wide block, the two point
// blocks, so that each writes a whole chunk. The first point of the tile is row 0 at byte
// offset tb * rsb of the resource. Orders sb against the wavefront's earlier and later LDS use.
template <bool BF, int D>
constexpr int kStageBytes = 32 * D * (BF ? 2 : 4);
// The fused bf16 pass B of the tied path stores dx and dfx this way (1) or straight from the
// MFMA tiles, 8 bytes per lane (0).
#ifndef FS_BWDB_STAGE
#define FS_BWDB_STAGE 1
#endif
template <bool BF, int D>
__device__ __forceinline__ void store_tile_staged(char* sb, const f4 (&o)[D / 16][2],
                                                  __amdgpu_buffer_rsrc_t ro, int rsb, int tb, int lane) {
  constexpr int VB = D / 16, kSeg = D * (BF ? 2 : 4), kChunks = kSeg / 16;
  constexpr int kSwz = kChunks < 8 ? kChunks : 8, kSwzShift = kSwz == 2 ? 2 : kSwz == 4 ? 1 : 0;
  static_assert(kChunks % 2 == 0, "a 32-row tile spreads evenly over 64 lanes");
  auto at = [](int row, int chunk) { return row * kSeg + 16 * (chunk ^ ((row >> kSwzShift) & (kSwz - 1))); };
  const int i = lane & 15, j = lane >> 4;
  wave_lds_sync();
  if constexpr (BF) {
    constexpr int NQ = VB == 1 ? 1 : 2 * (VB / 2);
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int pb = VB == 1 ? 0 : q / (VB / 2), m = VB == 1 ? 0 : q % (VB / 2);
      const f4& a = VB == 1 ? o[0][0] : o[2 * m][pb];
      const f4& b = VB == 1 ? o[0][1] : o[2 * m + 1][pb];
      const auto sx = __builtin_amdgcn_permlane16_swap(bf_pair(a[0], a[1]), bf_pair(b[0], b[1]), false, false);
      const auto sy = __builtin_amdgcn_permlane16_swap(bf_pair(a[2], a[3]), bf_pair(b[2], b[3]), false, false);
      const int row = VB == 1 ? 16 * (j & 1) + i : 16 * pb + i;
      const int chunk = 2 * (VB == 1 ? 0 : 2 * m + (j & 1)) + (j >> 1);
      *reinterpret_cast<uint4*>(sb + at(row, chunk)) = uint4{sx[0], sy[0], sx[1], sy[1]};
    }
  } else {
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int vb = 0; vb < VB; ++vb) *reinterpret_cast<f4*>(sb + at(16 * pb + i, 4 * vb + j)) = o[vb][pb];
  }
  wave_lds_sync();
  // 32 rows of kChunks 16-byte chunks: kChunks / 2 chunks per lane
#pragma unroll
  for (int q = 0; q < kChunks / 2; ++q) {
    const int f = 64 * q + lane, row = f / kChunks, c16 = f % kChunks;
    const f4 v = *reinterpret_cast<const f4*>(sb + at(row, c16));
    bst128(ro, v, row * rsb + 16 * c16, tb * rsb);
  }
  wave_lds_sync();
}

// The base-2 normalisers of a 32-point tile for the T layout (lane 16 j + i: point 16 pb + i of
// block pb) from one load: lane 16 j + i reads point 16 (j % 2) + i (lse_load, issued with the
// tile's other loads), and at use a lane swap of rows j and j ^ 1 gives every lane both
// blocks' values (lse_pair). Points at or past npts get kMasked.
__device__ __forceinline__ float lse_load(__amdgpu_buffer_rsrc_t rl, int tb, int i, int j) {
  return bld32(rl, 4 * (16 * (j & 1) + i), 4 * tb);
}
__device__ __forceinline__ void lse_pair(float (&l2)[2], float raw, int tb, int npts, int i) {
  const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(raw), __float_as_uint(raw), false, false);
  l2[0] = tb + i < npts ? __uint_as_float(s[0]) : kMasked;
  l2[1] = tb + 16 + i < npts ? __uint_as_float(s[1]) : kMasked;
}

// Four values of one row in the storage dtype (the counterpart of bst_row4), as fp32.
template <bool BF>
__device__ __forceinline__ f4 bld_row4(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  if constexpr (!BF) {
    return bld128(r, voff, soff);
  } else {
    const uint2 v = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
    return f4{bf_to_f(v.x & 0xFFFFu), bf_to_f(v.x >> 16), bf_to_f(v.y & 0xFFFFu), bf_to_f(v.y >> 16)};
  }
}

// Row operand from a buffer: rowoff = byte offset of the lane's row (point 16 pb + i of the
// tile, scalar part in soff). Same register layout as load_row.
template <bool BF, int D>
__device__ __forceinline__ void load_row_buf(RowOp<BF, D>& o, __amdgpu_buffer_rsrc_t r,
                                             int rowoff, int soff, int j) {
  if constexpr (!BF) {
    constexpr int K = D / 4;
#pragma unroll
    for (int q = 0; q < K / 4; ++q) {
      const f4 t = bld128(r, rowoff + (j * K + 4 * q) * 4, soff);
      o.v[4 * q + 0] = t[0];
      o.v[4 * q + 1] = t[1];
      o.v[4 * q + 2] = t[2];
      o.v[4 * q + 3] = t[3];
    }
  } else {
    constexpr int K = (D + 31) / 32;
#pragma unroll
    for (int kk = 0; kk < K; ++kk) {
      uint4 t = bld128u(r, rowoff + kbase_bf<D>(j, kk) * 2, soff);
      if (D == 16 && j >= 2) t = uint4{0u, 0u, 0u, 0u};
      o.v[kk] = __builtin_bit_cast(bf8, t);
    }
  }
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

// Slot limit of the guarded slot reads: the real slot count G when the tiling pads the slots,
// else kNoPad (every slot real). G is a multiple of 16 and slot groups start at multiples of
// 16, so every 16-slot block is wholly real or wholly padding: a padding block reads the last
// real block (slots glim - 16 ..) scaled by zero. The block choice is wave-uniform and the
// guard arithmetic, never a branch: with a branch around the loads (or between guarded and
// plain reads) the compiler waited on each load separately, or moved the buffer descriptors
// of the streaming loops to vector registers; with per-lane clamped indices it spent more
// registers on addresses.
constexpr int kNoPad = 0x7fffffff;

// First slot to read for the 16-slot block starting at gblk (itself if real, else the last
// real block), and whether it is real.
__device__ __forceinline__ int slot_block(int gblk, int glim, bool& real) {
  real = gblk < glim;
  return real ? gblk : glim - 16;
}

// v where the slot is real, else pad (v finite), as one multiply-add.
__device__ __forceinline__ float slot_mask(bool real, float v, float pad) {
  return fmaf(v, real ? 1.f : 0.f, real ? 0.f : pad);
}

// TRANSPOSED = true: element (g, k) read from src[k * ld + g] (W_s (D,G)); else
// src[g * ld + k] - cen[k] (cen nullable: a per-column shift removed before rounding).
// Slots g >= glim (padding) are zero.
template <bool BF, int D, int GB, bool TRANSPOSED, bool SPLIT>
__device__ __forceinline__ void load_slotop(SlotOp<BF, D, GB>& o, const float* src, int ld,
                                            int g0, int glim, float sc, int i, int j,
                                            const float* cen = nullptr) {
  auto M = [&](int g, int k, float s) -> float {
    if (TRANSPOSED) return s * src[(int64_t)k * ld + g];
    return s * (src[(int64_t)g * ld + k] - (cen != nullptr ? cen[k] : 0.f));
  };
#pragma unroll
  for (int gb = 0; gb < GB; ++gb) {
    bool real;
    const int gc = slot_block(g0 + 16 * gb, glim, real) + i;
    const float s = real ? sc : 0.f;
    if constexpr (!BF) {
#pragma unroll
      for (int kk = 0; kk < D / 4; ++kk) o.v[gb][kk] = M(gc, kcol_f<D>(j, kk), s);
    } else {
#pragma unroll
      for (int kk = 0; kk < SlotOp<true, D, GB>::K; ++kk) {
        bf8 hi, lo;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int k = kcol_bf<D>(j, kk, e);
          float val = 0.f;
          if (k >= 0) val = M(gc, k, s);
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

// TRANSPOSED = true: M(g, c) = src[c * ld + g] * sc, else src[g * ld + c] * sc; zero for
// the padding slots g >= glim.
template <bool BF, int GB, int CB, bool TRANSPOSED>
__device__ __forceinline__ void load_gop(GOp<BF, GB, CB>& o, const float* src, int ld, int g0,
                                         int glim, float sc, int i, int j) {
  // element (16-slot block gblk, slot offset go within it, column c); padding blocks read the
  // last real block scaled by zero (see kNoPad)
  auto M = [&](int gblk, int go, int c) -> float {
    bool real;
    const int gc = slot_block(gblk, glim, real) + go;
    const float s = real ? sc : 0.f;
    return s * (TRANSPOSED ? src[(int64_t)c * ld + gc] : src[(int64_t)gc * ld + c]);
  };
  if constexpr (!BF) {
#pragma unroll
    for (int gb = 0; gb < GB; ++gb)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) o.v[gb][r][cb] = M(g0 + 16 * gb, 4 * j + r, 16 * cb + i);
  } else {
#pragma unroll
    for (int q = 0; q < GB / 2; ++q)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        bf8 t;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          t[e] = (__bf16)M(g0 + 32 * q + 16 * (e / 4), 4 * j + (e % 4), 16 * cb + i);
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
    for (int q = 0; q < GB / 2; ++q) acc = mfma_bf16(o.v[q][cb], to_bf8(t[2 * q][pb], t[2 * q + 1][pb]), acc);
  }
  return acc;
}

// A T-layout tile as the B operand of contractions over slots, converted once and reused for
// every output column block: fp32 keeps the tile itself; bf16 packs slot pairs q of column
// block pb into bf8 (element e = row 16 (e / 4) + 4 j + (e % 4) of the pair).
template <bool BF, int GB, int PB>
struct TileB;
template <int GB, int PB>
struct TileB<false, GB, PB> {
  const f4 (*t)[PB];
};
template <int GB, int PB>
struct TileB<true, GB, PB> {
  bf8 v[GB / 2][PB];
};
template <bool BF, int GB, int PB>
__device__ __forceinline__ TileB<BF, GB, PB> tile_b(const f4 (*t)[PB]) {
  TileB<BF, GB, PB> o;
  if constexpr (!BF) {
    o.t = t;
  } else {
#pragma unroll
    for (int q = 0; q < GB / 2; ++q)
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) o.v[q][pb] = to_bf8(t[2 * q][pb], t[2 * q + 1][pb]);
  }
  return o;
}
// out[cb] (+)= M^T-contraction with a converted tile (same result as mm_gop_tile).
template <bool BF, int GB, int CB, int PB>
__device__ __forceinline__ f4 mm_gop_b(const GOp<BF, GB, CB>& o, int cb, const TileB<BF, GB, PB>& tb,
                                       int pb, f4 acc) {
  if constexpr (!BF) {
#pragma unroll
    for (int gb = 0; gb < GB; ++gb)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc = mfma_f32(o.v[gb][r][cb], tb.t[gb][pb][r], acc);
  } else {
#pragma unroll
    for (int q = 0; q < GB / 2; ++q) acc = mfma_bf16(o.v[q][cb], tb.v[q][pb], acc);
  }
  return acc;
}

// Columns 0..16 DB-1 of a point-major matrix as the MFMA k operand of a contraction over the
// TP = 16 PB points of a pass-B tile (dW += X^T da): lane (j, i) holds column 16 d + i of
//   fp32: point 16 pb + 4 j + r for MFMA (pb, r);  bf16 (PB = 2): point 16 (e / 4) + 4 j + (e % 4).
// Loaded with the tile it belongs to, so the loads are in flight while earlier tiles compute.
template <bool BF, int DB, int PB>
struct KGather;
template <int DB, int PB>
struct KGather<false, DB, PB> {
  float v[PB][4][DB];
};
template <int DB, int PB>
struct KGather<true, DB, PB> {
  bf8 v[DB];
};
template <bool BF, int DB, int PB>
__device__ __forceinline__ void gather_k(KGather<BF, DB, PB>& g, __amdgpu_buffer_rsrc_t r,
                                         int rsb, int tb, int i, int j) {
  if constexpr (!BF) {
#pragma unroll
    for (int pb = 0; pb < PB; ++pb)
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int d = 0; d < DB; ++d)
          g.v[pb][q][d] = bld32(r, 4 * j * rsb + (16 * d + i) * 4, (tb + 16 * pb + q) * rsb);
  } else {
    static_assert(PB == 2, "bf16 pass-B tiles hold 32 points");
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        g.v[d][e] = __builtin_bit_cast(
            __bf16, bld16(r, 4 * j * rsb + (16 * d + i) * 2, (tb + 16 * (e / 4) + (e % 4)) * rsb));
  }
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

// gather_points from a buffer: lane (j, i) reads column 16 cb + i of points
// tb + 16 pb + 4 j + r (fp32) or tb + 16 (e / 4) + 4 j + (e % 4) (bf16); rsb = row stride in
// bytes, tbo = tb * rsb (wave-uniform).
template <bool BF, int CB>
__device__ __forceinline__ void gather_points_buf(PtGather<BF, CB>& g, __amdgpu_buffer_rsrc_t r,
                                                  int rsb, int tbo, int i, int j) {
  if constexpr (!BF) {
    const int lo = 4 * j * rsb + 4 * i;
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
          g.v[pb][rr][cb] = bld32(r, lo + 64 * cb, tbo + (16 * pb + rr) * rsb);
  } else {
    const int lo = 4 * j * rsb + 2 * i;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      bf8 bt;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        bt[e] = __builtin_bit_cast(__bf16, bld16(r, lo + 32 * cb, tbo + (16 * (e / 4) + (e % 4)) * rsb));
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
    for (int gb = 0; gb < GB; ++gb) at[gb] = to_bf8(w[0][gb], w[1][gb]);
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
  const u32x4* src = reinterpret_cast<const u32x4*>(&o);
#pragma unroll
  for (int q = 0; q < (int)(sizeof(Op) / 16); ++q) reinterpret_cast<u32x4*>(base)[q * 64 + lane] = src[q];
}
template <class Op>
__device__ __forceinline__ void lds_get(Op& o, const uint4* base, int lane) {
  u32x4* dst = reinterpret_cast<u32x4*>(&o);
#pragma unroll
  for (int q = 0; q < (int)(sizeof(Op) / 16); ++q) dst[q] = reinterpret_cast<const u32x4*>(base)[q * 64 + lane];
}
template <class Op>
constexpr int lds_chunks() {
  return (int)(sizeof(Op) / 16) * 64;
}

// ---------------------------------------------------------------------------------------
// Software pipeline over a wavefront's point tiles: the loads of tile t + PF are issued
// before tile t is computed, so PF tiles of global loads are in flight behind the compute.
// The PF + 1 buffers form a ring indexed with compile-time constants (the loop over the
// ring is unrolled), so they stay in registers. Prefetches are unconditional: load() must be
// safe for tiles past the end (the buffer loads return zeros there). A conditional prefetch
// would make the compiler's wait counts cover the path without it, i.e. wait for every load
// in flight before each tile.
// ---------------------------------------------------------------------------------------
template <int PF, class Tile, class Load, class Body>
__device__ __forceinline__ void pipeline(int ntile, Load&& load, Body&& body) {
  constexpr int DEPTH = PF + 1;
  Tile buf[DEPTH];
#pragma unroll
  for (int s = 0; s < PF; ++s) load(buf[s], s);
  for (int t0 = 0; t0 < ntile; t0 += DEPTH) {
#pragma unroll
    for (int u = 0; u < DEPTH; ++u) {
      const int t = t0 + u;
      if (t >= ntile) break;
      load(buf[(u + PF) % DEPTH], t + PF);
      body(buf[u], t);
    }
  }
}

// Prefetch distance (in tiles) of each streaming pass.
#ifndef FS_PF_SLICE
#define FS_PF_SLICE 1
#endif
#ifndef FS_PF_DESLICE
#define FS_PF_DESLICE 2
#endif
#ifndef FS_PF_BWD_A
#define FS_PF_BWD_A 2
#endif
#ifndef FS_PF_BWD_B
#define FS_PF_BWD_B 1
#endif
// Slot groups per tile from which the passes do not prefetch (their register budget is
// taken by the per-slot-group state).
#ifndef FS_NS_NOPF
#define FS_NS_NOPF 8
#endif
// Minimum wavefronts per SIMD each pass is compiled for (1: no register cap). Pass A at 2
// keeps its accumulators in ordinary VGPRs within 256 registers, so two wavefronts share a
// SIMD instead of one (the bf16 64-slot form needed 220 VGPRs plus 56 accumulation
// registers otherwise).
#ifndef FS_WPE_SLICE
#define FS_WPE_SLICE 1
#endif
// The deslice's target applies up to head width 32 (64 would spill at three).
#ifndef FS_WPE_DESLICE
#define FS_WPE_DESLICE 1
#endif
#ifndef FS_WPE_BWD_A
#define FS_WPE_BWD_A 2
#endif
// Pass B: bf16 (FS_WPE_BWD_B) stays at one (at two it would spill 60 registers and its
// 79 KB of LDS allow one workgroup per compute unit anyway); fp32 and the slot-blocked
// parameter pass (PM) at two fit in 256 VGPRs without spilling, the parameter pass then
// running two workgroups per compute unit (13% faster at G = 1024).
#ifndef FS_WPE_BWD_B
#define FS_WPE_BWD_B 1
#endif
#ifndef FS_WPE_BWD_B_F32
#define FS_WPE_BWD_B_F32 2
#endif
#ifndef FS_WPE_BWD_PM
#define FS_WPE_BWD_PM 2
#endif
// The one-kernel untied / LinearNO pass B with at most 32 slots fits two wavefronts per SIMD
// in 256 VGPRs without spilling (one otherwise: 336 registers in fp32, 412 in bf16).
#ifndef FS_WPE_BWD_B2_G32
#define FS_WPE_BWD_B2_G32 2
#endif

// Workgroup -> (chunk, slot block, b*H+h) over a 1-D grid of chunks * nblk * BH workgroups,
// chunks of one (head, slot block) consecutive. With the chunk count a multiple of 8 the
// H * nblk workgroups that read the same point rows (each its own D-element segment of every
// (B, N, H, D) row) get numbers equal mod 8, so the dispatcher, which deals workgroups
// round-robin to the 8 XCDs, places them on one XCD and its L2. On grids larger than
// FS_GROUP_GRID workgroups, which run in several waves, they are also numbered 8 apart
// (workgroup L is the (L / 8 mod H nblk)-th unit of (sample, chunk) group
// (L / 8 / (H nblk)) * 8 + L mod 8), so that they are dispatched together.
#ifndef FS_GROUP_GRID
#define FS_GROUP_GRID 4096
#endif
struct BlockPos {
  int chunk, blk, bh;
};
__device__ __forceinline__ BlockPos block_pos(const PassArgs& a) {
  BlockPos p;
  const int L = blockIdx.x;
  const int per = a.nblk * a.H;
  if ((int)gridDim.x > FS_GROUP_GRID && per > 1 && ((gridDim.x / per) & 7) == 0) {
    const int k = L >> 3;
    const int rg = (k / per) * 8 + (L & 7);
    const int u = k % per;
    p.chunk = rg % a.chunks;
    p.blk = u % a.nblk;
    p.bh = (rg / a.chunks) * a.H + u / a.nblk;
    return p;
  }
  p.chunk = L % a.chunks;
  const int r = L / a.chunks;
  p.blk = r % a.nblk;
  p.bh = r / a.nblk;
  return p;
}

struct HeadCtx {
  int chunk, blk;
  int bh, b, h, g0;
  float sc;  // log2(e) / tau_h
  const float* W;
  const float* bias;
  int64_t off;  // element offset of point 0 of this (b, h) in the (B, N, H, D) layout
};

template <int D>
__device__ __forceinline__ HeadCtx head_ctx(const PassArgs& a, int ws, int GS) {
  HeadCtx c;
  const BlockPos bp = block_pos(a);
  c.chunk = bp.chunk;
  c.blk = bp.blk;
  c.bh = bp.bh;
  c.b = c.bh / a.H;
  c.h = c.bh % a.H;
  // nblk > 1 only with one slot group per tile; ws is the wave's slot-group index (the same in
  // every lane: it comes from the wave number)
  c.g0 = (bp.blk + __builtin_amdgcn_readfirstlane(ws)) * GS;
  c.sc = kLog2e / a.tau[c.h];
  c.W = a.Ws + (a.ws_per_head ? (int64_t)c.h * D * a.G : 0);
  c.bias = a.bias + (a.ws_per_head ? (int64_t)c.h * a.G : 0);
  c.off = ((int64_t)c.b * a.N * a.H + c.h) * D;
  return c;
}

// Slot limit for the operand loaders (see kNoPad).
__device__ __forceinline__ int slot_lim(const PassArgs& a) { return a.padded ? a.G : kNoPad; }

// Scaled base-2 bias of slot gblk + go of the 16-slot block gblk (kMaskedSlot for padding).
__device__ __forceinline__ float slot_bias(const HeadCtx& c, const PassArgs& a, int gblk, int go) {
  bool real;
  const int gc = slot_block(gblk, slot_lim(a), real) + go;
  return slot_mask(real, c.sc * c.bias[gc], kMaskedSlot);
}
// The same for any slot g (per-lane block choice; for one-time set-up loops).
__device__ __forceinline__ float slot_bias_at(const HeadCtx& c, const PassArgs& a, int g) {
  return slot_bias(c, a, g & ~15, g & 15);
}

// =======================================================================================
// Dispatch over the compile-time tiling
// =======================================================================================
// Supported (GS, NS, NP, PB) tilings; pick_cfg in fs_api.cpp chooses among exactly these.
// PB = 1 (16-point tiles) exists for the fp32 backward pass B only.
#define FS_TILINGS(X, BF, D)                                                              \
  X(BF, D, 16, 1, 4, 2) X(BF, D, 32, 1, 4, 2) X(BF, D, 64, 1, 4, 2) X(BF, D, 64, 2, 2, 2) \
  X(BF, D, 64, 4, 1, 2) X(BF, D, 64, 8, 1, 2) X(BF, D, 64, 16, 1, 2)                     \
  X(BF, D, 16, 1, 4, 1) X(BF, D, 32, 1, 4, 1) X(BF, D, 64, 1, 4, 1)

// Runner<BF, D, GS, NS, NP, PB>::run launches one pass's kernel for one tiling.
template <int PASS, template <bool, int, int, int, int, int> class Runner, bool BF, int D>
hipError_t run_tiled(const PassCfg& cfg, int BH, const PassArgs& a, hipStream_t st) {
#define FS_CASE(BF_, D_, GS_, NS_, NP_, PB_)                                             \
  if (cfg.GS == GS_ && cfg.NS == NS_ && cfg.NP == NP_ && cfg.PB == PB_) {                \
    if constexpr (!(BF_ && GS_ < 32) && (PB_ == 2 || (!BF_ && PASS == PASS_BWD_B)))      \
      return Runner<BF_, D_, GS_, NS_, NP_, PB_>::run(cfg, BH, a, st);                   \
  }
  FS_TILINGS(FS_CASE, BF, D)
#undef FS_CASE
  return hipErrorInvalidConfiguration;
}

template <int PASS, template <bool, int, int, int, int, int> class Runner>
hipError_t run_pass_tilings(const Geom& g, const PassArgs& a, hipStream_t st) {
  const PassCfg cfg = pick_cfg(g, (Pass)PASS);
  const int BH = g.BH();
  if (g.bf16) {
    if (g.D == 16) return run_tiled<PASS, Runner, true, 16>(cfg, BH, a, st);
    if (g.D == 32) return run_tiled<PASS, Runner, true, 32>(cfg, BH, a, st);
    if (g.D == 64) return run_tiled<PASS, Runner, true, 64>(cfg, BH, a, st);
  } else {
    if (g.D == 16) return run_tiled<PASS, Runner, false, 16>(cfg, BH, a, st);
    if (g.D == 32) return run_tiled<PASS, Runner, false, 32>(cfg, BH, a, st);
    if (g.D == 64) return run_tiled<PASS, Runner, false, 64>(cfg, BH, a, st);
  }
  return hipErrorInvalidConfiguration;
}

}  // namespace
}  // namespace fs
