// Token-sized kernels of the path (fp32): fixed-order reductions of the per-workgroup
// partials written by the streaming passes, the G x G token mix and its backward, and the
// token gradients dU = dz / (s + eps), ds = -sum_v dz z / (s + eps).
// Their work is O(B H G V) or O(B H G^2 V), tiny next to the O(B N H G D) streaming passes;
// they are written to keep every thread busy so that they do not add latency to a step.

#include <hip/hip_runtime.h>

#include <algorithm>

#include "fs_internal.h"

namespace fs {
namespace {

constexpr int kThreads = 256;
constexpr int kRedThreads = 1024;  // column reductions: many row groups in flight per column
constexpr int kCols = 64;          // columns per workgroup (chunk reductions)
constexpr int kRowGroups = kRedThreads / kCols;
constexpr int kColsWide = 16;      // long reductions (over samples, heads and chunks)
constexpr int kRowGroupsWide = kRedThreads / kColsWide;
constexpr int kAttnThreads = 1024;

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) v += __shfl_xor(v, off);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

// ---------------------------------------------------------------------------------------
// Fixed-order column sums. Thread (row group rg, column cg) sums rows rg, rg + 4, ... of its
// column; the four row-group sums are then added in the order rg = 0, 1, 2, 3. The result is
// independent of scheduling, so repeated runs are bitwise identical.
// ---------------------------------------------------------------------------------------
struct RowMap {
  // row r of output o lives at in + ((o_outer * stride_o + r_hi * stride_hi + r_lo) * len);
  // used to walk (chunk) rows of one (b, h), or (b, chunk) rows of one head.
  int64_t base;
  int rows;
  int lo;        // rows per inner run (chunks)
  int64_t hi_stride;  // distance in rows between inner runs
};

// Sum of rows rg, rg + 4, ... of column c, in increasing row order. Loads are issued eight at
// a time ahead of the adds so that the row walk is not a chain of dependent memory latencies.
template <int RG = kRowGroups>
__device__ __forceinline__ float colsum(const float* in, int64_t len, const RowMap& m, int64_t c,
                                        int rg) {
  constexpr int U = 8;
  float acc = 0.f;
  for (int r0 = rg; r0 < m.rows; r0 += U * RG) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = r0 + u * RG;
      v[u] = 0.f;
      if (r < m.rows) {
        const int64_t row = m.base + (int64_t)(r / m.lo) * m.hi_stride + (r % m.lo);
        v[u] = in[row * len + c];
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc += v[u];
  }
  return acc;
}

template <int RG = kRowGroups, int NC = kCols>
__device__ __forceinline__ float combine_groups(float v, float (*red)[NC], int rg, int cg) {
  red[rg][cg] = v;
  __syncthreads();
  float out = 0.f;
  if (rg == 0) {
#pragma unroll
    for (int q = 0; q < RG; ++q) out += red[q][cg];
  }
  return out;
}

// z = (sum_chunks U) / (sum_chunks s + eps) and s. grid (ceil(G V / 64), BH).
__global__ __launch_bounds__(kRedThreads) void k_reduce_tokens(const float* partU,
                                                            const float* partS, float* z,
                                                            float* s, int chunks, int G, int V,
                                                            float eps) {
  __shared__ float red[kRowGroups][kCols];
  __shared__ float sred[kRowGroups][kCols];
  const int bh = blockIdx.y;
  const int cg = threadIdx.x % kCols, rg = threadIdx.x / kCols;
  const int64_t len = (int64_t)G * V;
  const int64_t c = (int64_t)blockIdx.x * kCols + cg;
  const RowMap m{(int64_t)bh * chunks, chunks, chunks, 0};
  // slot sums for the slots this workgroup's columns touch (at most kCols / V + 1 <= 5)
  const int g_lo = (int)(((int64_t)blockIdx.x * kCols) / V);
  const int g_hi = (int)(min((int64_t)(blockIdx.x + 1) * kCols, len) - 1) / V;
  const int ns = g_hi - g_lo + 1;
  float sv = 0.f;
  if (cg < ns) sv = colsum(partS, G, m, g_lo + cg, rg);
  sred[rg][cg] = sv;
  const float u = c < len ? colsum(partU, len, m, c, rg) : 0.f;
  const float tot = combine_groups(u, red, rg, cg);   // contains the barrier for sred too
  if (rg == 0) {
    if (cg < ns) {
      float st = 0.f;
#pragma unroll
      for (int q = 0; q < kRowGroups; ++q) st += sred[q][cg];
      sred[0][cg] = st;
    }
  }
  __syncthreads();
  if (rg == 0 && c < len) {
    const int g = (int)(c / V);
    const float sg = sred[0][g - g_lo];
    z[(int64_t)bh * len + c] = tot / (sg + eps);
    if (c % V == 0) s[(int64_t)bh * G + g] = sg;
  }
}

// out[bh][c] = sum over chunks of part[bh][chunk][c]. grid (ceil(len / 64), BH).
__global__ __launch_bounds__(kRedThreads) void k_reduce_rows(const float* part, float* out,
                                                          int chunks, int64_t len) {
  __shared__ float red[kRowGroups][kCols];
  const int bh = blockIdx.y;
  const int cg = threadIdx.x % kCols, rg = threadIdx.x / kCols;
  const int64_t c = (int64_t)blockIdx.x * kCols + cg;
  const RowMap m{(int64_t)bh * chunks, chunks, chunks, 0};
  const float v = c < len ? colsum(part, len, m, c, rg) : 0.f;
  const float tot = combine_groups(v, red, rg, cg);
  if (rg == 0 && c < len) out[(int64_t)bh * len + c] = tot;
}

// Mix-parameter gradient from per-(b, h) partials [BH][len]: summed over (b, h), or over b
// per head (per_head); column block cb of output head hh.
__device__ __forceinline__ void reduce_mixparams_block(const float* partM, float* dmix, int B,
                                                       int H, int64_t len, int per_head, int cb,
                                                       int hh, float (*red)[kColsWide]) {
  const int cg = threadIdx.x % kColsWide, rg = threadIdx.x / kColsWide;
  const int64_t c = (int64_t)cb * kColsWide + cg;
  RowMap m;
  if (per_head)
    m = RowMap{hh, B, 1, H};
  else
    m = RowMap{0, B * H, B * H, 0};
  const float v = c < len ? colsum<kRowGroupsWide>(partM, len, m, c, rg) : 0.f;
  const float tot = combine_groups<kRowGroupsWide, kColsWide>(v, red, rg, cg);
  if (rg == 0 && c < len) dmix[(per_head ? (int64_t)hh * len : 0) + c] = tot;
}

__global__ __launch_bounds__(kRedThreads) void k_reduce_mixparams(const float* partM, float* dmix,
                                                               int B, int H, int64_t len,
                                                               int per_head) {
  __shared__ float red[kRowGroupsWide][kColsWide];
  reduce_mixparams_block(partM, dmix, B, H, len, per_head, blockIdx.x, blockIdx.y, red);
}

// Parameter gradients from the backward-pass-B partials [BH][chunks][D G + G + 2] (the last
// two floats of each partial hold one fp64 dtau partial), and optionally the mix-parameter
// gradient from its per-(b, h) partials, in one launch.
// grid.x = [column blocks of dW_s and dbias] [one dtau block] [column blocks of dmix];
// blockIdx.y is the head for per-head outputs (rows: b = 0..B-1, chunk), else 0 with rows
// over every (b, h, chunk); blocks whose segment has fewer heads return at once.
__global__ __launch_bounds__(kRedThreads) void k_reduce_params(
    const float* part, float* dWs, float* dbias, float* dtau, int B, int H, int chunks,
    int nblk, int D, int G, int per_head, const float* partM, float* dmix, int64_t mix_len,
    int mix_per_head) {
  __shared__ float red[kRowGroupsWide][kColsWide];
  const int64_t len = (int64_t)D * G + G + 2LL * nblk;
  const int64_t ncol = (int64_t)D * G + G;
  const int nbp = (int)((ncol + kColsWide - 1) / kColsWide);
  const int hh = blockIdx.y;
  if ((int)blockIdx.x > nbp) {
    if (dmix != nullptr && (mix_per_head || hh == 0))
      reduce_mixparams_block(partM, dmix, B, H, mix_len, mix_per_head, blockIdx.x - nbp - 1, hh,
                             red);
    return;
  }
  if (!per_head && hh > 0) return;
  if ((int)blockIdx.x == nbp) {
    // dtau: one wavefront per head; lane l sums the fp64 partials l, l + 64, ... of the
    // head's (b, chunk, slot block) entries in order, then a butterfly over the 64 lanes
    // (fixed pairing)
    if (hh == 0) {
      const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
      const int rows = B * chunks * nblk;
      for (int h = wave; h < H; h += nw) {
        double t = 0.0;
        for (int r = lane; r < rows; r += 64) {
          const int b = r / (chunks * nblk), q = (r / nblk) % chunks, k = r % nblk;
          t += *reinterpret_cast<const double*>(part + ((int64_t)(b * H + h) * chunks + q) * len +
                                                ncol + 2 * k);
        }
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) t += __shfl_xor(t, off);
        if (lane == 0) dtau[h] = (float)t;
      }
    }
    return;
  }
  const int cg = threadIdx.x % kColsWide, rg = threadIdx.x / kColsWide;
  const int64_t c = (int64_t)blockIdx.x * kColsWide + cg;
  RowMap m;
  if (per_head)  // rows (b, chunk) of head hh: run of `chunks` rows every H * chunks rows
    m = RowMap{(int64_t)hh * chunks, B * chunks, chunks, (int64_t)H * chunks};
  else           // all (b, h, chunk) rows in order
    m = RowMap{0, B * H * chunks, B * H * chunks, 0};
  const float v = c < ncol ? colsum<kRowGroupsWide>(part, len, m, c, rg) : 0.f;
  const float tot = combine_groups<kRowGroupsWide, kColsWide>(v, red, rg, cg);
  if (rg == 0 && c < ncol) {
    if (c < (int64_t)D * G)
      dWs[(per_head ? (int64_t)hh * D * G : 0) + c] = tot;
    else
      dbias[(per_head ? (int64_t)hh * G : 0) + (c - (int64_t)D * G)] = tot;
  }
}

// ---------------------------------------------------------------------------------------
// Token mix: identity, fixed G x G matrix, per-token channel map (one thread per output).
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_mix_linear(const float* z, float* zmix,
                                                         const float* A, const float* Wc,
                                                         int kind, int a_per_head, int H, int G,
                                                         int V) {
  const int bh = blockIdx.y;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= G * V) return;
  const int g = idx / V, v = idx % V;
  const float* zb = z + (int64_t)bh * G * V;
  float acc = 0.f;
  if (kind == 0) {
    acc = zb[idx];
  } else if (kind == 1) {
    const float* Ah = A + (a_per_head ? (int64_t)(bh % H) * G * G : 0) + (int64_t)g * G;
    for (int k = 0; k < G; ++k) acc += Ah[k] * zb[(int64_t)k * V + v];
  } else {
    for (int k = 0; k < V; ++k) acc += zb[(int64_t)g * V + k] * Wc[(int64_t)k * V + v];
  }
  zmix[(int64_t)bh * G * V + idx] = acc;
}

// dz = Mix^T(dzmix) for the linear kinds (one thread per output).
__global__ __launch_bounds__(kThreads) void k_mix_dz_linear(const float* dzm, float* dz,
                                                            const float* A, const float* Wc,
                                                            int kind, int a_per_head, int H,
                                                            int G, int V) {
  const int bh = blockIdx.y;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= G * V) return;
  const int g = idx / V, v = idx % V;
  const float* db = dzm + (int64_t)bh * G * V;
  float acc = 0.f;
  if (kind == 0) {
    acc = db[idx];
  } else if (kind == 1) {
    const float* Ah = A + (a_per_head ? (int64_t)(bh % H) * G * G : 0);
    for (int k = 0; k < G; ++k) acc += Ah[(int64_t)k * G + g] * db[(int64_t)k * V + v];
  } else {
    for (int k = 0; k < V; ++k) acc += db[(int64_t)g * V + k] * Wc[(int64_t)v * V + k];
  }
  dz[(int64_t)bh * G * V + idx] = acc;
}

// Per-(b, h) mix-parameter partial for the linear kinds (one thread per output):
// LINEAR_G: dA_bh[g][k] = sum_v dzmix[g][v] z[k][v]; LINEAR_C: dWc_bh[c][v] = sum_g z[g][c] dzmix[g][v].
__global__ __launch_bounds__(kThreads) void k_mix_param_linear(const float* z, const float* dzm,
                                                               float* partM, int kind, int G,
                                                               int V) {
  const int bh = blockIdx.y;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  const float* zb = z + (int64_t)bh * G * V;
  const float* db = dzm + (int64_t)bh * G * V;
  if (kind == 1) {
    if (idx >= G * G) return;
    const int g = idx / G, k = idx % G;
    float acc = 0.f;
    for (int v = 0; v < V; ++v) acc += db[(int64_t)g * V + v] * zb[(int64_t)k * V + v];
    partM[(int64_t)bh * G * G + idx] = acc;
  } else {
    if (idx >= V * V) return;
    const int cc = idx / V, v = idx % V;
    float acc = 0.f;
    for (int g = 0; g < G; ++g) acc += zb[(int64_t)g * V + cc] * db[(int64_t)g * V + v];
    partM[(int64_t)bh * V * V + idx] = acc;
  }
}

// Token gradients and the shifts the backward pass B uses, one workgroup per (b, h):
// dU = dz / (s + eps), ds = -sum_v dz z / (s + eps), and the mass-weighted slot means
// cen = [sum_g m_g zmix[g][:], sum_g m_g dU[g][:], sum_g m_g ds[g]] with m_g = s_g / sum s.
__device__ void token_grads(const float* zb, const float* sb, const float* zmb, const float* dzb,
                            float* dUb, float* dsb, float* cenb, int G, int V, float eps) {
  for (int idx = threadIdx.x; idx < G * V; idx += blockDim.x) {
    const int g = idx / V;
    dUb[idx] = dzb[idx] / (sb[g] + eps);
  }
  for (int g = threadIdx.x; g < G; g += blockDim.x) {
    float acc = 0.f;
    for (int v = 0; v < V; ++v) acc += dzb[(int64_t)g * V + v] * zb[(int64_t)g * V + v];
    dsb[g] = -acc / (sb[g] + eps);
  }
  __syncthreads();
  __shared__ float tot_s;
  if (threadIdx.x < 64) {
    float t = 0.f;
    for (int g = threadIdx.x; g < G; g += 64) t += sb[g];
    t = wave_sum(t);
    if (threadIdx.x == 0) tot_s = t;
  }
  __syncthreads();
  const float inv = tot_s > 0.f ? 1.0f / tot_s : 0.f;
  for (int c = threadIdx.x; c < 2 * V + 1; c += blockDim.x) {
    float acc = 0.f;
    if (c < V) {
      for (int g = 0; g < G; ++g) acc += sb[g] * zmb[(int64_t)g * V + c];
    } else if (c < 2 * V) {
      for (int g = 0; g < G; ++g) acc += sb[g] * dUb[(int64_t)g * V + (c - V)];
    } else {
      for (int g = 0; g < G; ++g) acc += sb[g] * dsb[g];
    }
    cenb[c] = acc * inv;
  }
}

__global__ __launch_bounds__(kThreads) void k_token_grads(const float* z, const float* s,
                                                          const float* zmix, const float* dz,
                                                          float* dU, float* ds, float* cen,
                                                          int G, int V, float eps) {
  const int bh = blockIdx.x;
  const int64_t o = (int64_t)bh * G * V;
  token_grads(z + o, s + (int64_t)bh * G, zmix + o, dz + o, dU + o, ds + (int64_t)bh * G,
              cen + (int64_t)bh * (2 * V + 1), G, V, eps);
}

// ---------------------------------------------------------------------------------------
// Single-head token self-attention among the G tokens of one (b, h): q, k, v = z Wq, z Wk,
// z Wv; P = softmax_row(scale q k^T); zmix = P v. One workgroup per (b, h); q, k, v live in
// LDS; the G x G scores live in LDS up to G = 64, otherwise in the P output buffer.
// ---------------------------------------------------------------------------------------
constexpr int kAttnMaxGV = 8192;
constexpr int kAttnLdsG = 64;

__device__ void attn_project(const float* zb, const float* Wq, const float* Wk, const float* Wv,
                             float* q, float* k, float* v, int G, int V) {
  const int GV = G * V;
  for (int idx = threadIdx.x; idx < 3 * GV; idx += blockDim.x) {
    const int which = idx / GV, r = idx % GV;
    const int g = r / V, c = r % V;
    const float* W = which == 0 ? Wq : (which == 1 ? Wk : Wv);
    float acc = 0.f;
    for (int e = 0; e < V; ++e) acc += zb[(int64_t)g * V + e] * W[e * V + c];
    (which == 0 ? q : (which == 1 ? k : v))[r] = acc;
  }
}

// Row softmax of S (G x G) in place, one wavefront per row; also writes P when S != P.
__device__ void attn_softmax_rows(float* S, float* P, int G) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int g = wave; g < G; g += nw) {
    float m = -INFINITY;
    for (int u = lane; u < G; u += 64) m = fmaxf(m, S[(int64_t)g * G + u]);
    m = wave_max(m);
    float l = 0.f;
    for (int u = lane; u < G; u += 64) {
      const float e = expf(S[(int64_t)g * G + u] - m);
      S[(int64_t)g * G + u] = e;
      l += e;
    }
    l = wave_sum(l);
    const float inv = 1.0f / l;
    for (int u = lane; u < G; u += 64) {
      const float p = S[(int64_t)g * G + u] * inv;
      S[(int64_t)g * G + u] = p;
      if (P != S) P[(int64_t)g * G + u] = p;
    }
  }
}

// All-LDS variant for G V <= 2048, G <= 64, V <= 64: z, the three projections, q, k, v and
// the G x G scores all live in dynamically sized LDS, so no phase waits on global memory.
// Rows are padded by one float (VP = V + 1, GP = G + 1) so that lanes walking different rows
// of the same column hit different LDS banks.
constexpr int kAttnSmallGV = 2048;

inline int attn_small_fwd_floats(int G, int V) {
  const int VP = V + 1, GP = G + 1;
  return 4 * G * VP + 3 * V * VP + G * GP;
}
inline int attn_small_bwd_floats(int G, int V) {
  const int VP = V + 1, GP = G + 1;
  return 11 * G * VP + 3 * V * VP + 2 * G * GP + 3 * G;
}

// Ws: the three projections, [3][V][VP] (padded rows).
__device__ void attn_project_lds(const float* zs, const float* Ws, float* q, float* k, float* v,
                                 int G, int V) {
  const int GV = G * V, VP = V + 1;
  for (int idx = threadIdx.x; idx < 3 * GV; idx += blockDim.x) {
    const int which = idx / GV, r = idx % GV;
    const int g = r / V, c = r % V;
    const float* W = Ws + which * V * VP;
    float acc = 0.f;
#pragma unroll 8
    for (int e = 0; e < V; ++e) acc += zs[g * VP + e] * W[e * VP + c];
    (which == 0 ? q : (which == 1 ? k : v))[g * VP + c] = acc;
  }
}

__global__ __launch_bounds__(kAttnThreads) void k_attn_fwd_small(const float* z, float* zmix,
                                                                 float* P, const float* Wq,
                                                                 const float* Wk,
                                                                 const float* Wv, float scale,
                                                                 int G, int V) {
  extern __shared__ float lds[];
  const int GV = G * V, VV = V * V, VP = V + 1, GP = G + 1;
  float* zs = lds;              // [G][VP]
  float* Ws = zs + G * VP;      // [3][V][VP]
  float* q = Ws + 3 * V * VP;   // [G][VP]
  float* k = q + G * VP;
  float* v = k + G * VP;
  float* S = v + G * VP;        // [G][GP]
  const int bh = blockIdx.x;
  for (int idx = threadIdx.x; idx < GV; idx += blockDim.x)
    zs[(idx / V) * VP + idx % V] = z[(int64_t)bh * GV + idx];
  for (int idx = threadIdx.x; idx < VV; idx += blockDim.x) {
    const int o = (idx / V) * VP + idx % V;
    Ws[o] = Wq[idx];
    Ws[V * VP + o] = Wk[idx];
    Ws[2 * V * VP + o] = Wv[idx];
  }
  __syncthreads();
  attn_project_lds(zs, Ws, q, k, v, G, V);
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * G; idx += blockDim.x) {
    const int g = idx / G, u = idx % G;
    float acc = 0.f;
#pragma unroll 8
    for (int c = 0; c < V; ++c) acc += q[g * VP + c] * k[u * VP + c];
    S[g * GP + u] = scale * acc;
  }
  __syncthreads();
  {  // row softmax, one wavefront per row; P is written unpadded
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    float* Pb = P + (int64_t)bh * G * G;
    for (int g = wave; g < G; g += nw) {
      float m = -INFINITY;
      for (int u = lane; u < G; u += 64) m = fmaxf(m, S[g * GP + u]);
      m = wave_max(m);
      float l = 0.f;
      for (int u = lane; u < G; u += 64) {
        const float e = expf(S[g * GP + u] - m);
        S[g * GP + u] = e;
        l += e;
      }
      l = wave_sum(l);
      const float inv = 1.0f / l;
      for (int u = lane; u < G; u += 64) {
        const float p = S[g * GP + u] * inv;
        S[g * GP + u] = p;
        Pb[(int64_t)g * G + u] = p;
      }
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < GV; idx += blockDim.x) {
    const int g = idx / V, c = idx % V;
    float acc = 0.f;
#pragma unroll 8
    for (int u = 0; u < G; ++u) acc += S[g * GP + u] * v[u * VP + c];
    zmix[(int64_t)bh * GV + idx] = acc;
  }
}

// token_grads with every operand in LDS (zs, zms, dzs, dUs: [G][VP]; ss, dsl: [G]).
__device__ void token_grads_lds(const float* zs, const float* ss, const float* zms,
                                const float* dzs, float* dUs, float* dsl, float* dUb,
                                float* dsb, float* cenb, int G, int V, float eps) {
  const int VP = V + 1;
  for (int idx = threadIdx.x; idx < G * V; idx += blockDim.x) {
    const int g = idx / V, c = idx % V;
    const float u = dzs[g * VP + c] / (ss[g] + eps);
    dUs[g * VP + c] = u;
    dUb[idx] = u;
  }
  for (int g = threadIdx.x; g < G; g += blockDim.x) {
    float acc = 0.f;
#pragma unroll 8
    for (int c = 0; c < V; ++c) acc += dzs[g * VP + c] * zs[g * VP + c];
    const float d = -acc / (ss[g] + eps);
    dsl[g] = d;
    dsb[g] = d;
  }
  __syncthreads();
  float tot = 0.f;
  for (int g = 0; g < G; ++g) tot += ss[g];
  const float inv = tot > 0.f ? 1.0f / tot : 0.f;
  for (int c = threadIdx.x; c < 2 * V + 1; c += blockDim.x) {
    float acc = 0.f;
    if (c < V) {
#pragma unroll 8
      for (int g = 0; g < G; ++g) acc += ss[g] * zms[g * VP + c];
    } else if (c < 2 * V) {
#pragma unroll 8
      for (int g = 0; g < G; ++g) acc += ss[g] * dUs[g * VP + (c - V)];
    } else {
      for (int g = 0; g < G; ++g) acc += ss[g] * dsl[g];
    }
    cenb[c] = acc * inv;
  }
}

__global__ __launch_bounds__(kAttnThreads) void k_attn_bwd_small(
    const float* z, const float* s, const float* zmix, const float* P, const float* dzm,
    float* dz, float* dU, float* ds, float* cen, float* partM, const float* Wq,
    const float* Wk, const float* Wv, float scale, int G, int V, float eps) {
  extern __shared__ float lds[];
  const int GV = G * V, VV = V * V, GG = G * G, VP = V + 1, GP = G + 1;
  float* zs = lds;              // [G][VP] each, unless noted
  float* Ws = zs + G * VP;      // [3][V][VP]
  float* q = Ws + 3 * V * VP;
  float* k = q + G * VP;
  float* v = k + G * VP;
  float* gz = v + G * VP;
  float* dq = gz + G * VP;
  float* dk = dq + G * VP;
  float* dv = dk + G * VP;
  float* Ps = dv + G * VP;      // [G][GP]
  float* dS = Ps + G * GP;      // [G][GP]
  float* rs = dS + G * GP;      // [G]
  float* dzs = rs + G;          // dz, then the token gradients
  float* zms = dzs + G * VP;    // zmix
  float* dUs = zms + G * VP;
  float* ss = dUs + G * VP;     // [G]
  float* dsl = ss + G;          // [G]
  const int bh = blockIdx.x;
  for (int idx = threadIdx.x; idx < GV; idx += blockDim.x) {
    const int o = (idx / V) * VP + idx % V;
    zs[o] = z[(int64_t)bh * GV + idx];
    gz[o] = dzm[(int64_t)bh * GV + idx];
  }
  for (int idx = threadIdx.x; idx < VV; idx += blockDim.x) {
    const int o = (idx / V) * VP + idx % V;
    Ws[o] = Wq[idx];
    Ws[V * VP + o] = Wk[idx];
    Ws[2 * V * VP + o] = Wv[idx];
  }
  for (int idx = threadIdx.x; idx < GG; idx += blockDim.x)
    Ps[(idx / G) * GP + idx % G] = P[(int64_t)bh * GG + idx];
  __syncthreads();
  attn_project_lds(zs, Ws, q, k, v, G, V);
  __syncthreads();
  for (int idx = threadIdx.x; idx < GG; idx += blockDim.x) {   // dP
    const int g = idx / G, u = idx % G;
    float acc = 0.f;
#pragma unroll 8
    for (int c = 0; c < V; ++c) acc += gz[g * VP + c] * v[u * VP + c];
    dS[g * GP + u] = acc;
  }
  __syncthreads();
  {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    for (int g = wave; g < G; g += nw) {
      float acc = 0.f;
      for (int u = lane; u < G; u += 64) acc += dS[g * GP + u] * Ps[g * GP + u];
      acc = wave_sum(acc);
      if (lane == 0) rs[g] = acc;
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < GG; idx += blockDim.x) {
    const int o = (idx / G) * GP + idx % G;
    dS[o] = Ps[o] * (dS[o] - rs[idx / G]);
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 3 * GV; idx += blockDim.x) {
    const int which = idx / GV, r = idx % GV;
    const int a = r / V, c = r % V;
    float acc = 0.f;
    if (which == 0) {        // dq[a] = scale sum_u dS[a][u] k[u]
#pragma unroll 8
      for (int u = 0; u < G; ++u) acc += dS[a * GP + u] * k[u * VP + c];
      dq[a * VP + c] = scale * acc;
    } else if (which == 1) { // dk[a] = scale sum_g dS[g][a] q[g]
#pragma unroll 8
      for (int g = 0; g < G; ++g) acc += dS[g * GP + a] * q[g * VP + c];
      dk[a * VP + c] = scale * acc;
    } else {                 // dv[a] = sum_g P[g][a] dzmix[g]
#pragma unroll 8
      for (int g = 0; g < G; ++g) acc += Ps[g * GP + a] * gz[g * VP + c];
      dv[a * VP + c] = acc;
    }
  }
  __syncthreads();
  float* dzb = dz + (int64_t)bh * GV;
  for (int idx = threadIdx.x; idx < GV; idx += blockDim.x) {
    const int g = idx / V, e = idx % V;
    float acc = 0.f;
#pragma unroll 8
    for (int c = 0; c < V; ++c)
      acc += dq[g * VP + c] * Ws[e * VP + c] + dk[g * VP + c] * Ws[V * VP + e * VP + c] +
             dv[g * VP + c] * Ws[2 * V * VP + e * VP + c];
    dzb[idx] = acc;
    dzs[g * VP + e] = acc;
  }
  float* pm = partM + (int64_t)bh * 3 * VV;
  for (int idx = threadIdx.x; idx < 3 * VV; idx += blockDim.x) {
    const int which = idx / VV, r = idx % VV;
    const int e = r / V, c = r % V;
    const float* d = which == 0 ? dq : (which == 1 ? dk : dv);
    float acc = 0.f;
#pragma unroll 8
    for (int g = 0; g < G; ++g) acc += zs[g * VP + e] * d[g * VP + c];
    pm[idx] = acc;
  }
  if (s == nullptr) return;
  for (int idx = threadIdx.x; idx < GV; idx += blockDim.x)
    zms[(idx / V) * VP + idx % V] = zmix[(int64_t)bh * GV + idx];
  for (int g = threadIdx.x; g < G; g += blockDim.x) ss[g] = s[(int64_t)bh * G + g];
  __syncthreads();
  token_grads_lds(zs, ss, zms, dzs, dUs, dsl, dU + (int64_t)bh * GV, ds + (int64_t)bh * G,
                  cen + (int64_t)bh * (2 * V + 1), G, V, eps);
}

__global__ __launch_bounds__(kThreads) void k_attn_fwd(const float* z, float* zmix, float* P,
                                                       const float* Wq, const float* Wk,
                                                       const float* Wv, float scale, int G,
                                                       int V) {
  __shared__ float q[kAttnMaxGV], k[kAttnMaxGV], v[kAttnMaxGV];
  __shared__ float Sl[kAttnLdsG * kAttnLdsG];
  const int bh = blockIdx.x;
  const float* zb = z + (int64_t)bh * G * V;
  float* Pb = P + (int64_t)bh * G * G;
  float* S = G <= kAttnLdsG ? Sl : Pb;
  attn_project(zb, Wq, Wk, Wv, q, k, v, G, V);
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * G; idx += blockDim.x) {
    const int g = idx / G, u = idx % G;
    float acc = 0.f;
    for (int c = 0; c < V; ++c) acc += q[g * V + c] * k[u * V + c];
    S[idx] = scale * acc;
  }
  __syncthreads();
  attn_softmax_rows(S, Pb, G);
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * V; idx += blockDim.x) {
    const int g = idx / V, c = idx % V;
    float acc = 0.f;
    for (int u = 0; u < G; ++u) acc += S[(int64_t)g * G + u] * v[u * V + c];
    zmix[(int64_t)bh * G * V + idx] = acc;
  }
}

// Attention backward for one (b, h): dv = P^T dzmix; dP = dzmix v^T;
// dS = P * (dP - rowsum(dP * P)); dq = scale dS k; dk = scale dS^T q;
// dz = dq Wq^T + dk Wk^T + dv Wv^T; parameter partial [dWq; dWk; dWv] = z^T [dq; dk; dv].
// scr per (b, h): dq, dk, dv (G V each) and dS (G G) when G > 64. With s given, also the token
// gradients and shifts (token_grads).
__global__ __launch_bounds__(kThreads) void k_attn_bwd(
    const float* z, const float* s, const float* zmix, const float* P, const float* dzm,
    float* dz, float* dU, float* ds, float* cen, float* scr, float* partM, const float* Wq,
    const float* Wk, const float* Wv, float scale, int G, int V, float eps) {
  __shared__ float q[kAttnMaxGV], k[kAttnMaxGV], v[kAttnMaxGV], gz[kAttnMaxGV];
  __shared__ float Sl[kAttnLdsG * kAttnLdsG];
  __shared__ float rs[256];
  const int bh = blockIdx.x;
  const int GV = G * V;
  const float* zb = z + (int64_t)bh * GV;
  const float* Pb = P + (int64_t)bh * G * G;
  float* dq = scr + (int64_t)bh * (3 * GV + (int64_t)G * G);
  float* dk = dq + GV;
  float* dv = dk + GV;
  float* dS = G <= kAttnLdsG ? Sl : dv + GV;
  attn_project(zb, Wq, Wk, Wv, q, k, v, G, V);
  for (int idx = threadIdx.x; idx < GV; idx += blockDim.x) gz[idx] = dzm[(int64_t)bh * GV + idx];
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * G; idx += blockDim.x) {   // dP
    const int g = idx / G, u = idx % G;
    float acc = 0.f;
    for (int c = 0; c < V; ++c) acc += gz[g * V + c] * v[u * V + c];
    dS[idx] = acc;
  }
  __syncthreads();
  {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    for (int g = wave; g < G; g += nw) {
      float acc = 0.f;
      for (int u = lane; u < G; u += 64) acc += dS[(int64_t)g * G + u] * Pb[(int64_t)g * G + u];
      acc = wave_sum(acc);
      if (lane == 0) rs[g] = acc;
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * G; idx += blockDim.x) {
    const int g = idx / G;
    dS[idx] = Pb[idx] * (dS[idx] - rs[g]);
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 3 * GV; idx += blockDim.x) {
    const int which = idx / GV, r = idx % GV;
    const int a = r / V, c = r % V;
    float acc = 0.f;
    if (which == 0) {        // dq[a] = scale sum_u dS[a][u] k[u]
      for (int u = 0; u < G; ++u) acc += dS[(int64_t)a * G + u] * k[u * V + c];
      dq[r] = scale * acc;
    } else if (which == 1) { // dk[a] = scale sum_g dS[g][a] q[g]
      for (int g = 0; g < G; ++g) acc += dS[(int64_t)g * G + a] * q[g * V + c];
      dk[r] = scale * acc;
    } else {                 // dv[a] = sum_g P[g][a] dzmix[g]
      for (int g = 0; g < G; ++g) acc += Pb[(int64_t)g * G + a] * gz[g * V + c];
      dv[r] = acc;
    }
  }
  __syncthreads();
  float* dzb = dz + (int64_t)bh * GV;
  for (int idx = threadIdx.x; idx < GV; idx += blockDim.x) {
    const int g = idx / V, e = idx % V;
    float acc = 0.f;
    for (int c = 0; c < V; ++c)
      acc += dq[(int64_t)g * V + c] * Wq[e * V + c] + dk[(int64_t)g * V + c] * Wk[e * V + c] +
             dv[(int64_t)g * V + c] * Wv[e * V + c];
    dzb[idx] = acc;
  }
  float* pm = partM + (int64_t)bh * 3 * V * V;
  for (int idx = threadIdx.x; idx < 3 * V * V; idx += blockDim.x) {
    const int which = idx / (V * V), r = idx % (V * V);
    const int e = r / V, c = r % V;
    const float* d = which == 0 ? dq : (which == 1 ? dk : dv);
    float acc = 0.f;
    for (int g = 0; g < G; ++g) acc += zb[(int64_t)g * V + e] * d[(int64_t)g * V + c];
    pm[idx] = acc;
  }
  if (s == nullptr) return;
  __syncthreads();
  token_grads(zb, s + (int64_t)bh * G, zmix + (int64_t)bh * GV, dzb, dU + (int64_t)bh * GV,
              ds + (int64_t)bh * G, cen + (int64_t)bh * (2 * V + 1), G, V, eps);
}

inline unsigned blocks(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }
// Floats of one (b, h) mix-parameter partial.
inline int64_t mix_partial_len(const Geom& g, int kind) {
  return kind == 1 ? (int64_t)g.G * g.G : (kind == 2 ? (int64_t)g.V * g.V : 3LL * g.V * g.V);
}
inline bool attn_small(const Geom& g) {
  return g.G * g.V <= kAttnSmallGV && g.G <= 64 && g.V <= 64;
}
// Dynamic LDS above 64 KB has to be allowed per kernel once.
template <typename K>
hipError_t allow_lds(K kernel, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

}  // namespace

hipError_t launch_reduce_tokens(const Geom& g, const float* partU, const float* partS,
                                int chunks, float* z, float* s, hipStream_t st) {
  dim3 grid(blocks((int64_t)g.G * g.V, kCols), g.BH());
  hipLaunchKernelGGL(k_reduce_tokens, grid, dim3(kRedThreads), 0, st, partU, partS, z, s, chunks,
                     g.G, g.V, g.eps);
  return hipGetLastError();
}

hipError_t launch_reduce_rows(const Geom& g, const float* part, float* out, int chunks,
                              int64_t len, hipStream_t st) {
  dim3 grid(blocks(len, kCols), g.BH());
  hipLaunchKernelGGL(k_reduce_rows, grid, dim3(kRedThreads), 0, st, part, out, chunks, len);
  return hipGetLastError();
}

hipError_t launch_reduce_params(const Geom& g, const float* part, float* dWs, float* dbias,
                                float* dtau, int chunks, int nblk, const MixArgs* m,
                                const float* partM, float* dmix, hipStream_t st) {
  const int64_t ncol = (int64_t)g.D * g.G + g.G;
  const bool with_mix = m != nullptr && dmix != nullptr && m->kind != 0;
  const int64_t mix_len = with_mix ? mix_partial_len(g, m->kind) : 0;
  const bool mix_per_head = with_mix && m->kind == 1 && m->a_per_head;
  const unsigned nb = blocks(ncol, kColsWide) + 1 + (with_mix ? blocks(mix_len, kColsWide) : 0);
  const int heads = std::max(g.ws_per_head ? g.H : 1, mix_per_head ? g.H : 1);
  hipLaunchKernelGGL(k_reduce_params, dim3(nb, heads), dim3(kRedThreads), 0, st, part, dWs,
                     dbias, dtau, (int)g.B, g.H, chunks, nblk, g.D, g.G, g.ws_per_head ? 1 : 0, partM,
                     with_mix ? dmix : nullptr, mix_len, mix_per_head ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_mix(const Geom& g, const MixArgs& m, const float* z, float* zmix,
                      float* attn, hipStream_t st) {
  const int BH = g.BH();
  if (tok_fused(g, m.kind)) return launch_tok_fwd(g, m, z, zmix, attn, st);
  if (m.kind == 3) {
    if (attn_small(g)) {
      const size_t lds = sizeof(float) * (size_t)attn_small_fwd_floats(g.G, g.V);
      hipError_t e = allow_lds(k_attn_fwd_small, lds);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(k_attn_fwd_small, dim3(BH), dim3(kAttnThreads), lds, st, z, zmix, attn,
                         m.Wq, m.Wk, m.Wv, m.scale, g.G, g.V);
    } else {
      hipLaunchKernelGGL(k_attn_fwd, dim3(BH), dim3(kThreads), 0, st, z, zmix, attn, m.Wq,
                         m.Wk, m.Wv, m.scale, g.G, g.V);
    }
  } else {
    dim3 grid(blocks((int64_t)g.G * g.V, kThreads), BH);
    hipLaunchKernelGGL(k_mix_linear, grid, dim3(kThreads), 0, st, z, zmix, m.A, m.Wc, m.kind,
                       m.a_per_head ? 1 : 0, g.H, g.G, g.V);
  }
  return hipGetLastError();
}

hipError_t launch_mix_bwd(const Geom& g, const MixArgs& m, const float* z, const float* s,
                          const float* zmix, const float* attn, const float* dzm, float* dz,
                          float* dU, float* ds, float* cen, float* scr, float* partM,
                          float* dmix, bool reduce_params, hipStream_t st) {
  const int BH = g.BH();
  hipError_t e;
  if (tok_fused(g, m.kind)) {
    e = launch_tok_bwd(g, m, z, s, zmix, attn, dzm, dz, dU, ds, cen, partM, st);
  } else if (m.kind == 3) {
    if (attn_small(g)) {
      const size_t lds = sizeof(float) * (size_t)attn_small_bwd_floats(g.G, g.V);
      hipError_t e = allow_lds(k_attn_bwd_small, lds);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(k_attn_bwd_small, dim3(BH), dim3(kAttnThreads), lds, st, z, s, zmix, attn,
                         dzm, dz, dU, ds, cen, partM, m.Wq, m.Wk, m.Wv, m.scale, g.G, g.V, g.eps);
    } else {
      hipLaunchKernelGGL(k_attn_bwd, dim3(BH), dim3(kThreads), 0, st, z, s, zmix, attn, dzm, dz,
                         dU, ds, cen, scr, partM, m.Wq, m.Wk, m.Wv, m.scale, g.G, g.V, g.eps);
    }
  } else {
    dim3 grid(blocks((int64_t)g.G * g.V, kThreads), BH);
    hipLaunchKernelGGL(k_mix_dz_linear, grid, dim3(kThreads), 0, st, dzm, dz, m.A, m.Wc, m.kind,
                       m.a_per_head ? 1 : 0, g.H, g.G, g.V);
    if (dmix != nullptr && m.kind != 0) {
      const int64_t len = m.kind == 1 ? (int64_t)g.G * g.G : (int64_t)g.V * g.V;
      dim3 pg(blocks(len, kThreads), BH);
      hipLaunchKernelGGL(k_mix_param_linear, pg, dim3(kThreads), 0, st, z, dzm, partM, m.kind,
                         g.G, g.V);
    }
    if (s != nullptr)
      hipLaunchKernelGGL(k_token_grads, dim3(BH), dim3(kThreads), 0, st, z, s, zmix, dz, dU, ds,
                         cen, g.G, g.V, g.eps);
  }
  if (!tok_fused(g, m.kind)) e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (reduce_params && dmix != nullptr && m.kind != 0) {
    const int64_t len = mix_partial_len(g, m.kind);
    const bool per_head = m.kind == 1 && m.a_per_head;
    dim3 grid(blocks(len, kColsWide), per_head ? g.H : 1);
    hipLaunchKernelGGL(k_reduce_mixparams, grid, dim3(kRedThreads), 0, st, partM, dmix, (int)g.B,
                       g.H, len, per_head ? 1 : 0);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace fs
