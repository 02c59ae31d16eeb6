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
// Linear token maps for token sets too large for the single-workgroup LDS kernels: batched
// fp32 products C_o = alpha sum_s A_{o,s} B_{o,s} on MFMA, one wavefront per 16 x 16 output
// tile, operands read straight from global memory (they are small and cache resident). A
// strided descriptor covers the forward map, its transpose, and the parameter gradients
// summed over samples and heads without partials.
// ---------------------------------------------------------------------------------------
struct GemmDesc {
  // element (m, k) of A for output o and summand s: A[(o % a_mod) * a_o + s * a_s + m * a_rs + k * a_cs]
  const float* A;
  int64_t a_rs, a_cs, a_o, a_s;
  int a_mod;
  const float* B;  // element (k, n): B[o * b_o + s * b_s + k * b_rs + n * b_cs]
  int64_t b_rs, b_cs, b_o, b_s;
  float* C;  // element (m, n): C[o * c_o + m * c_rs + n]
  int64_t c_rs, c_o;
  int M, N, K, nsum;
  float alpha;
  int accumulate;  // nonzero: C += alpha * product
};

constexpr int kGemmWaves = 4;

__global__ __launch_bounds__(64 * kGemmWaves) void k_tile_gemm(GemmDesc d) {
  typedef float f4 __attribute__((ext_vector_type(4)));
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int t = blockIdx.x * kGemmWaves + (threadIdx.x >> 6);
  const int tn = d.N >> 4;
  if (t >= (d.M >> 4) * tn) return;  // whole wavefronts only
  const int m0 = (t / tn) << 4, n0 = (t % tn) << 4;
  const int o = blockIdx.y;
  const float* Ao = d.A + (int64_t)(o % d.a_mod) * d.a_o + (int64_t)(m0 + i) * d.a_rs;
  const float* Bo = d.B + (int64_t)o * d.b_o + (int64_t)(n0 + i) * d.b_cs;
  // four independent accumulation chains (k steps round robin), added at the end: shorter
  // rounding-error walks over long K and overlapping MFMA latencies
  f4 ch[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) ch[c] = f4{0.f, 0.f, 0.f, 0.f};
  for (int sidx = 0; sidx < d.nsum; ++sidx) {
    const float* As = Ao + (int64_t)sidx * d.a_s;
    const float* Bs = Bo + (int64_t)sidx * d.b_s;
    int k = 0;
    const int kfull = d.K & ~31;
    if (kfull > 0) {
      // eight products' operands per block; the next block's loads are issued before the
      // current block's MFMAs (the last block reloads itself, so every load is in bounds)
      float av[8], bv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        av[u] = As[(int64_t)(4 * u + j) * d.a_cs];
        bv[u] = Bs[(int64_t)(4 * u + j) * d.b_rs];
      }
      for (; k < kfull; k += 32) {
        const int kn = k + 32 < kfull ? k + 32 : k;
        float an[8], bn[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          an[u] = As[(int64_t)(kn + 4 * u + j) * d.a_cs];
          bn[u] = Bs[(int64_t)(kn + 4 * u + j) * d.b_rs];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
          ch[u & 3] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u], bv[u], ch[u & 3], 0, 0, 0);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          av[u] = an[u];
          bv[u] = bn[u];
        }
      }
    }
    for (int u = 0; k < d.K; k += 4, ++u)
      ch[u & 3] = __builtin_amdgcn_mfma_f32_16x16x4f32(As[(int64_t)(k + j) * d.a_cs],
                                                       Bs[(int64_t)(k + j) * d.b_rs], ch[u & 3], 0,
                                                       0, 0);
  }
  const f4 acc = (ch[0] + ch[1]) + (ch[2] + ch[3]);
  float* Co = d.C + (int64_t)o * d.c_o + n0 + i;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float* c = Co + (int64_t)(m0 + 4 * j + r) * d.c_rs;
    *c = d.accumulate ? *c + d.alpha * acc[r] : d.alpha * acc[r];
  }
}

static hipError_t run_gemm(const GemmDesc& d, int nout, hipStream_t st) {
  const int tiles = (d.M / 16) * (d.N / 16);
  hipLaunchKernelGGL(k_tile_gemm, dim3((tiles + kGemmWaves - 1) / kGemmWaves, nout),
                     dim3(64 * kGemmWaves), 0, st, d);
  return hipGetLastError();
}

// Token gradients and the shifts the backward pass B uses, one 1024-thread workgroup per
// (b, h): dU = dz / (s + eps), ds = -sum_v dz z / (s + eps), and the mass-weighted slot means
// cen = [sum_g m_g zmix[g][:], sum_g m_g dU[g][:], sum_g m_g ds[g]] with m_g = s_g / sum s.
// Each of the 2V + 1 mean columns is summed by 16 threads over interleaved slots, then
// combined over those threads in a fixed order.
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
  __threadfence_block();
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
  const int ncol = 2 * V + 1;
  for (int base = 0; base < ncol * 16; base += blockDim.x) {
    const int idx = base + threadIdx.x;
    const int c = idx >> 4, part = idx & 15;
    float acc = 0.f;
    if (c < ncol) {
      if (c < V) {
        for (int g = part; g < G; g += 16) acc += sb[g] * zmb[(int64_t)g * V + c];
      } else if (c < 2 * V) {
        for (int g = part; g < G; g += 16) acc += sb[g] * dUb[(int64_t)g * V + (c - V)];
      } else {
        for (int g = part; g < G; g += 16) acc += sb[g] * dsb[g];
      }
    }
    // fixed-order sum over the 16 threads of a column (aligned groups of 16 lanes)
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, 16);
    if (c < ncol && part == 0) cenb[c] = acc * inv;
  }
}

constexpr int kTokGradThreads = 1024;

__global__ __launch_bounds__(kTokGradThreads) void k_token_grads(const float* z, const float* s,
                                                                 const float* zmix,
                                                                 const float* dz, float* dU,
                                                                 float* ds, float* cen, int G,
                                                                 int V, float eps) {
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
constexpr int kAttnMaxGV = 8192;   // q, k, v of one (b, h) in LDS
constexpr int kAttnLdsMaxG = 256;
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

// ---------------------------------------------------------------------------------------
// Attention among large token sets (beyond the LDS kernels' limits), any G multiple of 16.
// Forward: one wavefront per (b, h, block of 16 token rows) computes those rows with fp32
// MFMA and needs no workspace. With r = (z Wq) Wk^T for its rows, the scores are
// S[g][u] = scale r_g . z_u (= scale q_g . k_u). A first sweep over the key tiles forms each
// row's maximum and sum of exponentials, a second recomputes the scores, writes
// P = softmax_row(S) and accumulates T = P z, and zmix = T Wv (= P v by associativity, so
// v is never formed). Operands come from global memory (small, cache resident); LDS only
// re-lays out 16-row intermediates between products.
// MFMA 16x16x4 lane layout (lane = i + 16 j): A[m = i][k = j], B[k = j][n = i],
// C[m = 4 j + r][n = i] in register r.
// ---------------------------------------------------------------------------------------
constexpr int kAttnRowWaves = 4;

__device__ __forceinline__ void lane_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}
__device__ __forceinline__ float row16_max_x(float v) {
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 16));
  return v;
}
__device__ __forceinline__ float row16_sum_x(float v) {
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) v += __shfl_xor(v, off, 16);
  return v;
}

template <int V>
__global__ __launch_bounds__(64 * kAttnRowWaves) void k_attn_rows(
    const float* z, float* zmix, float* P, const float* Wq, const float* Wk, const float* Wv,
    float scale, int G, int BH) {
  typedef float f4 __attribute__((ext_vector_type(4)));
  constexpr int VT = V / 16, VK = V / 4;
  constexpr float kLog2e = 1.4426950408889634f;
  __shared__ float stage[kAttnRowWaves][16 * V];
  __shared__ float ptile[kAttnRowWaves][16 * 16];
  const int lane = threadIdx.x & 63, i = lane & 15, j = lane >> 4;
  const int wv = threadIdx.x >> 6;
  const int nrb = G >> 4;
  const int64_t job = (int64_t)blockIdx.x * kAttnRowWaves + wv;
  if (job >= (int64_t)BH * nrb) return;  // whole wavefronts; no workgroup barrier follows
  const int bh = (int)(job / nrb), g0 = (int)(job % nrb) << 4;
  const float* zb = z + (int64_t)bh * G * V;
  float* Pb = P + (int64_t)bh * G * G;
  float* sg = stage[wv];
  float* pt = ptile[wv];
  auto mfma = [](float a, float b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  };
  f4 acc[VT];
  // q = z[g0 : g0 + 16] Wq
#pragma unroll
  for (int nt = 0; nt < VT; ++nt) acc[nt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k0 = 0; k0 < V; k0 += 4) {
    const float a = zb[(int64_t)(g0 + i) * V + k0 + j];
#pragma unroll
    for (int nt = 0; nt < VT; ++nt) acc[nt] = mfma(a, Wq[(k0 + j) * V + 16 * nt + i], acc[nt]);
  }
#pragma unroll
  for (int nt = 0; nt < VT; ++nt)
#pragma unroll
    for (int r = 0; r < 4; ++r) sg[(4 * j + r) * V + 16 * nt + i] = acc[nt][r];
  lane_lds_sync();
  // r = q Wk^T (B[k][n] = Wk[n][k])
#pragma unroll
  for (int nt = 0; nt < VT; ++nt) acc[nt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k0 = 0; k0 < V; k0 += 4) {
    const float a = sg[i * V + k0 + j];
#pragma unroll
    for (int nt = 0; nt < VT; ++nt) acc[nt] = mfma(a, Wk[(16 * nt + i) * V + k0 + j], acc[nt]);
  }
  lane_lds_sync();
#pragma unroll
  for (int nt = 0; nt < VT; ++nt)
#pragma unroll
    for (int r = 0; r < 4; ++r) sg[(4 * j + r) * V + 16 * nt + i] = acc[nt][r];
  lane_lds_sync();
  // score A operand, in base-2 units: ra[kk] = scale log2(e) r[g0 + i][4 kk + j]
  float ra[VK];
#pragma unroll
  for (int kk = 0; kk < VK; ++kk) ra[kk] = (scale * kLog2e) * sg[i * V + 4 * kk + j];
  // tile ut of the scores: s[r] = S2[g0 + 4 j + r][16 ut + i]
  auto score = [&](int ut) {
    f4 sc = {0.f, 0.f, 0.f, 0.f};
    const float* zu = zb + (int64_t)(16 * ut + i) * V + j;
#pragma unroll
    for (int kk = 0; kk < VK; ++kk) sc = mfma(ra[kk], zu[4 * kk], sc);
    return sc;
  };
  // sweep 1: per-lane running max and sum over the lane's own columns, then over the row
  float mr[4], lr[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    mr[r] = -INFINITY;
    lr[r] = 0.f;
  }
  for (int ut = 0; ut < nrb; ++ut) {
    const f4 sc = score(ut);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float mn = fmaxf(mr[r], sc[r]);
      lr[r] = lr[r] * exp2f(mr[r] - mn) + exp2f(sc[r] - mn);
      mr[r] = mn;
    }
  }
  float M[4], invL[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    M[r] = row16_max_x(mr[r]);
    invL[r] = 1.0f / row16_sum_x(lr[r] * exp2f(mr[r] - M[r]));
  }
  // sweep 2: P and T^T = z^T P^T (C layout: T[ct][r] = T[g0 + i][16 ct + 4 j + r]), in four
  // accumulation chains (one per k step of a key tile) added at the end
  f4 Tc[4][VT];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int ct = 0; ct < VT; ++ct) Tc[c][ct] = f4{0.f, 0.f, 0.f, 0.f};
  for (int ut = 0; ut < nrb; ++ut) {
    const f4 sc = score(ut);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float p = exp2f(sc[r] - M[r]) * invL[r];
      Pb[(int64_t)(g0 + 4 * j + r) * G + 16 * ut + i] = p;
      pt[(4 * j + r) * 16 + i] = p;
    }
    lane_lds_sync();
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float b = pt[i * 16 + 4 * c + j];   // P[g0 + i][16 ut + 4 c + j]
      const float* zr = zb + (int64_t)(16 * ut + 4 * c + j) * V + i;
#pragma unroll
      for (int ct = 0; ct < VT; ++ct) Tc[c][ct] = mfma(zr[16 * ct], b, Tc[c][ct]);
    }
    lane_lds_sync();
  }
  f4 T[VT];
#pragma unroll
  for (int ct = 0; ct < VT; ++ct) T[ct] = (Tc[0][ct] + Tc[1][ct]) + (Tc[2][ct] + Tc[3][ct]);
  // zmix = T Wv: A[i][k0 + j] = T[g0 + i][k0 + j] through LDS
#pragma unroll
  for (int ct = 0; ct < VT; ++ct)
#pragma unroll
    for (int r = 0; r < 4; ++r) sg[i * V + 16 * ct + 4 * j + r] = T[ct][r];
  lane_lds_sync();
#pragma unroll
  for (int nt = 0; nt < VT; ++nt) acc[nt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k0 = 0; k0 < V; k0 += 4) {
    const float a = sg[i * V + k0 + j];
#pragma unroll
    for (int nt = 0; nt < VT; ++nt) acc[nt] = mfma(a, Wv[(k0 + j) * V + 16 * nt + i], acc[nt]);
  }
  float* zo = zmix + ((int64_t)bh * G + g0) * V;
#pragma unroll
  for (int nt = 0; nt < VT; ++nt)
#pragma unroll
    for (int r = 0; r < 4; ++r) zo[(4 * j + r) * V + 16 * nt + i] = acc[nt][r];
}

// dS = P * (dP - rowsum(dP * P)) in place over dP, one wavefront per row of one (b, h).
__global__ __launch_bounds__(256) void k_attn_ds(const float* P, float* dS, int64_t rows,
                                                 int G) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const float* p = P + row * G;
  float* d = dS + row * G;
  float acc = 0.f;
  for (int u = lane; u < G; u += 64) acc += d[u] * p[u];
  acc = wave_sum(acc);
  for (int u = lane; u < G; u += 64) d[u] = p[u] * (d[u] - acc);
}

inline unsigned blocks(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }
// Floats of one (b, h) mix-parameter partial.
inline int64_t mix_partial_len(const Geom& g, int kind) {
  return kind == 1 ? (int64_t)g.G * g.G : (kind == 2 ? (int64_t)g.V * g.V : 3LL * g.V * g.V);
}


}  // namespace

bool attn_rows(const Geom& g, int kind) {
  return kind == 3 && !tok_fused(g, kind) && (g.G > kAttnLdsMaxG || (int64_t)g.G * g.V > kAttnMaxGV);
}

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

// Whether the mix-parameter gradient goes through per-(b, h) partials (the LDS kernels and
// attention) or is written directly (the batched products of the linear maps).
static bool mix_params_in_partials(const Geom& g, int kind) {
  return tok_fused(g, kind) || (kind == 3 && !attn_rows(g, kind));
}

hipError_t launch_reduce_params(const Geom& g, const float* part, float* dWs, float* dbias,
                                float* dtau, int chunks, int nblk, const MixArgs* m,
                                const float* partM, float* dmix, hipStream_t st) {
  const int64_t ncol = (int64_t)g.D * g.G + g.G;
  const bool with_mix =
      m != nullptr && dmix != nullptr && m->kind != 0 && mix_params_in_partials(g, m->kind);
  const int64_t mix_len = with_mix ? mix_partial_len(g, m->kind) : 0;
  const bool mix_per_head = with_mix && m->kind == 1 && m->a_per_head;
  const unsigned nb = blocks(ncol, kColsWide) + 1 + (with_mix ? blocks(mix_len, kColsWide) : 0);
  const int heads = std::max(g.ws_per_head ? g.H : 1, mix_per_head ? g.H : 1);
  hipLaunchKernelGGL(k_reduce_params, dim3(nb, heads), dim3(kRedThreads), 0, st, part, dWs,
                     dbias, dtau, (int)g.B, g.H, chunks, nblk, g.D, g.G, g.ws_per_head ? 1 : 0, partM,
                     with_mix ? dmix : nullptr, mix_len, mix_per_head ? 1 : 0);
  return hipGetLastError();
}

// Linear maps of one (b, h) per output: zmix = A z (fixed matrix) or z W_c (channel map).
static GemmDesc mix_fwd_desc(const Geom& g, const MixArgs& m, const float* z, float* zmix) {
  const int64_t GV = (int64_t)g.G * g.V;
  GemmDesc d{};
  if (m.kind == 1) {  // (G x G) x (G x V)
    d = GemmDesc{m.A, g.G, 1, (int64_t)g.G * g.G, 0, m.a_per_head ? g.H : 1,
                 z, g.V, 1, GV, 0, zmix, g.V, GV, g.G, g.V, g.G, 1, 1.0f};
  } else {            // (G x V) x (V x V)
    d = GemmDesc{z, g.V, 1, GV, 0, 1 << 30, m.Wc, g.V, 1, 0, 0, zmix, g.V, GV, g.G, g.V, g.V, 1, 1.0f};
  }
  return d;
}

hipError_t launch_mix(const Geom& g, const MixArgs& m, const float* z, float* zmix,
                      float* attn, hipStream_t st) {
  const int BH = g.BH();
  if (tok_fused(g, m.kind)) return launch_tok_fwd(g, m, z, zmix, attn, st);
  if (attn_rows(g, m.kind)) {
    const int64_t jobs = (int64_t)BH * (g.G / 16);
    const dim3 grid(blocks(jobs, kAttnRowWaves)), block(64 * kAttnRowWaves);
    if (g.V == 16)
      hipLaunchKernelGGL(k_attn_rows<16>, grid, block, 0, st, z, zmix, attn, m.Wq, m.Wk, m.Wv,
                         m.scale, g.G, BH);
    else if (g.V == 32)
      hipLaunchKernelGGL(k_attn_rows<32>, grid, block, 0, st, z, zmix, attn, m.Wq, m.Wk, m.Wv,
                         m.scale, g.G, BH);
    else if (g.V == 64)
      hipLaunchKernelGGL(k_attn_rows<64>, grid, block, 0, st, z, zmix, attn, m.Wq, m.Wk, m.Wv,
                         m.scale, g.G, BH);
    else
      return hipErrorInvalidValue;
    return hipGetLastError();
  }
  if (m.kind == 3) {
    hipLaunchKernelGGL(k_attn_fwd, dim3(BH), dim3(kThreads), 0, st, z, zmix, attn, m.Wq,
                       m.Wk, m.Wv, m.scale, g.G, g.V);
    return hipGetLastError();
  }
  if (m.kind == 0) {
    return hipMemcpyAsync(zmix, z, sizeof(float) * (size_t)BH * g.G * g.V,
                          hipMemcpyDeviceToDevice, st);
  }
  return run_gemm(mix_fwd_desc(g, m, z, zmix), BH, st);
}

// out[c] = sum over r of part[r][c] (rows summed in a fixed order), one output row.
static hipError_t launch_sum_rows(const float* part, float* out, int rows, int64_t len,
                                  hipStream_t st) {
  dim3 grid((unsigned)((len + kCols - 1) / kCols), 1);
  hipLaunchKernelGGL(k_reduce_rows, grid, dim3(kRedThreads), 0, st, part, out, rows, len);
  return hipGetLastError();
}

// Backward of the large-token-set attention as batched MFMA products (k_tile_gemm) and one
// row kernel. scr: q, k, v (B H G V each), dS (B H G G), dq, dk, dv (B H G V each).
//   q, k, v = z W;  dP = dzmix v^T;  dS = P * (dP - rowsum(dP * P));  dv = P^T dzmix;
//   dq = scale dS k;  dk = scale dS^T q;  dz = dq Wq^T + dk Wk^T + dv Wv^T;
//   [dWq; dWk; dWv] = sum over (b, h) of z^T [dq; dk; dv].
static hipError_t attn_rows_bwd(const Geom& g, const MixArgs& m, const float* z, const float* s,
                                const float* zmix, const float* P, const float* dzm, float* dz,
                                float* dU, float* ds, float* cen, float* scr, float* dmix,
                                hipStream_t st) {
  const int BH = g.BH(), G = g.G, V = g.V;
  const int64_t GV = (int64_t)G * V, GG = (int64_t)G * G, T = BH * GV;
  constexpr int kPer = 1 << 30;  // a_mod: A advances with the output index
  float* q = scr;
  float* k = q + T;
  float* v = k + T;
  float* dS = v + T;
  float* dq = dS + BH * GG;
  float* dk = dq + T;
  float* dv = dk + T;
  const float* W[3] = {m.Wq, m.Wk, m.Wv};
  float* qkv[3] = {q, k, v};
  float* dqkv[3] = {dq, dk, dv};
  hipError_t e = hipSuccess;
  for (int w = 0; w < 3 && e == hipSuccess; ++w)  // q, k, v = z W
    e = run_gemm(GemmDesc{z, V, 1, GV, 0, kPer, W[w], V, 1, 0, 0, qkv[w], V, GV, G, V, V, 1,
                          1.0f, 0},
                 BH, st);
  if (e == hipSuccess)  // dP = dzmix v^T (into dS)
    e = run_gemm(GemmDesc{dzm, V, 1, GV, 0, kPer, v, 1, V, GV, 0, dS, G, GG, G, G, V, 1, 1.0f, 0},
                 BH, st);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(k_attn_ds, dim3(blocks((int64_t)BH * G, 4)), dim3(256), 0, st, P, dS,
                       (int64_t)BH * G, G);
    e = hipGetLastError();
  }
  if (e == hipSuccess)  // dv = P^T dzmix
    e = run_gemm(GemmDesc{P, 1, G, GG, 0, kPer, dzm, V, 1, GV, 0, dv, V, GV, G, V, G, 1, 1.0f, 0},
                 BH, st);
  if (e == hipSuccess)  // dq = scale dS k
    e = run_gemm(GemmDesc{dS, G, 1, GG, 0, kPer, k, V, 1, GV, 0, dq, V, GV, G, V, G, 1, m.scale, 0},
                 BH, st);
  if (e == hipSuccess)  // dk = scale dS^T q
    e = run_gemm(GemmDesc{dS, 1, G, GG, 0, kPer, q, V, 1, GV, 0, dk, V, GV, G, V, G, 1, m.scale, 0},
                 BH, st);
  for (int w = 0; w < 3 && e == hipSuccess; ++w)  // dz = sum_w d[w] W[w]^T
    e = run_gemm(GemmDesc{dqkv[w], V, 1, GV, 0, kPer, W[w], 1, V, 0, 0, dz, V, GV, G, V, V, 1,
                          1.0f, w > 0 ? 1 : 0},
                 BH, st);
  // dW = sum over (b, h, g) of z^T d[w]: the B H G products split over S workgroup-sized K
  // ranges whose partials (in the dS region, free by now) are then summed in order
  const int64_t KT = (int64_t)BH * G;
  int64_t Ks = 16;
  for (int64_t c : {256, 128, 64, 32})
    if (KT % c == 0 && KT / c >= 64) {
      Ks = c;
      break;
    }
  const int S = (int)(KT / Ks);
  if (dmix != nullptr && (int64_t)S * V * V > BH * GG) return hipErrorInvalidValue;
  for (int w = 0; w < 3 && e == hipSuccess && dmix != nullptr; ++w) {
    e = run_gemm(GemmDesc{z, 1, V, Ks * V, 0, kPer, dqkv[w], V, 1, Ks * V, 0, dS, V,
                          (int64_t)V * V, V, V, (int)Ks, 1, 1.0f, 0},
                 S, st);
    if (e == hipSuccess) e = launch_sum_rows(dS, dmix + (int64_t)w * V * V, S, (int64_t)V * V, st);
  }
  if (e == hipSuccess && s != nullptr) {
    hipLaunchKernelGGL(k_token_grads, dim3(BH), dim3(kTokGradThreads), 0, st, z, s, zmix, dz, dU,
                       ds, cen, G, V, g.eps);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_mix_bwd(const Geom& g, const MixArgs& m, const float* z, const float* s,
                          const float* zmix, const float* attn, const float* dzm, float* dz,
                          float* dU, float* ds, float* cen, float* scr, float* partM,
                          float* dmix, bool reduce_params, hipStream_t st) {
  const int BH = g.BH();
  const int64_t GV = (int64_t)g.G * g.V;
  hipError_t e = hipSuccess;
  if (tok_fused(g, m.kind)) {
    e = launch_tok_bwd(g, m, z, s, zmix, attn, dzm, dz, dU, ds, cen, partM, st);
  } else if (attn_rows(g, m.kind)) {
    e = attn_rows_bwd(g, m, z, s, zmix, attn, dzm, dz, dU, ds, cen, scr, dmix, st);
  } else if (m.kind == 3) {
    hipLaunchKernelGGL(k_attn_bwd, dim3(BH), dim3(kThreads), 0, st, z, s, zmix, attn, dzm, dz,
                       dU, ds, cen, scr, partM, m.Wq, m.Wk, m.Wv, m.scale, g.G, g.V, g.eps);
    e = hipGetLastError();
  } else {
    if (m.kind == 0) {
      e = hipMemcpyAsync(dz, dzm, sizeof(float) * (size_t)BH * GV, hipMemcpyDeviceToDevice, st);
    } else if (m.kind == 1) {  // dz = A^T dzmix
      e = run_gemm(GemmDesc{m.A, 1, g.G, (int64_t)g.G * g.G, 0, m.a_per_head ? g.H : 1, dzm,
                            g.V, 1, GV, 0, dz, g.V, GV, g.G, g.V, g.G, 1, 1.0f},
                   BH, st);
    } else {                   // dz = dzmix W_c^T
      e = run_gemm(GemmDesc{dzm, g.V, 1, GV, 0, 1 << 30, m.Wc, 1, g.V, 0, 0, dz, g.V, GV, g.G,
                            g.V, g.V, 1, 1.0f},
                   BH, st);
    }
    if (e == hipSuccess && dmix != nullptr && m.kind == 1) {
      // dA = sum over (b, h) of dzmix z^T, or over b for each head's own A
      if (m.a_per_head)
        e = run_gemm(GemmDesc{dzm, g.V, 1, GV, (int64_t)g.H * GV, 1 << 30, z, 1, g.V, GV,
                              (int64_t)g.H * GV, dmix, g.G, (int64_t)g.G * g.G, g.G, g.G, g.V,
                              (int)g.B, 1.0f},
                     g.H, st);
      else
        e = run_gemm(GemmDesc{dzm, g.V, 1, 0, GV, 1, z, 1, g.V, 0, GV, dmix, g.G, 0, g.G, g.G,
                              g.V, BH, 1.0f},
                     1, st);
    }
    if (e == hipSuccess && dmix != nullptr && m.kind == 2)  // dW_c = sum over (b, h) of z^T dzmix
      e = run_gemm(GemmDesc{z, 1, g.V, 0, GV, 1, dzm, g.V, 1, 0, GV, dmix, g.V, 0, g.V, g.V,
                            g.G, BH, 1.0f},
                   1, st);
    if (e == hipSuccess && s != nullptr) {
      hipLaunchKernelGGL(k_token_grads, dim3(BH), dim3(kTokGradThreads), 0, st, z, s, zmix, dz,
                         dU, ds, cen, g.G, g.V, g.eps);
      e = hipGetLastError();
    }
  }
  if (e != hipSuccess) return e;
  if (reduce_params && dmix != nullptr && m.kind != 0 && mix_params_in_partials(g, m.kind)) {
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
