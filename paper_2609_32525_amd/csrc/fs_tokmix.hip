// Token mix and its backward for token sets that fit in LDS: one workgroup per (sample, head)
// holds z, the mix parameters and every intermediate in LDS, and each G x V, G x G or V x V
// product is a set of 16 x 16 MFMA tiles (v_mfma_f32_16x16x4_f32) spread over the
// workgroup's wavefronts. Kinds (paper: Sec. 2; Eq. (1) with a constant or attention core):
//   identity     z' = z
//   fixed matrix z'_g = sum_h A[g][h] z_h                 (A shared by heads or per head)
//   channel map  z' = z W_c                                (the attention-free variant)
//   attention    q, k, v = z W_q, z W_k, z W_v;  P = softmax_row(scale q k^T);  z' = P v
// The backward computes dz = Mix^T(dz'), the per-(b, h) parameter partials, and the token
// gradients of the slice normalisation: dU = dz / (s + eps), ds = -sum_v dz z / (s + eps),
// with the mass-weighted slot means of z', dU and ds that the backward pass B subtracts.
//
// LDS matrices are row-major with one float of padding per row (stride V + 1 or G + 1), so
// the MFMA operand reads (16 rows of one column, or 16 columns of one row) and the
// transposed reads of the backward are free of bank conflicts.

#include <hip/hip_runtime.h>

#include "fs_internal.h"

namespace fs {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kTokThreads = 1024;
constexpr size_t kTokLdsMax = 160 * 1024;

// Element (r, c) of an LDS matrix at p[r * rs + c * cs].
struct Mat {
  const float* p;
  int rs, cs;
  __device__ float at(int r, int c) const { return p[r * rs + c * cs]; }
};
__device__ __forceinline__ Mat mat(const float* p, int rs, int cs) { return Mat{p, rs, cs}; }

// One 16 x 16 tile of C = A B over k in [0, K), K a multiple of 4. Lane (j, i) feeds
// A(m0 + i, k + j) and B(k + j, n0 + i); the result acc[r] is C(m0 + 4 j + r, n0 + i).
// Two accumulators take alternate k steps, halving the chain of dependent MFMAs.
__device__ __forceinline__ f4 mm16(const Mat& A, const Mat& B, int m0, int n0, int K, int i,
                                   int j, f4 acc) {
  f4 acc2{0.f, 0.f, 0.f, 0.f};
  int k = 0;
#pragma unroll 2
  for (; k + 8 <= K; k += 8) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.at(m0 + i, k + j), B.at(k + j, n0 + i), acc,
                                               0, 0, 0);
    acc2 = __builtin_amdgcn_mfma_f32_16x16x4f32(A.at(m0 + i, k + 4 + j), B.at(k + 4 + j, n0 + i),
                                                acc2, 0, 0, 0);
  }
  if (k < K)
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.at(m0 + i, k + j), B.at(k + j, n0 + i), acc,
                                               0, 0, 0);
  return acc + acc2;
}

struct Job {
  Mat A, B;
  int M, N, K;
  __device__ int tiles() const { return (M >> 4) * (N >> 4); }
};

// Runs up to four independent products; their 16 x 16 output tiles are dealt round-robin to
// the wavefronts. store(q, row, col, value) receives every element of product q once.
template <class Store>
__device__ __forceinline__ void run_jobs(const Job& j0, const Job& j1, const Job& j2,
                                         const Job& j3, int nj, Store&& store) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int i = lane & 15, j = lane >> 4;
  const int t0 = j0.tiles(), t1 = nj > 1 ? j1.tiles() : 0, t2 = nj > 2 ? j2.tiles() : 0,
            t3 = nj > 3 ? j3.tiles() : 0;
  const int total = t0 + t1 + t2 + t3;
  for (int t = wave; t < total; t += nw) {
    // the job index is wave-uniform; each branch inlines its own tile loop so that no job
    // descriptor is indexed dynamically (which would spill them to scratch)
    auto tile = [&](const Job& jb, int q, int tt) {
      const int tn = jb.N >> 4;
      const int m0 = (tt / tn) << 4, n0 = (tt % tn) << 4;
      const f4 acc = mm16(jb.A, jb.B, m0, n0, jb.K, i, j, f4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
      for (int r = 0; r < 4; ++r) store(q, m0 + 4 * j + r, n0 + i, acc[r]);
    };
    if (t < t0)
      tile(j0, 0, t);
    else if (t < t0 + t1)
      tile(j1, 1, t - t0);
    else if (t < t0 + t1 + t2)
      tile(j2, 2, t - t0 - t1);
    else
      tile(j3, 3, t - t0 - t1 - t2);
  }
}
template <class Store>
__device__ __forceinline__ void run_job(const Job& j0, Store&& store) {
  run_jobs(j0, j0, j0, j0, 1, store);
}

__device__ __forceinline__ float wave_sum64(float v) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) v += __shfl_xor(v, off);
  return v;
}
__device__ __forceinline__ float wave_max64(float v) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

// One global -> LDS copy: dst[r][c] (row stride ld) = src[r * cols + c], rows x cols.
struct Ld {
  float* dst;
  int ld;
  const float* src;
  int rows, cols;
};
// Copies several blocks at once: each round issues every block's load for this thread before
// any LDS store, so the global latencies overlap instead of adding up.
template <int NL>
__device__ __forceinline__ void load_all(const Ld (&l)[NL]) {
  int n_max = 0;
#pragma unroll
  for (int q = 0; q < NL; ++q) n_max = max(n_max, l[q].rows * l[q].cols);
  for (int base = 0; base < n_max; base += blockDim.x) {
    const int idx = base + threadIdx.x;
    float v[NL];
#pragma unroll
    for (int q = 0; q < NL; ++q) v[q] = idx < l[q].rows * l[q].cols ? l[q].src[idx] : 0.f;
#pragma unroll
    for (int q = 0; q < NL; ++q)
      if (idx < l[q].rows * l[q].cols) l[q].dst[(idx / l[q].cols) * l[q].ld + idx % l[q].cols] = v[q];
  }
}

// LDS layout (in floats) of the forward and backward kernels, shared with the host.
struct TokLayout {
  int zs, q, k, v, S, W, total;                           // forward
  int gz, dzs, zms, dUs, ss, dsl, dq, dk, dv, dS;  // backward extras
};

__host__ __device__ inline TokLayout tok_layout(int kind, int G, int V, bool bwd) {
  const int VP = V + 1, GP = G + 1;
  const int gv = G * VP, vv = V * VP, gg = G * GP;
  TokLayout L{};
  int off = 0;
  auto take = [&](int n) {
    const int o = off;
    off += n;
    return o;
  };
  L.zs = take(gv);
  if (kind == 1) L.W = take(gg);              // A
  if (kind == 2) L.W = take(vv);              // W_c
  if (kind == 3) {
    L.W = take(3 * vv);                       // W_q, W_k, W_v
    L.q = take(gv);
    L.k = take(gv);
    L.v = take(gv);
    L.S = take(gg);                           // scores / probabilities
  }
  if (bwd) {
    L.gz = take(gv);
    L.dzs = take(gv);
    L.zms = take(gv);
    L.dUs = take(gv);
    L.ss = take(G);
    L.dsl = take(G);
    if (kind == 3) {
      L.dq = take(gv);
      L.dk = take(gv);
      L.dv = take(gv);
      L.dS = take(gg);
    }
  }
  L.total = off;
  return L;
}

// Forward: zmix = Mix(z) for one (b, h) per workgroup; P (attention) is written for the
// backward.
template <int KIND>
__global__ __launch_bounds__(kTokThreads) void k_tok_fwd(const float* z, float* zmix, float* P,
                                                        const float* A, const float* Wc,
                                                        const float* Wq, const float* Wk,
                                                        const float* Wv, float scale,
                                                        int a_per_head, int H, int G, int V) {
  extern __shared__ float lds[];
  const TokLayout L = tok_layout(KIND, G, V, false);
  const int VP = V + 1, GP = G + 1, GV = G * V;
  const int bh = blockIdx.x;
  float* zs = lds + L.zs;
  float* W = lds + L.W;
  float* out = zmix + (int64_t)bh * GV;
  if constexpr (KIND == 0) {
    for (int idx = threadIdx.x; idx < GV; idx += blockDim.x) out[idx] = z[(int64_t)bh * GV + idx];
    return;
  }
  const Ld lz{zs, VP, z + (int64_t)bh * GV, G, V};
  if constexpr (KIND == 1) {
    const Ld l[2] = {lz, {W, GP, A + (a_per_head ? (int64_t)(bh % H) * G * G : 0), G, G}};
    load_all(l);
  } else if constexpr (KIND == 2) {
    const Ld l[2] = {lz, {W, VP, Wc, V, V}};
    load_all(l);
  } else {
    const Ld l[4] = {lz, {W, VP, Wq, V, V}, {W + V * VP, VP, Wk, V, V},
                     {W + 2 * V * VP, VP, Wv, V, V}};
    load_all(l);
  }
  __syncthreads();
  auto to_out = [&](int, int r, int c, float val) { out[r * V + c] = val; };
  if constexpr (KIND == 1) {
    run_job(Job{mat(W, GP, 1), mat(zs, VP, 1), G, V, G}, to_out);
  } else if constexpr (KIND == 2) {
    run_job(Job{mat(zs, VP, 1), mat(W, VP, 1), G, V, V}, to_out);
  } else {
    float* q = lds + L.q;
    float* kk = lds + L.k;
    float* v = lds + L.v;
    float* S = lds + L.S;
    const Job jq{mat(zs, VP, 1), mat(W, VP, 1), G, V, V};
    const Job jk{mat(zs, VP, 1), mat(W + V * VP, VP, 1), G, V, V};
    const Job jv{mat(zs, VP, 1), mat(W + 2 * V * VP, VP, 1), G, V, V};
    run_jobs(jq, jk, jv, jv, 3, [&](int which, int r, int c, float val) {
      (which == 0 ? q : (which == 1 ? kk : v))[r * VP + c] = val;
    });
    __syncthreads();
    // scores S = scale q k^T
    run_job(Job{mat(q, VP, 1), mat(kk, 1, VP), G, G, V},
            [&](int, int r, int c, float val) { S[r * GP + c] = scale * val; });
    __syncthreads();
    {  // row softmax, one wavefront per row (G <= 64: one column per lane)
      const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
      float* Pb = P + (int64_t)bh * G * G;
      for (int g = wave; g < G; g += nw) {
        const float x = lane < G ? S[g * GP + lane] : -INFINITY;
        const float m = wave_max64(x);
        const float e = lane < G ? expf(x - m) : 0.f;
        const float l = wave_sum64(e);
        const float p = e / l;
        if (lane < G) {
          S[g * GP + lane] = p;
          Pb[g * G + lane] = p;
        }
      }
    }
    __syncthreads();
    run_job(Job{mat(S, GP, 1), mat(v, VP, 1), G, V, G}, to_out);
  }
}

// Backward for one (b, h) per workgroup: dz = Mix^T(dzm), the per-(b, h) parameter partial
// in partM, and (when s is given) dU, ds and the slot-mean shifts cen [2V + 1].
// With dzm_part given, dzm is not read: it is summed here over the chunks of pass A's
// partials [BH][chunks][G V] (chunk 0 first) and written to dzm_out.
template <int KIND>
__global__ __launch_bounds__(kTokThreads) void k_tok_bwd(
    const float* z, const float* s, const float* zmix, const float* P, const float* dzm,
    const float* dzm_part, int chunks, float* dzm_out, float* dz, float* dU, float* ds,
    float* cen, float* partM, const float* A, const float* Wc, const float* Wq, const float* Wk,
    const float* Wv, float scale, int a_per_head, int H, int G, int V, float eps) {
  extern __shared__ float lds[];
  const TokLayout L = tok_layout(KIND, G, V, true);
  const int VP = V + 1, GP = G + 1, GV = G * V, VV = V * V;
  const int bh = blockIdx.x;
  float* zs = lds + L.zs;
  float* W = lds + L.W;
  float* gz = lds + L.gz;
  float* dzs = lds + L.dzs;
  float* zms = lds + L.zms;
  float* dUs = lds + L.dUs;
  float* ss = lds + L.ss;
  float* dsl = lds + L.dsl;
  const int64_t tok = (int64_t)bh * GV;
  {
    // the token gradients (s given) also need zmix and s
    const int tg = s != nullptr ? 1 : 0;
    const int rg = dzm_part != nullptr ? 0 : 1;  // dzm comes from the partials instead
    const Ld lz{zs, VP, z + tok, G, V}, lg{gz, VP, rg ? dzm + tok : nullptr, G * rg, V};
    const Ld lm{zms, VP, tg ? zmix + tok : nullptr, G * tg, V};
    const Ld ls{ss, G, tg ? s + (int64_t)bh * G : nullptr, tg, G};
    if constexpr (KIND == 0) {
      const Ld l[4] = {lz, lg, lm, ls};
      load_all(l);
    } else if constexpr (KIND == 1) {
      const Ld l[5] = {lz, lg, lm, ls,
                       {W, GP, A + (a_per_head ? (int64_t)(bh % H) * G * G : 0), G, G}};
      load_all(l);
    } else if constexpr (KIND == 2) {
      const Ld l[5] = {lz, lg, lm, ls, {W, VP, Wc, V, V}};
      load_all(l);
    } else {
      const Ld l[8] = {lz, lg, lm, ls, {W, VP, Wq, V, V}, {W + V * VP, VP, Wk, V, V},
                       {W + 2 * V * VP, VP, Wv, V, V}, {lds + L.S, GP, P + (int64_t)bh * G * G, G, G}};
      load_all(l);
    }
  }
  if (dzm_part != nullptr) {
    const float* pp = dzm_part + (int64_t)bh * chunks * GV;
    for (int idx = threadIdx.x; idx < GV; idx += blockDim.x) {
      float acc = 0.f;
#pragma unroll 16
      for (int q = 0; q < chunks; ++q) acc += pp[(int64_t)q * GV + idx];
      gz[(idx / V) * VP + idx % V] = acc;
      dzm_out[tok + idx] = acc;
    }
  }
  __syncthreads();
  float* dzb = dz + tok;
  auto to_dz = [&](int r, int c, float val) {
    dzs[r * VP + c] = val;
    dzb[r * V + c] = val;
  };
  if constexpr (KIND == 0) {
    for (int idx = threadIdx.x; idx < GV; idx += blockDim.x)
      to_dz(idx / V, idx % V, gz[(idx / V) * VP + idx % V]);
  } else if constexpr (KIND == 1) {
    // dz = A^T dzm;  dA_bh = dzm z^T
    float* pm = partM + (int64_t)bh * G * G;
    run_jobs(Job{mat(W, 1, GP), mat(gz, VP, 1), G, V, G},
             Job{mat(gz, VP, 1), mat(zs, 1, VP), G, G, V}, Job{}, Job{}, 2,
             [&](int q, int r, int c, float val) {
               if (q == 0)
                 to_dz(r, c, val);
               else
                 pm[r * G + c] = val;
             });
  } else if constexpr (KIND == 2) {
    // dz = dzm W_c^T;  dW_c,bh = z^T dzm
    float* pm = partM + (int64_t)bh * VV;
    run_jobs(Job{mat(gz, VP, 1), mat(W, 1, VP), G, V, V},
             Job{mat(zs, 1, VP), mat(gz, VP, 1), V, V, G}, Job{}, Job{}, 2,
             [&](int q, int r, int c, float val) {
               if (q == 0)
                 to_dz(r, c, val);
               else
                 pm[r * V + c] = val;
             });
  } else {
    float* q = lds + L.q;
    float* kk = lds + L.k;
    float* v = lds + L.v;
    float* Pm = lds + L.S;
    float* dS = lds + L.dS;
    float* dq = lds + L.dq;
    float* dk = lds + L.dk;
    float* dv = lds + L.dv;
    const Job jq{mat(zs, VP, 1), mat(W, VP, 1), G, V, V};
    const Job jk{mat(zs, VP, 1), mat(W + V * VP, VP, 1), G, V, V};
    const Job jv{mat(zs, VP, 1), mat(W + 2 * V * VP, VP, 1), G, V, V};
    run_jobs(jq, jk, jv, jv, 3, [&](int which, int r, int c, float val) {
      (which == 0 ? q : (which == 1 ? kk : v))[r * VP + c] = val;
    });
    __syncthreads();
    // dP = dzm v^T
    run_job(Job{mat(gz, VP, 1), mat(v, 1, VP), G, G, V},
            [&](int, int r, int c, float val) { dS[r * GP + c] = val; });
    __syncthreads();
    {  // dS = P (dP - sum_u P dP), one wavefront per row
      const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
      for (int g = wave; g < G; g += nw) {
        const float p = lane < G ? Pm[g * GP + lane] : 0.f;
        const float d = lane < G ? dS[g * GP + lane] : 0.f;
        const float r = wave_sum64(p * d);
        if (lane < G) dS[g * GP + lane] = p * (d - r);
      }
    }
    __syncthreads();
    // dq = scale dS k;  dk = scale dS^T q;  dv = P^T dzm
    run_jobs(Job{mat(dS, GP, 1), mat(kk, VP, 1), G, V, G},
             Job{mat(dS, 1, GP), mat(q, VP, 1), G, V, G},
             Job{mat(Pm, 1, GP), mat(gz, VP, 1), G, V, G}, Job{}, 3,
             [&](int which, int r, int c, float val) {
               if (which == 0)
                 dq[r * VP + c] = scale * val;
               else if (which == 1)
                 dk[r * VP + c] = scale * val;
               else
                 dv[r * VP + c] = val;
             });
    __syncthreads();
    // dz = dq W_q^T + dk W_k^T + dv W_v^T (one accumulator per tile); the three parameter
    // partials dW_x,bh = z^T dx go to partM [3][V][V]
    {
      const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
      const int i = lane & 15, j = lane >> 4;
      const int tz = (G >> 4) * (V >> 4), tw = (V >> 4) * (V >> 4);
      float* pm = partM + (int64_t)bh * 3 * VV;
      for (int t = wave; t < tz + 3 * tw; t += nw) {
        f4 acc{0.f, 0.f, 0.f, 0.f};
        if (t < tz) {
          const int m0 = (t / (V >> 4)) << 4, n0 = (t % (V >> 4)) << 4;
          // three independent chains, added at the end
          acc = mm16(mat(dq, VP, 1), mat(W, 1, VP), m0, n0, V, i, j, acc) +
                mm16(mat(dk, VP, 1), mat(W + V * VP, 1, VP), m0, n0, V, i, j,
                     f4{0.f, 0.f, 0.f, 0.f}) +
                mm16(mat(dv, VP, 1), mat(W + 2 * V * VP, 1, VP), m0, n0, V, i, j,
                     f4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
          for (int r = 0; r < 4; ++r) to_dz(m0 + 4 * j + r, n0 + i, acc[r]);
        } else {
          const int which = (t - tz) / tw, tt = (t - tz) % tw;
          const int m0 = (tt / (V >> 4)) << 4, n0 = (tt % (V >> 4)) << 4;
          const float* d = which == 0 ? dq : (which == 1 ? dk : dv);
          acc = mm16(mat(zs, 1, VP), mat(d, VP, 1), m0, n0, G, i, j, acc);
#pragma unroll
          for (int r = 0; r < 4; ++r) pm[which * VV + (m0 + 4 * j + r) * V + n0 + i] = acc[r];
        }
      }
    }
  }
  if (s == nullptr) return;
  __syncthreads();
  // token gradients: dU = dz / (s + eps); ds = -sum_v dz z / (s + eps)
  float* dUb = dU + tok;
  for (int idx = threadIdx.x; idx < GV; idx += blockDim.x) {
    const int g = idx / V, c = idx % V;
    const float u = dzs[g * VP + c] / (ss[g] + eps);
    dUs[g * VP + c] = u;
    dUb[idx] = u;
  }
  __shared__ float tot_s;
  {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    for (int g = wave; g < G; g += nw) {
      const float t = lane < V ? dzs[g * VP + lane] * zs[g * VP + lane] : 0.f;
      const float acc = wave_sum64(t);
      if (lane == 0) {
        const float d = -acc / (ss[g] + eps);
        dsl[g] = d;
        ds[(int64_t)bh * G + g] = d;
      }
    }
    if (wave == nw - 1) {  // total slot mass, fixed order
      float t = 0.f;
      for (int g = lane; g < G; g += 64) t += ss[g];
      t = wave_sum64(t);
      if (lane == 0) tot_s = t;
    }
  }
  __syncthreads();
  // shifts: cen = [sum_g m_g zmix[g][:], sum_g m_g dU[g][:], sum_g m_g ds[g]], m_g = s_g / sum s;
  // each column is summed by 16 threads over interleaved slots, then over those threads
  const float inv = tot_s > 0.f ? 1.0f / tot_s : 0.f;
  float* cb = cen + (int64_t)bh * (2 * V + 1);
  const int ncol = 2 * V + 1;
  for (int base = 0; base < ncol * 16; base += blockDim.x) {
    const int idx = base + threadIdx.x;
    const int c = idx >> 4, part = idx & 15;
    float acc = 0.f;
    if (c < ncol) {
      if (c < V) {
        for (int g = part; g < G; g += 16) acc += ss[g] * zms[g * VP + c];
      } else if (c < 2 * V) {
        for (int g = part; g < G; g += 16) acc += ss[g] * dUs[g * VP + (c - V)];
      } else {
        for (int g = part; g < G; g += 16) acc += ss[g] * dsl[g];
      }
    }
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, 16);
    if (c < ncol && part == 0) cb[c] = acc * inv;
  }
}

template <typename K>
hipError_t allow(K kernel, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

size_t tok_bytes(int kind, const Geom& g, bool bwd) {
  return sizeof(float) * (size_t)tok_layout(kind, g.G, g.V, bwd).total;
}

}  // namespace

bool tok_fused(const Geom& g, int kind) {
  if (kind == 3 && g.G > 64) return false;  // softmax rows: one column per lane
  return tok_bytes(kind, g, true) <= kTokLdsMax;
}

hipError_t launch_tok_fwd(const Geom& g, const MixArgs& m, const float* z, float* zmix,
                          float* attn, hipStream_t st) {
  const size_t lds = tok_bytes(m.kind, g, false);
  const dim3 grid(g.BH()), block(kTokThreads);
  const int aph = m.a_per_head ? 1 : 0;
#define FS_TOK_FWD(K)                                                                          \
  {                                                                                            \
    hipError_t e = allow(k_tok_fwd<K>, lds);                                                   \
    if (e != hipSuccess) return e;                                                             \
    hipLaunchKernelGGL(k_tok_fwd<K>, grid, block, lds, st, z, zmix, attn, m.A, m.Wc, m.Wq,     \
                       m.Wk, m.Wv, m.scale, aph, g.H, g.G, g.V);                               \
    return hipGetLastError();                                                                  \
  }
  switch (m.kind) {
    case 0: FS_TOK_FWD(0)
    case 1: FS_TOK_FWD(1)
    case 2: FS_TOK_FWD(2)
    case 3: FS_TOK_FWD(3)
    default: return hipErrorInvalidValue;
  }
#undef FS_TOK_FWD
}

static hipError_t tok_bwd(const Geom& g, const MixArgs& m, const float* z, const float* s,
                          const float* zmix, const float* attn, const float* dzm,
                          const float* dzm_part, int chunks, float* dzm_out, float* dz, float* dU,
                          float* ds, float* cen, float* partM, hipStream_t st) {
  const size_t lds = tok_bytes(m.kind, g, true);
  const dim3 grid(g.BH()), block(kTokThreads);
  const int aph = m.a_per_head ? 1 : 0;
#define FS_TOK_BWD(K)                                                                          \
  {                                                                                            \
    hipError_t e = allow(k_tok_bwd<K>, lds);                                                   \
    if (e != hipSuccess) return e;                                                             \
    hipLaunchKernelGGL(k_tok_bwd<K>, grid, block, lds, st, z, s, zmix, attn, dzm, dzm_part,    \
                       chunks, dzm_out, dz, dU, ds, cen, partM, m.A, m.Wc, m.Wq, m.Wk, m.Wv,   \
                       m.scale, aph, g.H, g.G, g.V, g.eps);                                    \
    return hipGetLastError();                                                                  \
  }
  switch (m.kind) {
    case 0: FS_TOK_BWD(0)
    case 1: FS_TOK_BWD(1)
    case 2: FS_TOK_BWD(2)
    case 3: FS_TOK_BWD(3)
    default: return hipErrorInvalidValue;
  }
#undef FS_TOK_BWD
}

hipError_t launch_tok_bwd(const Geom& g, const MixArgs& m, const float* z, const float* s,
                          const float* zmix, const float* attn, const float* dzm, float* dz,
                          float* dU, float* ds, float* cen, float* partM, hipStream_t st) {
  return tok_bwd(g, m, z, s, zmix, attn, dzm, nullptr, 0, nullptr, dz, dU, ds, cen, partM, st);
}

hipError_t launch_tok_bwd_from_parts(const Geom& g, const MixArgs& m, const float* z,
                                     const float* s, const float* zmix, const float* attn,
                                     const float* dzm_part, int chunks, float* dzm_out,
                                     float* dz, float* dU, float* ds, float* cen, float* partM,
                                     hipStream_t st) {
  return tok_bwd(g, m, z, s, zmix, attn, nullptr, dzm_part, chunks, dzm_out, dz, dU, ds, cen,
                 partM, st);
}

}  // namespace fs
