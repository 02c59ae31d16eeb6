// Internal interface between the C-ABI host layer (fs_api.cpp) and the HIP kernels
// (fs_kernels.hip). Not installed; no torch types anywhere.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace fs {

// Problem geometry after validation.
struct Geom {
  int64_t B, N;
  int H, D, V, G;
  bool bf16;
  float eps;
  bool ws_per_head;
  int BH() const { return (int)(B * H); }
};

enum Pass { PASS_SLICE = 0, PASS_DESLICE = 1, PASS_BWD_A = 2, PASS_BWD_B = 3 };

// Launch shape of one streaming pass over the points.
//   GS: slots owned by one wavefront; NS = G / GS wavefronts share each point tile;
//   NP: independent point groups per workgroup; a workgroup has NS * NP wavefronts.
//   chunks: workgroups per (sample, head) along the points, each covering chunk_pts points.
struct PassCfg {
  int GS, NS, NP;
  int PB;  // 16-point blocks per wavefront tile
  int chunks;
  int64_t chunk_pts;
};

PassCfg pick_cfg(const Geom& g, Pass pass);

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

// One streaming pass over the points with the tiling pick_cfg chooses (fs_pass_*.hip).
hipError_t run_pass_slice(const Geom& g, const PassArgs& a, hipStream_t st);
hipError_t run_pass_deslice(const Geom& g, const PassArgs& a, hipStream_t st);
hipError_t run_pass_bwd_a(const Geom& g, const PassArgs& a, hipStream_t st);
hipError_t run_pass_bwd_b(const Geom& g, const PassArgs& a, hipStream_t st);

// Per-thread measurement events recorded around the streaming passes (fs_set_pass_events).
struct PassEvents {
  hipEvent_t before[4] = {nullptr, nullptr, nullptr, nullptr};
  hipEvent_t after[4] = {nullptr, nullptr, nullptr, nullptr};
};
PassEvents& pass_events();

// Workspace carve-up (byte offsets, 256-byte aligned).
struct FwdWs {
  size_t partU, partS, total;
};
struct BwdWs {
  size_t partDZ, dzm, dz, dU, ds, cen, partP, partM, scr, total;
};
FwdWs fwd_ws_layout(const Geom& g);
BwdWs bwd_ws_layout(const Geom& g, int mix_kind);
size_t mix_param_count(const Geom& g, int mix_kind, bool a_per_head);

struct MixArgs {
  int kind;
  bool a_per_head;
  const float* A;
  const float* Wc;
  const float* Wq;
  const float* Wk;
  const float* Wv;
  float scale;
};

// Launchers; each returns the hipError_t of its launches.
hipError_t launch_slice(const Geom& g, const void* x, const void* fx, const float* Ws,
                        const float* bias, const float* tau, float* z, float* s, float* lse,
                        float* partU, float* partS, hipStream_t st);
hipError_t launch_deslice(const Geom& g, const void* x, const float* Ws, const float* bias,
                          const float* tau, const float* zmix, const float* lse, void* out,
                          hipStream_t st);
hipError_t launch_mix(const Geom& g, const MixArgs& m, const float* z, float* zmix,
                      float* attn, hipStream_t st);
// dz = Mix^T(dzm); with s given also dU = dz / (s + eps), ds and the slot-mean shifts cen
// [BH][2V + 1]; per-(b,h) parameter partials into partM, reduced into dmix (nullable) here
// when reduce_params, else left for launch_reduce_params. scr: attention scratch
// [BH][3 G V + G G].
hipError_t launch_mix_bwd(const Geom& g, const MixArgs& m, const float* z, const float* s,
                          const float* zmix, const float* attn, const float* dzm, float* dz,
                          float* dU, float* ds, float* cen, float* scr, float* partM,
                          float* dmix, bool reduce_params, hipStream_t st);
// Single-workgroup-per-(b, h) token mix kernels with every operand in LDS (fs_tokmix.hip);
// tok_fused tells whether they apply to this problem and mix kind.
bool tok_fused(const Geom& g, int mix_kind);
hipError_t launch_tok_fwd(const Geom& g, const MixArgs& m, const float* z, float* zmix,
                          float* attn, hipStream_t st);
hipError_t launch_tok_bwd(const Geom& g, const MixArgs& m, const float* z, const float* s,
                          const float* zmix, const float* attn, const float* dzm, float* dz,
                          float* dU, float* ds, float* cen, float* partM, hipStream_t st);
// Fixed-order reductions of per-workgroup partials (fs_tokens.hip).
hipError_t launch_reduce_tokens(const Geom& g, const float* partU, const float* partS,
                                int chunks, float* z, float* s, hipStream_t st);
hipError_t launch_reduce_rows(const Geom& g, const float* part, float* out, int chunks,
                              int64_t len, hipStream_t st);
// dW_s, dbias, dtau from the pass-B partials; with m and dmix given, also the mix-parameter
// gradient from partM (same launch).
hipError_t launch_reduce_params(const Geom& g, const float* part, float* dWs, float* dbias,
                                float* dtau, int chunks, const MixArgs* m, const float* partM,
                                float* dmix, hipStream_t st);
hipError_t launch_bwd(const Geom& g, const MixArgs& m, const void* x, const void* fx,
                      const float* Ws, const float* bias, const float* tau, const float* z,
                      const float* s, const float* zmix, const float* attn, const float* lse,
                      const void* dout, void* dx, void* dfx, float* dWs, float* dbias,
                      float* dtau, float* dmix, float* dzm_out, char* ws, hipStream_t st);

}  // namespace fs
