// Launchers of the fused slice -> token mix -> deslice path: each streaming pass (one kernel
// per pass, in fs_pass_*.hip) optionally bracketed by the caller's measurement events, the
// forward slice with its token reduction, the deslice, and the backward sequence
// pass A -> reduce -> mix backward -> pass B -> parameter reductions.

#include <hip/hip_runtime.h>

#include "fs_internal.h"

namespace fs {
namespace {

// Launch one streaming pass, bracketed by the caller's measurement events if requested.
template <int PASS>
hipError_t run_pass(const Geom& g, const PassArgs& a, hipStream_t st) {
  const PassEvents& ev = pass_events();
  if (ev.before[PASS] != nullptr) {
    hipError_t e = hipEventRecord(ev.before[PASS], st);
    if (e != hipSuccess) return e;
  }
  hipError_t e = PASS == PASS_SLICE     ? run_pass_slice(g, a, st)
                 : PASS == PASS_DESLICE ? run_pass_deslice(g, a, st)
                 : PASS == PASS_BWD_A   ? run_pass_bwd_a(g, a, st)
                                        : run_pass_bwd_b(g, a, st);
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
                     reinterpret_cast<float*>(ws + L.scr), partM, dmix, false, st);
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
  e = launch_reduce_params(g, partP, dWs, dbias, dtau, b.chunks, &m, partM, dmix, st);
  return e;
}

}  // namespace fs
