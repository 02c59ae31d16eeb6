// Launchers of the fused slice -> token mix -> deslice path: each streaming pass (one kernel
// per pass, in fs_pass_*.hip) optionally bracketed by the caller's measurement events, the
// forward slice with its token reduction, the deslice, and the backward sequence
// pass A -> reduce -> mix backward -> pass B -> parameter reductions.

#include <hip/hip_runtime.h>

#include "fs_internal.h"

namespace fs {
namespace {

// Launch the kernels of one logical streaming pass (f), bracketed by the caller's measurement
// events if requested.
template <class F>
hipError_t timed(int pass, hipStream_t st, F&& f) {
  const PassEvents& ev = pass_events();
  if (ev.before[pass] != nullptr) {
    hipError_t e = hipEventRecord(ev.before[pass], st);
    if (e != hipSuccess) return e;
  }
  hipError_t e = f();
  if (e == hipSuccess && ev.after[pass] != nullptr) e = hipEventRecord(ev.after[pass], st);
  return e;
}

PassArgs base_args(const Geom& g, Pass p, int np = 0) {
  PassArgs a{};
  const PassCfg cfg = pick_cfg(g, p, np);
  a.N = g.N;
  a.H = g.H;
  a.G = g.G;
  a.ws_per_head = g.ws_per_head ? 1 : 0;
  a.nblk = cfg.nblk;
  a.chunks = cfg.chunks;
  a.chunk_pts = cfg.chunk_pts;
  a.nsub = cfg.nsub;
  a.sub_pts = cfg.sub_pts;
  // slots the tiling covers: GS per slot wave, NS waves, nblk blocks (the point-owned passes
  // sweep blocks of 64)
  const int covered = p == PASS_POINT ? 64 * ((g.G + 63) / 64) : cfg.GS * cfg.NS * cfg.nblk;
  a.padded = covered != g.G ? 1 : 0;
  return a;
}

inline hipError_t first_err(hipError_t a, hipError_t b) { return a != hipSuccess ? a : b; }

}  // namespace

// =======================================================================================
// Launchers
// =======================================================================================
hipError_t launch_slice(const Geom& g, const void* x, const void* fx, const float* Ws,
                        const float* bias, const float* tau, float* z, float* s, float* lse,
                        char* ws, hipStream_t st) {
  const FwdWs L = fwd_ws_layout(g);
  float* partU = reinterpret_cast<float*>(ws + L.partU);
  float* partS = reinterpret_cast<float*>(ws + L.partS);
  PassArgs a = base_args(g, PASS_SLICE);
  a.x = x;
  a.fx = fx;
  a.Ws = Ws;
  a.bias = bias;
  a.tau = tau;
  a.part = partU;
  a.part2 = partS;
  hipError_t e;
  if (blocked(g)) {
    // statistics pass (lse), then the slot-owned slice reading it
    PassArgs sa = base_args(g, FS_STATS_POINT ? PASS_POINT : PASS_STATS);
    sa.x = x;
    sa.Ws = Ws;
    sa.bias = bias;
    sa.tau = tau;
    sa.lse_out = lse != nullptr ? lse : reinterpret_cast<float*>(ws + L.lse);
    a.lse_in = sa.lse_out;
    e = timed(PASS_SLICE, st, [&] {
      hipError_t e1 = g.D > 32 ? run_pass_stats_stream(g, sa, ws + L.simg, st)
                               : FS_STATS_POINT ? run_pass_stats_pt(g, sa, st)
                                                : run_pass_stats(g, sa, st);
      return e1 != hipSuccess ? e1 : run_pass_slice_blk(g, a, st);
    });
  } else {
    a.lse_out = lse;
    e = timed(PASS_SLICE, st, [&] { return run_pass_slice(g, a, st); });
  }
  if (e != hipSuccess) return e;
  return launch_reduce_tokens(g, partU, partS, a.chunks, z, s, st);
}

hipError_t launch_linearno_slice(const Geom& g, const void* x, const void* fx, const float* Ws,
                                 const float* bias, const float* tau, float* z, float* clse,
                                 char* ws, hipStream_t st) {
  const FwdWs L = linearno_fwd_ws_layout(g);
  float* partU = reinterpret_cast<float*>(ws + L.partU);
  float* partML = reinterpret_cast<float*>(ws + L.partS);
  PassArgs a = base_args(g, PASS_SLICE);
  a.x = x;
  a.fx = fx;
  a.Ws = Ws;
  a.bias = bias;
  a.tau = tau;
  a.part = partU;
  a.part2 = partML;
  hipError_t e = timed(PASS_SLICE, st, [&] { return run_pass_slice_col(g, a, st); });
  if (e != hipSuccess) return e;
  return launch_reduce_col(g, partU, partML, a.chunks, z, clse, st);
}

hipError_t launch_deslice(const Geom& g, const void* x, const float* Ws, const float* bias,
                          const float* tau, const float* zmix, const float* lse, float* lse_out,
                          void* out, hipStream_t st) {
  const bool pt = deslice_point_owned(g);
  PassArgs a = base_args(g, pt ? PASS_POINT : PASS_DESLICE, pt ? deslice_pt_waves(g) : 0);
  a.x = x;
  a.Ws = Ws;
  a.bias = bias;
  a.tau = tau;
  a.zmix = zmix;
  a.lse_in = lse;      // null: the deslice computes the softmax statistics itself
  a.lse_out = lse_out;  // with lse null only; nullable
  a.out = out;
  return timed(PASS_DESLICE, st, [&] { return run_pass_deslice(g, a, st); });
}

hipError_t launch_bwd(const Geom& g, const MixArgs& m, const void* x, const void* fx,
                      const float* Ws, const float* bias, const float* tau, const float* z,
                      const float* s, const float* zmix, const float* attn, const float* lse,
                      const void* dout, void* dx, void* dfx, float* dWs, float* dbias,
                      float* dtau, float* dmix, float* dzm_out, char* ws, hipStream_t st,
                      const UntiedArgs* u, const float* clse) {
  const BwdWs L = bwd_ws_layout(g, m.kind);
  float* partDZ = reinterpret_cast<float*>(ws + L.partDZ);
  float* dzm = dzm_out != nullptr ? dzm_out : reinterpret_cast<float*>(ws + L.dzm);
  float* dz = reinterpret_cast<float*>(ws + L.dz);
  float* dU = reinterpret_cast<float*>(ws + L.dU);
  float* dsv = reinterpret_cast<float*>(ws + L.ds);
  float* partP = reinterpret_cast<float*>(ws + L.partP);
  float* partM = reinterpret_cast<float*>(ws + L.partM);
  // pass A: dzmix = w^T dout (the deslice weights)
  PassArgs a = base_args(g, PASS_BWD_A);
  a.x = x;
  a.dout = dout;
  a.Ws = u ? u->Wd : Ws;
  a.bias = u ? u->bd : bias;
  a.tau = u ? u->taud : tau;
  a.lse_in = u ? u->lse_d : lse;
  a.part = partDZ;
  hipError_t e = timed(PASS_BWD_A, st, [&] { return run_pass_bwd_a(g, a, st); });
  if (e != hipSuccess) return e;
  // the single-workgroup token kernels sum pass A's partials themselves; the other mixes
  // get dzmix from the reduction kernel first
  const bool fused_red = tok_fused(g, m.kind);
  if (!fused_red) {
    e = launch_reduce_rows(g, partDZ, dzm, a.chunks, (int64_t)g.G * g.V, st);
    if (e != hipSuccess) return e;
  }
  // mix backward: dz, dU, ds, the slot-mean shifts (+ parameter gradients)
  float* cen = reinterpret_cast<float*>(ws + L.cen);
  Geom gm = g;
  const float* sm = s;
  if (clse != nullptr) {
    // LinearNO: the tokens carry no weight-sum normalisation, so dU = dz and
    // ds = -sum_v dz z (the token gradients with unit weight sums and no eps)
    float* ones = reinterpret_cast<float*>(ws + L.ones);
    e = launch_fill(ones, 1.0f, (int64_t)g.BH() * g.G, st);
    if (e != hipSuccess) return e;
    gm.eps = 0.f;
    sm = ones;
  }
  if (fused_red)
    e = launch_tok_bwd_from_parts(gm, m, z, sm, zmix, attn, partDZ, a.chunks, dzm, dz, dU, dsv,
                                  cen, partM, st);
  else
    e = launch_mix_bwd(gm, m, z, sm, zmix, attn, dzm, dz, dU, dsv, cen,
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
  // slot-blocked family: the point-owned pass (dx, dfx, per-point c and tb) with the operand
  // images of one weight set, ahead of its slot-owned parameter pass
  float* cpt = reinterpret_cast<float*>(ws + L.cpt);
  auto point_args = [&](const PassArgs& w) {
    PassArgs pa = base_args(g, PASS_POINT);
    pa.x = x;
    pa.fx = fx;
    pa.dout = dout;
    pa.out = dx;
    pa.out2 = dfx;
    pa.Ws = w.Ws;
    pa.bias = w.bias;
    pa.tau = w.tau;
    pa.zmix = zmix;
    pa.dU = dU;
    pa.ds = dsv;
    pa.cen = cen;
    pa.lse_in = w.lse_in;
    pa.clse = w.clse;
    pa.cpt_out = cpt;
    pa.img = ws + L.img;
    return pa;
  };
  if (u != nullptr) {
    // untied: the slice weights' part writes dx and dfx; the deslice weights' part (own
    // projection, bias, temperature and normaliser) adds its dx contribution
    PassArgs b2 = b;
    b2.Ws = u->Wd;
    b2.bias = u->bd;
    b2.tau = u->taud;
    b2.lse_in = u->lse_d;
    b2.part = reinterpret_cast<float*>(ws + L.partP2);
    b.clse = clse;
    const int role1 = clse != nullptr ? 3 : 1;
    if (blocked(g)) {
      // each weight set: point-owned pass, then its parameter pass (they share the images
      // and the per-point (c, tb) buffer, in stream order)
      const PassArgs p1 = point_args(b), p2 = point_args(b2);
      b.cpt = b2.cpt = cpt;
      e = timed(PASS_BWD_B, st, [&] {
        hipError_t e1 = run_pass_point(g, p1, role1, st);
        if (e1 == hipSuccess) e1 = run_pass_bwd_params(g, b, role1, st);
        if (e1 == hipSuccess) e1 = run_pass_point(g, p2, 2, st);
        return e1 != hipSuccess ? e1 : run_pass_bwd_params(g, b2, 2, st);
      });
    } else if (fused_untied_bwd_b(g)) {
      // both weight sets per tile in one kernel: X read once, dx written once
      b.Wd = u->Wd;
      b.bd = u->bd;
      b.taud = u->taud;
      b.lse_d = u->lse_d;
      b.part_d = b2.part;
      e = timed(PASS_BWD_B, st, [&] { return run_pass_bwd_b2(g, b, clse != nullptr, st); });
    } else {
      e = timed(PASS_BWD_B, st, [&] {
        hipError_t e1 = run_pass_bwd_b_untied(g, b, role1, st);
        return e1 != hipSuccess ? e1 : run_pass_bwd_b_untied(g, b2, 2, st);
      });
    }
    if (e != hipSuccess) return e;
    e = launch_reduce_params(g, partP, dWs, dbias, dtau, b.chunks, b.nblk, &m, partM, dmix, st);
    if (e != hipSuccess) return e;
    return launch_reduce_params(g, b2.part, u->dWd, u->dbd, u->dtaud, b.chunks, b.nblk, nullptr,
                                nullptr, nullptr, st);
  }
  if (blocked(g)) {
    // point-owned pass (dx, dfx, per-point c and tb), then the slot-owned parameter pass
    const PassArgs pa = point_args(b);
    b.cpt = cpt;
    e = timed(PASS_BWD_B, st, [&] {
      hipError_t e1 = run_pass_point(g, pa, 0, st);
      return e1 != hipSuccess ? e1 : run_pass_bwd_params(g, b, 0, st);
    });
  } else {
    e = timed(PASS_BWD_B, st, [&] { return run_pass_bwd_b(g, b, st); });
  }
  if (e != hipSuccess) return e;
  e = launch_reduce_params(g, partP, dWs, dbias, dtau, b.chunks, b.nblk, &m, partM, dmix, st);
  return e;
}

}  // namespace fs
