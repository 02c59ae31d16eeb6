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
  bool untied = false;    // backward of the untied variant (separate deslice projection)
  bool linearno = false;  // LinearNO: untied, slice weights normalised over the points
  int BH() const { return (int)(B * H); }
};

// The four streaming passes (also the ids of fs_set_pass_events), and the two extra kernels
// of the slot-blocked family used for large G: a statistics pass ahead of the slice and a
// point-owned pass ahead of the backward pass B.
enum Pass {
  PASS_SLICE = 0,
  PASS_DESLICE = 1,
  PASS_BWD_A = 2,
  PASS_BWD_B = 3,
  PASS_STATS = 4,
  PASS_POINT = 5
};

// Slot-blocked family (large G): the slice, backward pass A and the parameter half of
// backward pass B run slot-owned (a workgroup owns one block of 64 slots and streams its
// chunk of points), with the per-point softmax statistics from a statistics pass and the
// per-point correction c = sum_g w dw from a point-owned pass that also writes dx and dfx
// (once per weight set for the untied variant and LinearNO). Head widths up to 32. Below the
// threshold every pass is one kernel whose wavefronts split the slots of a tile.
bool blocked(const Geom& g);
// The slot-blocked family's deslice: point-owned with streamed slot blocks (1), or the
// cooperative kernel with one slot wave per 64 slots (0).
#ifndef FS_DESLICE_POINT
#define FS_DESLICE_POINT 1
#endif
// Above this slot count (bf16 N = 2^18: G = 512 deslice 497 -> 300 us, G = 1024 859 -> 544 us;
// at G = 256 the four-wave cooperative kernel is faster, 151 against 176 us).
#ifndef FS_DESLICE_POINT_MIN_G
#define FS_DESLICE_POINT_MIN_G 256
#endif
// Whether the deslice runs point-owned (its launch arguments then take the chunking of
// PASS_POINT, not PASS_DESLICE).
inline bool deslice_point_owned(const Geom& g) {
  return FS_DESLICE_POINT && blocked(g) && g.G > FS_DESLICE_POINT_MIN_G;
}
// Wavefronts per workgroup of the point-owned deslice at head width up to 32 (16 measured 3%
// faster than 12 and 8 at G = 512 and 1024).
#ifndef FS_DESLICE_PT_WAVES
#define FS_DESLICE_PT_WAVES 16
#endif
// Wavefronts per workgroup of the point-owned pass, and the range of resident wavefronts per
// SIMD it is compiled for (the minimum caps its registers). Twelve wavefronts with three per
// SIMD (a few registers spilled) measured 5-8% faster than eight with two; six and four
// were slower.
#ifndef FS_POINT_WAVES
#define FS_POINT_WAVES 12
#endif
// Wavefronts per workgroup of the point-owned passes at head width 64 (one per SIMD: their
// register footprint is about twice that of head width 32).
#ifndef FS_POINT_WAVES_WIDE
#define FS_POINT_WAVES_WIDE 4
#endif
inline int deslice_pt_waves(const Geom& g) { return g.D > 32 ? FS_POINT_WAVES_WIDE : FS_DESLICE_PT_WAVES; }
#ifndef FS_POINT_WPE
#define FS_POINT_WPE 3
#endif
// The statistics pass of the slot-blocked family: point-owned (1) or cooperative (0).
#ifndef FS_STATS_POINT
#define FS_STATS_POINT 1
#endif
#ifndef FS_POINT_WPE_MIN
#define FS_POINT_WPE_MIN 3
#endif

// Launch shape of one streaming pass over the points.
//   GS: slots owned by one wavefront; NS = G / GS wavefronts share each point tile
//   (1 in the slot-owned passes of the blocked family);
//   NP: independent point groups per workgroup; a workgroup has NS * NP wavefronts.
//   nblk: slot blocks of GS slots in the grid (blocked slot-owned passes), else 1.
//   chunks: workgroups per (sample, head[, slot block]) along the points, each covering
//   chunk_pts points.
struct PassCfg {
  int GS, NS, NP;
  int PB;  // 16-point blocks per wavefront tile
  int nblk;
  int chunks;
  int64_t chunk_pts;
  // On long streams a chunk is a set of sub-chunks of sub_pts points, sub-chunks c, c + chunks,
  // c + 2 chunks, ... of the nsub along the points (nsub = chunks, sub_pts = chunk_pts
  // otherwise): a pass with per-chunk partials keeps its partial count while its workgroups
  // sweep the rows together.
  int64_t nsub, sub_pts;
};

// np > 0: the point group count of PASS_POINT's chunking (the point-owned kernels sweep a
// chunk in steps of 32 np points; a chunk that is a whole number of them leaves no wavefront
// idle in its last step)
PassCfg pick_cfg(const Geom& g, Pass pass, int np = 0);

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
  const float* clse;  // LinearNO: per-slot base-2 normaliser over the points, [BH][G]
  // the deslice's own weight set (untied, LinearNO) for the one-kernel backward pass B
  const float* Wd;
  const float* bd;
  const float* taud;
  const float* lse_d;
  float* part_d;
  float* lse_out;
  float* part;   // slice: U partials; bwd_a: dzmix partials; bwd_b: parameter partials
  float* part2;  // slice: s partials
  const void* img;   // point-owned pass: per-(b, h) operand images of the slot blocks
  const float* cpt;  // blocked bwd_b: per point (c, tb, lse2, 0) from the point-owned pass
  float* cpt_out;    // point-owned pass: per point (c, tb, lse2, 0), [BH][N][4]
  int64_t N;
  int H, G;
  int ws_per_head;
  int nblk;
  int chunks;
  int64_t chunk_pts;
  int64_t nsub, sub_pts;  // sub-chunks (see PassCfg)
  int padded;  // the tiling covers more slots than G: slots >= G are padding (masked)
};

// One streaming pass over the points with the tiling pick_cfg chooses (fs_pass_*.hip).
hipError_t run_pass_slice(const Geom& g, const PassArgs& a, hipStream_t st);
hipError_t run_pass_deslice(const Geom& g, const PassArgs& a, hipStream_t st);
hipError_t run_pass_bwd_a(const Geom& g, const PassArgs& a, hipStream_t st);
hipError_t run_pass_bwd_b(const Geom& g, const PassArgs& a, hipStream_t st);
// Slot-blocked family: statistics pass (lse only), slot-owned slice, point-owned backward pass
// (dx, dfx and per-point (c, tb)), slot-owned parameter half of backward pass B.
hipError_t run_pass_stats(const Geom& g, const PassArgs& a, hipStream_t st);
hipError_t run_pass_slice_blk(const Geom& g, const PassArgs& a, hipStream_t st);
// role: 0 tied; 1 / 2 the untied slice / deslice weights; 3 LinearNO's slice weights (the
// same roles as run_pass_bwd_b_untied).
hipError_t run_pass_point(const Geom& g, const PassArgs& a, int role, hipStream_t st);
// point-owned statistics pass of the slot-blocked family (lse only; chunks of PASS_POINT)
hipError_t run_pass_stats_pt(const Geom& g, const PassArgs& a, hipStream_t st);
size_t point_image_bytes(const Geom& g);  // workspace of the point-owned pass's operand images
// Head width 64: the statistics pass with its slot blocks' images streamed through LDS (built
// into img, stat_image_bytes of workspace, first).
size_t stat_image_bytes(const Geom& g);
hipError_t run_pass_stats_stream(const Geom& g, const PassArgs& a, void* img, hipStream_t st);
hipError_t run_pass_bwd_params(const Geom& g, const PassArgs& a, int role, hipStream_t st);
// Untied variant, backward pass B in two parts: role 1 the slice weights (writes dx, dfx),
// role 2 the deslice weights (adds to dx); each writes its own parameter partials.
hipError_t run_pass_bwd_b_untied(const Geom& g, const PassArgs& a, int role, hipStream_t st);
// Both weight sets of the untied variant (or LinearNO, coln) in one backward pass B kernel,
// when one wavefront covers the tile's slots (fused_untied_bwd_b).
bool fused_untied_bwd_b(const Geom& g);
hipError_t run_pass_bwd_b2(const Geom& g, const PassArgs& a, bool coln, hipStream_t st);
// LinearNO slice: per-(sample, head, chunk) partials U [G][V] and [G] maxima + [G] sums of
// 2^(a - max) over the chunk's points, merged by launch_reduce_col into z and clse.
hipError_t run_pass_slice_col(const Geom& g, const PassArgs& a, hipStream_t st);
hipError_t launch_reduce_col(const Geom& g, const float* partU, const float* partML, int chunks,
                             float* z, float* clse, hipStream_t st);
hipError_t launch_linearno_slice(const Geom& g, const void* x, const void* fx, const float* Ws,
                                 const float* bias, const float* tau, float* z, float* clse,
                                 char* ws, hipStream_t st);
// Static per-device scratch of fs_slice_fwd_noalloc (fs_noalloc.hip): its size, and the
// device address of `device`'s copy (looked up once per device, with that device current).
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
hipError_t static_scratch(int device, void** ptr);
// Fills n floats with v (workspace constants; a kernel, so it may be captured in a graph).
hipError_t launch_fill(float* p, float v, int64_t n, hipStream_t st);

// Per-thread measurement events recorded around the streaming passes (fs_set_pass_events).
struct PassEvents {
  hipEvent_t before[4] = {nullptr, nullptr, nullptr, nullptr};
  hipEvent_t after[4] = {nullptr, nullptr, nullptr, nullptr};
};
PassEvents& pass_events();

// Workspace carve-up (byte offsets, 256-byte aligned).
struct FwdWs {
  size_t partU, partS, lse, simg, total;  // lse: [BH][N] when the blocked family needs it;
                                          // simg: the streamed statistics pass's images
};
struct BwdWs {
  size_t partDZ, dzm, dz, dU, ds, cen, partP, partM, scr, cpt, img, partP2, ones, total;
};
// Floats of one parameter partial of backward pass B: [D G] dW_s, [G] dbias, then one fp64
// dtau partial per slot block.
inline int64_t param_partial_len(const Geom& g, int nblk) {
  return (int64_t)g.D * g.G + g.G + 2LL * nblk;
}
FwdWs fwd_ws_layout(const Geom& g);
// LinearNO slice: partU as in the forward, partS holding 2 G floats per chunk.
FwdWs linearno_fwd_ws_layout(const Geom& g);
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
                        char* ws, hipStream_t st);
hipError_t launch_deslice(const Geom& g, const void* x, const float* Ws, const float* bias,
                          const float* tau, const float* zmix, const float* lse, float* lse_out,
                          void* out, hipStream_t st);
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
// As launch_tok_bwd, but dzm is first summed from pass A's per-chunk partials
// [BH][chunks][G V] (fixed chunk order) inside the kernel and written to dzm_out.
hipError_t launch_tok_bwd_from_parts(const Geom& g, const MixArgs& m, const float* z,
                                     const float* s, const float* zmix, const float* attn,
                                     const float* dzm_part, int chunks, float* dzm_out,
                                     float* dz, float* dU, float* ds, float* cen, float* partM,
                                     hipStream_t st);
// Single-workgroup-per-(b, h) token mix kernels with every operand in LDS (fs_tokmix.hip);
// tok_fused tells whether they apply to this problem and mix kind.
bool tok_fused(const Geom& g, int mix_kind);
// Attention over token sets beyond the single-workgroup LDS kernels: the row-block forward
// (no workspace) and the backward as batched products.
bool attn_rows(const Geom& g, int mix_kind);
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
                                float* dtau, int chunks, int nblk, const MixArgs* m,
                                const float* partM, float* dmix, hipStream_t st);
// The deslice's own projection, bias, temperature and normaliser, and their gradients.
struct UntiedArgs {
  const float* Wd;
  const float* bd;
  const float* taud;
  const float* lse_d;
  float* dWd;
  float* dbd;
  float* dtaud;
};
// Backward of the path; with u given, of the untied variant (g.untied set); with clse also
// given, of LinearNO (g.linearno set; s is unused).
hipError_t launch_bwd(const Geom& g, const MixArgs& m, const void* x, const void* fx,
                      const float* Ws, const float* bias, const float* tau, const float* z,
                      const float* s, const float* zmix, const float* attn, const float* lse,
                      const void* dout, void* dx, void* dfx, float* dWs, float* dbias,
                      float* dtau, float* dmix, float* dzm_out, char* ws, hipStream_t st,
                      const UntiedArgs* u = nullptr, const float* clse = nullptr);

}  // namespace fs
