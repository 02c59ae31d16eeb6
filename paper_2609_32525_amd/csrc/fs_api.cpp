// C-ABI entry points of libflashslice: host-side validation, launch-shape selection,
// workspace carve-up and dispatch to the HIP kernels. Every check runs before anything is
// enqueued, and no HIP runtime call is made on an error path, so the whole validation layer
// also works on a machine without a GPU.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <initializer_list>

#include "../../include/flashslice.h"
#include "fs_internal.h"

namespace fs {

namespace {
thread_local int g_last_hip_error = 0;

constexpr size_t kAlign = 256;
constexpr int64_t kCUs = 256;  // MI355X compute units
size_t up(size_t v, size_t a = kAlign) { return (v + a - 1) / a * a; }

#ifndef FS_TARGET_PARTIAL
#define FS_TARGET_PARTIAL 512
#endif
#ifndef FS_BLOCKED_MIN_G
#define FS_BLOCKED_MIN_G 128
#endif
#ifndef FS_TARGET_DESLICE
#define FS_TARGET_DESLICE 512
#endif
#ifndef FS_PB_F32
#define FS_PB_F32 1
#endif
#ifndef FS_MIN_TILES
#define FS_MIN_TILES 4
#endif
#ifndef FS_TARGET_LONG
#define FS_TARGET_LONG 1024
#endif
// The slice on long streams: chunks made of strided sub-chunks of FS_MAX_TILES tiles (1).
#ifndef FS_SLICE_STRIDE
#define FS_SLICE_STRIDE 1
#endif
// Chunk counts rounded up to a multiple of 8 (1).
#ifndef FS_XCD_CHUNKS
#define FS_XCD_CHUNKS 1
#endif
// Most point tiles per chunk on long streams (0: no limit).
#ifndef FS_MAX_TILES
#define FS_MAX_TILES 64
#endif

}  // namespace

PassEvents& pass_events() {
  static thread_local PassEvents ev;
  return ev;
}

// Head width 64 takes the slot-blocked family above 64 slots: the cooperative kernels with two
// 64-slot waves per tile spill at that width (bf16, N = 2^18, G = 128: 2.65 -> 1.93 ms).
#ifndef FS_BLOCKED_MIN_G_D64
#define FS_BLOCKED_MIN_G_D64 64
#endif
bool blocked(const Geom& g) {
  // head width 64: bf16 storage and the tied path (fp32 images of a 64-slot block would not
  // fit twice in LDS)
  return g.G > (g.D == 64 ? FS_BLOCKED_MIN_G_D64 : FS_BLOCKED_MIN_G) &&
         (g.D <= 32 || (g.D == 64 && g.bf16 && !g.untied));
}

PassCfg pick_cfg(const Geom& g, Pass pass, int np) {
  PassCfg c{};
  c.nblk = 1;
  const bool blk = blocked(g);
  const bool slot_owned = blk && (pass == PASS_SLICE || pass == PASS_BWD_A || pass == PASS_BWD_B);
  // Slot counts that are not a whole tiling are padded up to one: the padding slots get a
  // masked logit (zero weight) and zero operands, and nothing of theirs is stored.
  if (g.G <= 64) {
    c.GS = g.G <= 16 && !g.bf16 ? 16 : (g.G <= 32 ? 32 : 64);  // bf16: 32-slot MFMA k sets
    c.NS = 1;
    c.NP = 4;
  } else if (slot_owned) {
    c.GS = 64;
    c.NS = 1;
    c.NP = 4;
    c.nblk = (g.G + 63) / 64;
  } else if (pass == PASS_POINT) {
    c.GS = 64;  // slot block streamed through LDS
    c.NS = 1;
    c.NP = np > 0 ? np : g.D > 32 ? FS_POINT_WAVES_WIDE : FS_POINT_WAVES;
  } else {
    c.GS = 64;
    c.NS = 2;  // the slot-wave counts with a tiling: 2, 4, 8, 16
    while (64 * c.NS < g.G) c.NS *= 2;
    c.NP = c.NS == 2 ? 2 : 1;
  }
  // fp32 backward pass B works on 16-point tiles (its register footprint is the largest)
  c.PB = (pass == PASS_BWD_B && !g.bf16 && c.NS == 1) ? FS_PB_F32 : 2;
  // Workgroups along the points per (sample, head[, slot block]): enough to fill 256 CUs
  // several times, but few enough that the per-workgroup partials stay small next to the
  // streamed data.
  const bool partials = pass != PASS_DESLICE && pass != PASS_STATS && pass != PASS_POINT;
  int target;
  if (c.NS >= 8)
    target = partials ? 256 : 512;
  else
    target = partials ? FS_TARGET_PARTIAL : FS_TARGET_DESLICE;
  const int64_t step = 16LL * c.PB * c.NP;
  const int64_t ntiles = std::max<int64_t>(1, (g.N + step - 1) / step);
  const int64_t units = (int64_t)g.BH() * c.nblk;
  int64_t chunks = std::max<int64_t>(1, (target + units - 1) / units);
  // passes that write partials give every chunk at least 4 tiles per point group, so the
  // partials stay small next to the points they summarise
  chunks = std::min<int64_t>(chunks, partials ? std::max<int64_t>(1, ntiles / FS_MIN_TILES) : ntiles);
  // but never fewer workgroups than compute units while tiles remain to spread (small N;
  // two tiles per point group at least where partials are written)
  chunks = std::max<int64_t>(
      chunks, std::min<int64_t>(partials ? ntiles / 2 : ntiles, (kCUs + units - 1) / units));
  // long streams take twice as many workgroups where every chunk still keeps 16 tiles: the
  // shorter per-workgroup runs shrink the tail of the last wave of workgroups
  if (c.NS < 8 && FS_TARGET_LONG > target) {
    const int64_t more = std::min<int64_t>((FS_TARGET_LONG + units - 1) / units, ntiles / 16);
    chunks = std::max<int64_t>(chunks, more);
  }
  // very long streams of the passes without partials (so the workspace stays bounded): at
  // most FS_MAX_TILES tiles per chunk, so that the head workgroups of one chunk, which share
  // the 128 B lines of the point rows through one L2, stay close together along the rows
  // (block_pos dispatches them one after another on such grids)
  if (FS_MAX_TILES > 0 && c.NS < 8 && !blk && !partials)
    chunks = std::max<int64_t>(chunks, (ntiles + FS_MAX_TILES - 1) / FS_MAX_TILES);
  // the kernels address a chunk's rows with 32-bit byte offsets (raw buffer loads)
  const int64_t row_bytes = (int64_t)g.H * g.D * (g.bf16 ? 2 : 4);
  const int64_t max_tiles = std::max<int64_t>(1, (((int64_t)1 << 31) - 1) / (row_bytes * step) - 1);
  chunks = std::max<int64_t>(chunks, (ntiles + max_tiles - 1) / max_tiles);
  int64_t tiles_per_chunk = (ntiles + chunks - 1) / chunks;
  c.chunk_pts = tiles_per_chunk * step;
  c.chunks = (int)std::max<int64_t>(1, (g.N + c.chunk_pts - 1) / c.chunk_pts);
  // the head (and slot-block) workgroups of one chunk are numbered `chunks` apart, and the 8
  // XCDs take workgroups round robin: a multiple of 8 puts them on one XCD, so the 128 B lines
  // that neighbouring heads' row segments share are fetched once into its L2. Chunks past the
  // last point are empty (their workgroups exit, their partials are zero).
  if (FS_XCD_CHUNKS && units > 1 && c.chunks >= 8 && c.chunks % 8 != 0)
    c.chunks = (c.chunks + 7) / 8 * 8;
  c.nsub = c.chunks;
  c.sub_pts = c.chunk_pts;
  // very long streams of the slice: a chunk's points are sub-chunks of at most FS_MAX_TILES
  // tiles spread over the stream (chunk c takes sub-chunks c, c + chunks, ...), so that the
  // head workgroups of every row block, which share its lines through one L2, reach it close
  // together, with the partial count (and so the workspace) unchanged
  if (FS_MAX_TILES > 0 && FS_SLICE_STRIDE && pass == PASS_SLICE && c.NS < 8 && !blk &&
      tiles_per_chunk > FS_MAX_TILES) {
    c.sub_pts = (int64_t)FS_MAX_TILES * step;
    c.nsub = (g.N + c.sub_pts - 1) / c.sub_pts;
  }
  return c;
}

size_t mix_param_count(const Geom& g, int kind, bool a_per_head) {
  switch (kind) {
    case FS_MIX_LINEAR_G:
      return (size_t)(a_per_head ? g.H : 1) * g.G * g.G;
    case FS_MIX_LINEAR_C:
      return (size_t)g.V * g.V;
    case FS_MIX_ATTN:
      return 3 * (size_t)g.V * g.V;
    default:
      return 0;
  }
}

FwdWs fwd_ws_layout(const Geom& g) {
  const PassCfg c = pick_cfg(g, PASS_SLICE);
  FwdWs L{};
  size_t off = 0;
  L.partU = off;
  off += up(sizeof(float) * (size_t)g.BH() * c.chunks * g.G * g.V);
  L.partS = off;
  off += up(sizeof(float) * (size_t)g.BH() * c.chunks * g.G);
  L.lse = off;
  off += up(blocked(g) ? sizeof(float) * (size_t)g.BH() * (size_t)g.N : 0);
  L.simg = off;
  off += up(blocked(g) ? stat_image_bytes(g) : 0);
  L.total = off;
  return L;
}

FwdWs linearno_fwd_ws_layout(const Geom& g) {
  const PassCfg c = pick_cfg(g, PASS_SLICE);
  FwdWs L{};
  size_t off = 0;
  L.partU = off;
  off += up(sizeof(float) * (size_t)g.BH() * c.chunks * g.G * g.V);
  L.partS = off;
  off += up(sizeof(float) * (size_t)g.BH() * c.chunks * 2 * g.G);
  L.lse = L.simg = off;
  L.total = off;
  return L;
}

BwdWs bwd_ws_layout(const Geom& g, int kind) {
  const PassCfg ca = pick_cfg(g, PASS_BWD_A);
  const PassCfg cb = pick_cfg(g, PASS_BWD_B);
  const size_t tok = sizeof(float) * (size_t)g.BH() * g.G * g.V;
  BwdWs L{};
  size_t off = 0;
  L.partDZ = off;
  off += up(sizeof(float) * (size_t)g.BH() * ca.chunks * g.G * g.V);
  L.dzm = off;
  off += up(tok);
  L.dz = off;
  off += up(tok);
  L.dU = off;
  off += up(tok);
  L.ds = off;
  off += up(sizeof(float) * (size_t)g.BH() * g.G);
  L.cen = off;
  off += up(sizeof(float) * (size_t)g.BH() * (2 * (size_t)g.V + 1));
  L.partP = off;
  off += up(sizeof(float) * (size_t)g.BH() * cb.chunks * (size_t)param_partial_len(g, cb.nblk));
  L.partM = off;
  size_t per_bh = 0;
  if (kind == FS_MIX_LINEAR_G) per_bh = (size_t)g.G * g.G;
  if (kind == FS_MIX_LINEAR_C) per_bh = (size_t)g.V * g.V;
  if (kind == FS_MIX_ATTN) per_bh = 3 * (size_t)g.V * g.V;
  off += up(sizeof(float) * (size_t)g.BH() * per_bh);
  L.scr = off;
  off += up(kind == FS_MIX_ATTN
                ? (attn_rows(g, kind) ? 6 : 3) * tok + sizeof(float) * (size_t)g.BH() * g.G * g.G
                : 0);
  L.cpt = off;
  off += up(blocked(g) ? 4 * sizeof(float) * (size_t)g.BH() * (size_t)g.N : 0);
  L.img = off;
  off += up(blocked(g) ? point_image_bytes(g) : 0);
  L.partP2 = off;  // the deslice weights' parameter partials (untied variant)
  off += up(g.untied ? sizeof(float) * (size_t)g.BH() * cb.chunks *
                           (size_t)param_partial_len(g, cb.nblk)
                     : 0);
  L.ones = off;    // LinearNO: unit weight sums for the token gradients
  off += up(g.linearno ? sizeof(float) * (size_t)g.BH() * g.G : 0);
  L.total = off;
  return L;
}

}  // namespace fs

using fs::Geom;

namespace {

struct Buf {
  const void* p;
  size_t bytes;
  bool required;
};

int check_problem(const fs_problem* p, Geom* g) {
  if (p == nullptr) return FS_ERR_NULL;
  if (p->B < 1 || p->N < 0 || p->H < 1 || p->D < 1 || p->V < 1 || p->G < 1) return FS_ERR_SHAPE;
  if (p->dtype != FS_F32 && p->dtype != FS_BF16) return FS_ERR_DTYPE;
  if (!std::isfinite(p->eps) || p->eps < 0.f) return FS_ERR_ARG;
  if (p->ws_per_head != 0 && p->ws_per_head != 1) return FS_ERR_ARG;
  // what the kernels implement
  if (p->D != p->V) return FS_ERR_UNSUPPORTED;
  if (p->D != 16 && p->D != 32 && p->D != 64) return FS_ERR_UNSUPPORTED;
  if (p->G % 16 != 0 || p->G > 1024) return FS_ERR_UNSUPPORTED;
  if (p->B * (int64_t)p->H > 65535) return FS_ERR_UNSUPPORTED;
  if (p->N > ((int64_t)1 << 40)) return FS_ERR_UNSUPPORTED;
  g->B = p->B;
  g->N = p->N;
  g->H = p->H;
  g->D = p->D;
  g->V = p->V;
  g->G = p->G;
  g->bf16 = p->dtype == FS_BF16;
  g->eps = p->eps;
  g->ws_per_head = p->ws_per_head != 0;
  return FS_OK;
}

int check_mix(const fs_mix_desc* m, const Geom& g) {
  if (m == nullptr) return FS_ERR_NULL;
  if (m->kind < FS_MIX_IDENTITY || m->kind > FS_MIX_ATTN) return FS_ERR_ARG;
  if (m->a_per_head != 0 && m->a_per_head != 1) return FS_ERR_ARG;
  if (m->kind == FS_MIX_LINEAR_G && m->A == nullptr) return FS_ERR_NULL;
  if (m->kind == FS_MIX_LINEAR_C && m->Wc == nullptr) return FS_ERR_NULL;
  if (m->kind == FS_MIX_ATTN) {
    if (m->Wq == nullptr || m->Wk == nullptr || m->Wv == nullptr) return FS_ERR_NULL;
    if (!std::isfinite(m->scale)) return FS_ERR_ARG;
  }
  return FS_OK;
}

fs::MixArgs mix_args(const fs_mix_desc* m) {
  fs::MixArgs a{};
  a.kind = m->kind;
  a.a_per_head = m->a_per_head != 0;
  a.A = m->A;
  a.Wc = m->Wc;
  a.Wq = m->Wq;
  a.Wk = m->Wk;
  a.Wv = m->Wv;
  a.scale = m->scale;
  return a;
}

// Mix parameters as buffers (inputs), for the alias check.
void mix_bufs(const fs_mix_desc* m, const Geom& g, Buf* out, int* n) {
  const size_t vv = sizeof(float) * (size_t)g.V * g.V;
  *n = 0;
  if (m->kind == FS_MIX_LINEAR_G)
    out[(*n)++] = {m->A, sizeof(float) * (size_t)(m->a_per_head ? g.H : 1) * g.G * g.G, true};
  if (m->kind == FS_MIX_LINEAR_C) out[(*n)++] = {m->Wc, vv, true};
  if (m->kind == FS_MIX_ATTN) {
    out[(*n)++] = {m->Wq, vv, true};
    out[(*n)++] = {m->Wk, vv, true};
    out[(*n)++] = {m->Wv, vv, true};
  }
}

bool overlap(const Buf& a, const Buf& b) {
  if (a.p == nullptr || b.p == nullptr || a.bytes == 0 || b.bytes == 0) return false;
  const uintptr_t a0 = (uintptr_t)a.p, a1 = a0 + a.bytes;
  const uintptr_t b0 = (uintptr_t)b.p, b1 = b0 + b.bytes;
  return a0 < b1 && b0 < a1;
}

// Null, alignment and aliasing checks. Buffers of zero bytes may be anything.
int check_bufs(const Buf* in, int nin, const Buf* out, int nout) {
  for (int k = 0; k < nin + nout; ++k) {
    const Buf& b = k < nin ? in[k] : out[k - nin];
    if (b.bytes == 0) continue;
    if (b.p == nullptr) {
      if (b.required) return FS_ERR_NULL;
      continue;
    }
    if (((uintptr_t)b.p) % 16 != 0) return FS_ERR_ALIGN;
  }
  for (int o = 0; o < nout; ++o) {
    for (int k = 0; k < nin; ++k)
      if (overlap(out[o], in[k])) return FS_ERR_ALIAS;
    for (int k = 0; k < o; ++k)
      if (overlap(out[o], out[k])) return FS_ERR_ALIAS;
  }
  return FS_OK;
}

struct Sizes {
  size_t x, fx, Ws, b, tau, tok, s, lse, attn;
};
Sizes sizes(const Geom& g) {
  const size_t elt = g.bf16 ? 2 : 4;
  Sizes z{};
  z.x = elt * (size_t)g.B * g.N * g.H * g.D;
  z.fx = elt * (size_t)g.B * g.N * g.H * g.V;
  z.Ws = sizeof(float) * (size_t)(g.ws_per_head ? g.H : 1) * g.D * g.G;
  z.b = sizeof(float) * (size_t)(g.ws_per_head ? g.H : 1) * g.G;
  z.tau = sizeof(float) * (size_t)g.H;
  z.tok = sizeof(float) * (size_t)g.BH() * g.G * g.V;
  z.s = sizeof(float) * (size_t)g.BH() * g.G;
  z.lse = sizeof(float) * (size_t)g.BH() * g.N;
  z.attn = sizeof(float) * (size_t)g.BH() * g.G * g.G;
  return z;
}

// The backward workspace requirement is the one fs_workspace_bytes(prob, 1) documents: the
// largest over all mix kinds, so one workspace serves every mix.
size_t bwd_required(const Geom& g) {
  size_t mx = 0;
  for (int k = FS_MIX_IDENTITY; k <= FS_MIX_ATTN; ++k) mx = std::max(mx, fs::bwd_ws_layout(g, k).total);
  return mx;
}

int hip_status(hipError_t e) {
  if (e == hipSuccess) return FS_OK;
  fs::g_last_hip_error = (int)e;
  return FS_ERR_HIP;
}

}  // namespace

extern "C" {

int fs_workspace_bytes(const fs_problem* prob, int for_backward, size_t* bytes) {
  Geom g;
  int st = check_problem(prob, &g);
  if (st != FS_OK) return st;
  if (bytes == nullptr) return FS_ERR_NULL;
  switch (for_backward) {
    case 0:
      *bytes = fs::fwd_ws_layout(g).total;
      return FS_OK;
    case 1:
    case 2:
    case 4:
      g.untied = for_backward != 1;
      g.linearno = for_backward == 4;
      *bytes = bwd_required(g);
      return FS_OK;
    case 3:
      g.untied = g.linearno = true;
      *bytes = fs::linearno_fwd_ws_layout(g).total;
      return FS_OK;
    default:
      return FS_ERR_ARG;
  }
}

int fs_slice_fwd(const fs_problem* prob, const void* x, const void* fx, const float* Ws,
                 const float* bias, const float* tau, float* z, float* s, float* lse, void* ws,
                 size_t ws_bytes, void* hip_stream) {
  Geom g;
  int st = check_problem(prob, &g);
  if (st != FS_OK) return st;
  const Sizes zs = sizes(g);
  const fs::FwdWs L = fs::fwd_ws_layout(g);
  const Buf in[] = {{x, zs.x, true}, {fx, zs.fx, true}, {Ws, zs.Ws, true},
                    {bias, zs.b, true}, {tau, zs.tau, true}};
  const Buf out[] = {{z, zs.tok, true}, {s, zs.s, true}, {lse, zs.lse, false},
                     {ws, ws_bytes, true}};
  st = check_bufs(in, 5, out, 4);
  if (st != FS_OK) return st;
  if (ws == nullptr || ws_bytes < L.total) return FS_ERR_WORKSPACE;
  char* w = static_cast<char*>(ws);
  return hip_status(fs::launch_slice(g, x, fx, Ws, bias, tau, z, s, lse, w,
                                     static_cast<hipStream_t>(hip_stream)));
}

int fs_slice_fwd_noalloc(const fs_problem* prob, const void* x, const void* fx, const float* Ws,
                         const float* bias, const float* tau, float* z, float* s, float* lse,
                         void* hip_stream) {
  Geom g;
  int st = check_problem(prob, &g);
  if (st != FS_OK) return st;
  const Sizes zs = sizes(g);
  const Buf in[] = {{x, zs.x, true}, {fx, zs.fx, true}, {Ws, zs.Ws, true},
                    {bias, zs.b, true}, {tau, zs.tau, true}};
  const Buf out[] = {{z, zs.tok, true}, {s, zs.s, true}, {lse, zs.lse, false}};
  st = check_bufs(in, 5, out, 3);
  if (st != FS_OK) return st;
  if (fs::fwd_ws_layout(g).total > fs::kStaticScratchBytes) return FS_ERR_WORKSPACE;
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e);
  if (stream != nullptr) {
    int sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return hip_status(e);
    if (sdev != dev) return FS_ERR_ARG;
  }
  void* scratch = nullptr;
  e = fs::static_scratch(dev, &scratch);
  if (e != hipSuccess) return hip_status(e);
  return hip_status(fs::launch_slice(g, x, fx, Ws, bias, tau, z, s, lse,
                                     static_cast<char*>(scratch), stream));
}

int fs_mix(const fs_problem* prob, const fs_mix_desc* mix, const float* z, float* zmix,
           float* attn_probs, void* hip_stream) {
  Geom g;
  int st = check_problem(prob, &g);
  if (st != FS_OK) return st;
  st = check_mix(mix, g);
  if (st != FS_OK) return st;
  const Sizes zs = sizes(g);
  Buf in[5];
  int nin = 0;
  mix_bufs(mix, g, in, &nin);
  in[nin++] = {z, zs.tok, true};
  const bool attn = mix->kind == FS_MIX_ATTN;
  const Buf out[] = {{zmix, zs.tok, true}, {attn ? attn_probs : nullptr, attn ? zs.attn : 0, true}};
  st = check_bufs(in, nin, out, 2);
  if (st != FS_OK) return st;
  return hip_status(fs::launch_mix(g, mix_args(mix), z, zmix, attn_probs,
                                   static_cast<hipStream_t>(hip_stream)));
}

int fs_mix_bwd(const fs_problem* prob, const fs_mix_desc* mix, const float* z,
               const float* attn_probs, const float* dzmix, float* dz, float* dmix_params,
               void* ws, size_t ws_bytes, void* hip_stream) {
  Geom g;
  int st = check_problem(prob, &g);
  if (st != FS_OK) return st;
  st = check_mix(mix, g);
  if (st != FS_OK) return st;
  const Sizes zs = sizes(g);
  const fs::BwdWs L = fs::bwd_ws_layout(g, mix->kind);
  const bool attn = mix->kind == FS_MIX_ATTN;
  Buf in[7];
  int nin = 0;
  mix_bufs(mix, g, in, &nin);
  in[nin++] = {z, zs.tok, true};
  in[nin++] = {dzmix, zs.tok, true};
  in[nin++] = {attn ? attn_probs : nullptr, attn ? zs.attn : 0, true};
  const size_t np = sizeof(float) * fs::mix_param_count(g, mix->kind, mix->a_per_head != 0);
  const Buf out[] = {{dz, zs.tok, true}, {dmix_params, np, false}, {ws, ws_bytes, true}};
  st = check_bufs(in, nin, out, 3);
  if (st != FS_OK) return st;
  if (ws == nullptr || ws_bytes < bwd_required(g)) return FS_ERR_WORKSPACE;
  char* w = static_cast<char*>(ws);
  return hip_status(fs::launch_mix_bwd(
      g, mix_args(mix), z, nullptr, nullptr, attn_probs, dzmix, dz, nullptr, nullptr, nullptr,
      reinterpret_cast<float*>(w + L.scr), reinterpret_cast<float*>(w + L.partM),
      mix->kind == FS_MIX_IDENTITY ? nullptr : dmix_params, true,
      static_cast<hipStream_t>(hip_stream)));
}

int fs_deslice_fwd(const fs_problem* prob, const void* x, const float* Ws, const float* bias,
                   const float* tau, const float* zmix, const float* lse, void* out,
                   void* hip_stream) {
  Geom g;
  int st = check_problem(prob, &g);
  if (st != FS_OK) return st;
  const Sizes zs = sizes(g);
  const Buf in[] = {{x, zs.x, true},     {Ws, zs.Ws, true},     {bias, zs.b, true},
                    {tau, zs.tau, true}, {zmix, zs.tok, true},  {lse, zs.lse, false}};
  const Buf outb[] = {{out, zs.fx, true}};
  st = check_bufs(in, 6, outb, 1);
  if (st != FS_OK) return st;
  return hip_status(fs::launch_deslice(g, x, Ws, bias, tau, zmix, lse, nullptr, out,
                                       static_cast<hipStream_t>(hip_stream)));
}

int fs_deslice_stats_fwd(const fs_problem* prob, const void* x, const float* Ws,
                         const float* bias, const float* tau, const float* zmix, float* lse_out,
                         void* out, void* hip_stream) {
  Geom g;
  int st = check_problem(prob, &g);
  if (st != FS_OK) return st;
  const Sizes zs = sizes(g);
  const Buf in[] = {{x, zs.x, true},     {Ws, zs.Ws, true},   {bias, zs.b, true},
                    {tau, zs.tau, true}, {zmix, zs.tok, true}};
  const Buf outb[] = {{out, zs.fx, true}, {lse_out, zs.lse, false}};
  st = check_bufs(in, 5, outb, 2);
  if (st != FS_OK) return st;
  return hip_status(fs::launch_deslice(g, x, Ws, bias, tau, zmix, nullptr, lse_out, out,
                                       static_cast<hipStream_t>(hip_stream)));
}

int fs_slice_deslice_bwd(const fs_problem* prob, const fs_mix_desc* mix, const void* x,
                         const void* fx, const float* Ws, const float* bias, const float* tau,
                         const float* z, const float* s, const float* zmix,
                         const float* attn_probs, const float* lse, const void* dout, void* dx,
                         void* dfx, float* dWs, float* dbias, float* dtau, float* dmix_params,
                         float* dzmix_out, void* ws, size_t ws_bytes, void* hip_stream) {
  Geom g;
  int st = check_problem(prob, &g);
  if (st != FS_OK) return st;
  st = check_mix(mix, g);
  if (st != FS_OK) return st;
  const Sizes zs = sizes(g);
  const fs::BwdWs L = fs::bwd_ws_layout(g, mix->kind);
  const bool attn = mix->kind == FS_MIX_ATTN;
  Buf in[16];
  int nin = 0;
  mix_bufs(mix, g, in, &nin);
  in[nin++] = {x, zs.x, true};
  in[nin++] = {fx, zs.fx, true};
  in[nin++] = {Ws, zs.Ws, true};
  in[nin++] = {bias, zs.b, true};
  in[nin++] = {tau, zs.tau, true};
  in[nin++] = {z, zs.tok, true};
  in[nin++] = {s, zs.s, true};
  in[nin++] = {zmix, zs.tok, true};
  in[nin++] = {attn ? attn_probs : nullptr, attn ? zs.attn : 0, true};
  in[nin++] = {lse, zs.lse, true};
  in[nin++] = {dout, zs.fx, true};
  const size_t np = sizeof(float) * fs::mix_param_count(g, mix->kind, mix->a_per_head != 0);
  const Buf out[] = {{dx, zs.x, true},          {dfx, zs.fx, true},       {dWs, zs.Ws, true},
                     {dbias, zs.b, true},       {dtau, zs.tau, true},     {dmix_params, np, false},
                     {dzmix_out, zs.tok, false}, {ws, ws_bytes, true}};
  st = check_bufs(in, nin, out, 8);
  if (st != FS_OK) return st;
  if (ws == nullptr || ws_bytes < bwd_required(g)) return FS_ERR_WORKSPACE;
  return hip_status(fs::launch_bwd(g, mix_args(mix), x, fx, Ws, bias, tau, z, s, zmix,
                                   attn_probs, lse, dout, dx, dfx, dWs, dbias, dtau,
                                   mix->kind == FS_MIX_IDENTITY ? nullptr : dmix_params,
                                   dzmix_out, static_cast<char*>(ws),
                                   static_cast<hipStream_t>(hip_stream)));
}

int fs_linearno_slice_fwd(const fs_problem* prob, const void* x, const void* fx,
                          const float* Ws, const float* bias, const float* tau, float* z,
                          float* clse, void* ws, size_t ws_bytes, void* hip_stream) {
  Geom g;
  int st = check_problem(prob, &g);
  if (st != FS_OK) return st;
  g.untied = g.linearno = true;
  const Sizes zs = sizes(g);
  const Buf in[] = {{x, zs.x, true}, {fx, zs.fx, true}, {Ws, zs.Ws, true}, {bias, zs.b, true},
                    {tau, zs.tau, true}};
  const Buf out[] = {{z, zs.tok, true}, {clse, zs.s, false}, {ws, ws_bytes, true}};
  st = check_bufs(in, 5, out, 3);
  if (st != FS_OK) return st;
  if (ws == nullptr || ws_bytes < fs::linearno_fwd_ws_layout(g).total) return FS_ERR_WORKSPACE;
  return hip_status(fs::launch_linearno_slice(g, x, fx, Ws, bias, tau, z, clse,
                                              static_cast<char*>(ws),
                                              static_cast<hipStream_t>(hip_stream)));
}

int fs_linearno_bwd(const fs_problem* prob, const fs_mix_desc* mix, const void* x, const void* fx,
                    const float* Ws, const float* bias, const float* tau, const float* Wd,
                    const float* bd, const float* taud, const float* z, const float* clse,
                    const float* zmix, const float* attn_probs, const float* lse_d,
                    const void* dout, void* dx, void* dfx, float* dWs, float* dbias,
                    float* dtau, float* dWd, float* dbd, float* dtaud, float* dmix_params,
                    float* dzmix_out, void* ws, size_t ws_bytes, void* hip_stream) {
  Geom g;
  int st = check_problem(prob, &g);
  if (st != FS_OK) return st;
  st = check_mix(mix, g);
  if (st != FS_OK) return st;
  g.untied = g.linearno = true;
  const Sizes zs = sizes(g);
  const bool attn = mix->kind == FS_MIX_ATTN;
  Buf in[20];
  int nin = 0;
  mix_bufs(mix, g, in, &nin);
  in[nin++] = {x, zs.x, true};
  in[nin++] = {fx, zs.fx, true};
  in[nin++] = {Ws, zs.Ws, true};
  in[nin++] = {bias, zs.b, true};
  in[nin++] = {tau, zs.tau, true};
  in[nin++] = {Wd, zs.Ws, true};
  in[nin++] = {bd, zs.b, true};
  in[nin++] = {taud, zs.tau, true};
  in[nin++] = {z, zs.tok, true};
  in[nin++] = {clse, zs.s, true};
  in[nin++] = {zmix, zs.tok, true};
  in[nin++] = {attn ? attn_probs : nullptr, attn ? zs.attn : 0, true};
  in[nin++] = {lse_d, zs.lse, true};
  in[nin++] = {dout, zs.fx, true};
  const size_t np = sizeof(float) * fs::mix_param_count(g, mix->kind, mix->a_per_head != 0);
  const Buf out[] = {{dx, zs.x, true},       {dfx, zs.fx, true},        {dWs, zs.Ws, true},
                     {dbias, zs.b, true},    {dtau, zs.tau, true},      {dWd, zs.Ws, true},
                     {dbd, zs.b, true},      {dtaud, zs.tau, true},     {dmix_params, np, false},
                     {dzmix_out, zs.tok, false}, {ws, ws_bytes, true}};
  st = check_bufs(in, nin, out, 11);
  if (st != FS_OK) return st;
  if (ws == nullptr || ws_bytes < bwd_required(g)) return FS_ERR_WORKSPACE;
  const fs::UntiedArgs u{Wd, bd, taud, lse_d, dWd, dbd, dtaud};
  return hip_status(fs::launch_bwd(g, mix_args(mix), x, fx, Ws, bias, tau, z, nullptr, zmix,
                                   attn_probs, nullptr, dout, dx, dfx, dWs, dbias, dtau,
                                   mix->kind == FS_MIX_IDENTITY ? nullptr : dmix_params,
                                   dzmix_out, static_cast<char*>(ws),
                                   static_cast<hipStream_t>(hip_stream), &u, clse));
}

int fs_untied_bwd(const fs_problem* prob, const fs_mix_desc* mix, const void* x, const void* fx,
                  const float* Ws, const float* bias, const float* tau, const float* Wd,
                  const float* bd, const float* taud, const float* z, const float* s,
                  const float* zmix, const float* attn_probs, const float* lse,
                  const float* lse_d, const void* dout, void* dx, void* dfx, float* dWs,
                  float* dbias, float* dtau, float* dWd, float* dbd, float* dtaud,
                  float* dmix_params, float* dzmix_out, void* ws, size_t ws_bytes,
                  void* hip_stream) {
  Geom g;
  int st = check_problem(prob, &g);
  if (st != FS_OK) return st;
  st = check_mix(mix, g);
  if (st != FS_OK) return st;
  g.untied = true;
  const Sizes zs = sizes(g);
  const bool attn = mix->kind == FS_MIX_ATTN;
  Buf in[20];
  int nin = 0;
  mix_bufs(mix, g, in, &nin);
  in[nin++] = {x, zs.x, true};
  in[nin++] = {fx, zs.fx, true};
  in[nin++] = {Ws, zs.Ws, true};
  in[nin++] = {bias, zs.b, true};
  in[nin++] = {tau, zs.tau, true};
  in[nin++] = {Wd, zs.Ws, true};
  in[nin++] = {bd, zs.b, true};
  in[nin++] = {taud, zs.tau, true};
  in[nin++] = {z, zs.tok, true};
  in[nin++] = {s, zs.s, true};
  in[nin++] = {zmix, zs.tok, true};
  in[nin++] = {attn ? attn_probs : nullptr, attn ? zs.attn : 0, true};
  in[nin++] = {lse, zs.lse, true};
  in[nin++] = {lse_d, zs.lse, true};
  in[nin++] = {dout, zs.fx, true};
  const size_t np = sizeof(float) * fs::mix_param_count(g, mix->kind, mix->a_per_head != 0);
  const Buf out[] = {{dx, zs.x, true},       {dfx, zs.fx, true},        {dWs, zs.Ws, true},
                     {dbias, zs.b, true},    {dtau, zs.tau, true},      {dWd, zs.Ws, true},
                     {dbd, zs.b, true},      {dtaud, zs.tau, true},     {dmix_params, np, false},
                     {dzmix_out, zs.tok, false}, {ws, ws_bytes, true}};
  st = check_bufs(in, nin, out, 11);
  if (st != FS_OK) return st;
  if (ws == nullptr || ws_bytes < bwd_required(g)) return FS_ERR_WORKSPACE;
  const fs::UntiedArgs u{Wd, bd, taud, lse_d, dWd, dbd, dtaud};
  return hip_status(fs::launch_bwd(g, mix_args(mix), x, fx, Ws, bias, tau, z, s, zmix,
                                   attn_probs, lse, dout, dx, dfx, dWs, dbias, dtau,
                                   mix->kind == FS_MIX_IDENTITY ? nullptr : dmix_params,
                                   dzmix_out, static_cast<char*>(ws),
                                   static_cast<hipStream_t>(hip_stream), &u));
}

int fs_set_pass_events(int pass, void* before, void* after) {
  if (pass < -1 || pass > 3) return FS_ERR_ARG;
  fs::PassEvents& ev = fs::pass_events();
  if (pass < 0) {
    ev = fs::PassEvents{};
    return FS_OK;
  }
  ev.before[pass] = static_cast<hipEvent_t>(before);
  ev.after[pass] = static_cast<hipEvent_t>(after);
  return FS_OK;
}

const char* fs_status_string(int status) {
  switch (status) {
    case FS_OK:
      return "ok";
    case FS_ERR_NULL:
      return "a required pointer is NULL";
    case FS_ERR_SHAPE:
      return "invalid sizes";
    case FS_ERR_DTYPE:
      return "unknown storage dtype";
    case FS_ERR_UNSUPPORTED:
      return "shape not supported by this library";
    case FS_ERR_WORKSPACE:
      return "workspace missing or too small";
    case FS_ERR_ARG:
      return "invalid argument";
    case FS_ERR_ALIGN:
      return "device pointer not 16-byte aligned";
    case FS_ERR_ALIAS:
      return "an output overlaps an input or another output";
    case FS_ERR_HIP:
      return "HIP runtime error";
    default:
      return "unknown status";
  }
}

int fs_last_hip_error(void) { return fs::g_last_hip_error; }

}  // extern "C"
