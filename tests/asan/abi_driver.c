/* Exercises the host-side validation of every entry point of flashslice.h with fake device
 * addresses (never dereferenced): each call must return the expected status. Built with the
 * address and undefined-behaviour sanitizers against the C-ABI layer and host stubs of the
 * launchers (abi_stubs.cpp), so any out-of-bounds access, leak or undefined behaviour in the
 * validation code aborts the run. Exit status 0 when every expectation holds. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "../../include/flashslice.h"

static int failures = 0;
#define EXPECT(call, want)                                                        \
  do {                                                                            \
    int got_ = (call);                                                            \
    if (got_ != (want)) {                                                         \
      fprintf(stderr, "line %d: %s -> %d, want %d\n", __LINE__, #call, got_, want); \
      ++failures;                                                                 \
    }                                                                             \
  } while (0)

static uintptr_t next_addr = (uintptr_t)1 << 44;
static void* fake(void) { /* distinct, far apart, 256-byte aligned */
  next_addr += (uintptr_t)1 << 36;
  return (void*)next_addr;
}

static fs_problem prob(int64_t N, int G, int dtype) {
  fs_problem p;
  memset(&p, 0, sizeof p);
  p.B = 2; p.N = N; p.H = 3; p.D = 32; p.V = 32; p.G = G; p.dtype = dtype; p.eps = 1e-5f;
  p.ws_per_head = 0;
  return p;
}

int main(void) {
  size_t wsf = 0, wsb = 0, wsu = 0, wsl = 0, wslb = 0;
  fs_problem p = prob(1000, 64, FS_BF16);
  EXPECT(fs_workspace_bytes(&p, 0, &wsf), FS_OK);
  EXPECT(fs_workspace_bytes(&p, 1, &wsb), FS_OK);
  EXPECT(fs_workspace_bytes(&p, 2, &wsu), FS_OK);
  EXPECT(fs_workspace_bytes(&p, 3, &wsl), FS_OK);
  EXPECT(fs_workspace_bytes(&p, 4, &wslb), FS_OK);
  EXPECT(fs_workspace_bytes(&p, 5, &wsf), FS_ERR_ARG);
  EXPECT(fs_workspace_bytes(NULL, 0, &wsf), FS_ERR_NULL);
  EXPECT(fs_workspace_bytes(&p, 0, NULL), FS_ERR_NULL);

  /* problem validation */
  fs_problem bad = p; bad.B = 0;        EXPECT(fs_workspace_bytes(&bad, 0, &wsf), FS_ERR_SHAPE);
  bad = p; bad.N = -1;                  EXPECT(fs_workspace_bytes(&bad, 0, &wsf), FS_ERR_SHAPE);
  bad = p; bad.dtype = 9;               EXPECT(fs_workspace_bytes(&bad, 0, &wsf), FS_ERR_DTYPE);
  bad = p; bad.eps = -1.f;              EXPECT(fs_workspace_bytes(&bad, 0, &wsf), FS_ERR_ARG);
  bad = p; bad.G = 40;                  EXPECT(fs_workspace_bytes(&bad, 0, &wsf), FS_ERR_UNSUPPORTED);
  { size_t w48; bad = p; bad.G = 48;    EXPECT(fs_workspace_bytes(&bad, 0, &w48), FS_OK); }
  bad = p; bad.D = 32; bad.V = 16;      EXPECT(fs_workspace_bytes(&bad, 0, &wsf), FS_ERR_UNSUPPORTED);
  bad = p; bad.ws_per_head = 2;         EXPECT(fs_workspace_bytes(&bad, 0, &wsf), FS_ERR_ARG);

  void *x = fake(), *fx = fake(), *Ws = fake(), *b = fake(), *tau = fake(), *z = fake();
  void *s = fake(), *zm = fake(), *lse = fake(), *out = fake(), *ws = fake(), *P = fake();
  void *dout = fake(), *dx = fake(), *dfx = fake(), *dWs = fake(), *db = fake(), *dt = fake();
  void *A = fake(), *dA = fake(), *dzm = fake(), *Wd = fake(), *bd = fake(), *td = fake();
  void *lsed = fake(), *dWd = fake(), *dbd = fake(), *dtd = fake(), *clse = fake();
  fs_mix_desc m;
  memset(&m, 0, sizeof m);
  m.kind = FS_MIX_LINEAR_G; m.A = (const float*)A;

  /* slice */
  EXPECT(fs_slice_fwd(&p, x, fx, Ws, b, tau, z, s, lse, ws, wsf, NULL), FS_ERR_HIP);
  EXPECT(fs_slice_fwd(&p, NULL, fx, Ws, b, tau, z, s, lse, ws, wsf, NULL), FS_ERR_NULL);
  EXPECT(fs_slice_fwd(&p, (char*)x + 4, fx, Ws, b, tau, z, s, lse, ws, wsf, NULL), FS_ERR_ALIGN);
  EXPECT(fs_slice_fwd(&p, x, fx, Ws, b, tau, x, s, lse, ws, wsf, NULL), FS_ERR_ALIAS);
  EXPECT(fs_slice_fwd(&p, x, fx, Ws, b, tau, z, s, lse, ws, wsf - 1, NULL), FS_ERR_WORKSPACE);
  EXPECT(fs_slice_fwd_noalloc(&p, x, fx, Ws, b, tau, z, s, lse, NULL), FS_ERR_HIP);
  /* mix */
  EXPECT(fs_mix(&p, &m, z, zm, NULL, NULL), FS_ERR_HIP);
  EXPECT(fs_mix(&p, NULL, z, zm, NULL, NULL), FS_ERR_NULL);
  m.kind = 7; EXPECT(fs_mix(&p, &m, z, zm, NULL, NULL), FS_ERR_ARG); m.kind = FS_MIX_LINEAR_G;
  EXPECT(fs_mix(&p, &m, z, z, NULL, NULL), FS_ERR_ALIAS);
  m.kind = FS_MIX_ATTN;
  EXPECT(fs_mix(&p, &m, z, zm, P, NULL), FS_ERR_NULL);       /* Wq, Wk, Wv missing */
  m.kind = FS_MIX_LINEAR_G;
  EXPECT(fs_mix_bwd(&p, &m, z, NULL, dzm, s, dA, ws, wsb, NULL), FS_ERR_HIP);
  EXPECT(fs_mix_bwd(&p, &m, z, NULL, dzm, s, dA, ws, wsb - 1, NULL), FS_ERR_WORKSPACE);
  /* deslice */
  EXPECT(fs_deslice_fwd(&p, x, Ws, b, tau, zm, lse, out, NULL), FS_ERR_HIP);
  EXPECT(fs_deslice_fwd(&p, x, Ws, b, tau, zm, lse, x, NULL), FS_ERR_ALIAS);
  EXPECT(fs_deslice_stats_fwd(&p, x, Ws, b, tau, zm, lse, out, NULL), FS_ERR_HIP);
  EXPECT(fs_deslice_stats_fwd(&p, x, Ws, b, tau, zm, lse, lse, NULL), FS_ERR_ALIAS);
  /* backward */
  EXPECT(fs_slice_deslice_bwd(&p, &m, x, fx, Ws, b, tau, z, s, zm, NULL, lse, dout, dx, dfx,
                              dWs, db, dt, dA, dzm, ws, wsb, NULL), FS_ERR_HIP);
  EXPECT(fs_slice_deslice_bwd(&p, &m, x, fx, Ws, b, tau, z, s, zm, NULL, lse, dout, dx, dfx,
                              dWs, db, dt, dA, dzm, ws, wsb - 1, NULL), FS_ERR_WORKSPACE);
  EXPECT(fs_slice_deslice_bwd(&p, &m, x, fx, Ws, b, tau, z, s, zm, NULL, lse, dout, dx, dx,
                              dWs, db, dt, dA, dzm, ws, wsb, NULL), FS_ERR_ALIAS);
  EXPECT(fs_slice_deslice_bwd(&p, &m, x, fx, Ws, b, tau, z, s, zm, NULL, NULL, dout, dx, dfx,
                              dWs, db, dt, dA, dzm, ws, wsb, NULL), FS_ERR_NULL);
  /* untied and LinearNO */
  EXPECT(fs_untied_bwd(&p, &m, x, fx, Ws, b, tau, Wd, bd, td, z, s, zm, NULL, lse, lsed, dout,
                       dx, dfx, dWs, db, dt, dWd, dbd, dtd, dA, dzm, ws, wsu, NULL), FS_ERR_HIP);
  EXPECT(fs_untied_bwd(&p, &m, x, fx, Ws, b, tau, Wd, bd, td, z, s, zm, NULL, lse, lsed, dout,
                       dx, dfx, dWs, db, dt, dWd, dbd, dtd, dA, dzm, ws, wsu - 1, NULL),
         FS_ERR_WORKSPACE);
  EXPECT(fs_linearno_slice_fwd(&p, x, fx, Ws, b, tau, z, clse, ws, wsl, NULL), FS_ERR_HIP);
  EXPECT(fs_linearno_slice_fwd(&p, x, fx, Ws, b, tau, z, clse, ws, wsl - 1, NULL),
         FS_ERR_WORKSPACE);
  EXPECT(fs_linearno_bwd(&p, &m, x, fx, Ws, b, tau, Wd, bd, td, z, clse, zm, NULL, lsed, dout,
                         dx, dfx, dWs, db, dt, dWd, dbd, dtd, dA, dzm, ws, wslb, NULL), FS_ERR_HIP);
  /* status strings and the recorded HIP error */
  for (int st = 1; st >= -12; --st) EXPECT(fs_status_string(st) != NULL, 1);
  EXPECT(fs_last_hip_error() != 0, 1);
  EXPECT(fs_set_pass_events(9, NULL, NULL), FS_ERR_ARG);
  EXPECT(fs_set_pass_events(-1, NULL, NULL), FS_OK);
  if (failures) fprintf(stderr, "%d expectation(s) failed\n", failures);
  else printf("all expectations hold\n");
  return failures ? 1 : 0;
}
