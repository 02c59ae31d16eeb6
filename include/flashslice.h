/*
 * flashslice.h - C ABI of the fused slice -> token mix -> deslice path of Transolver
 * physics-attention on AMD Instinct MI355X (gfx950).
 *
 * What the calls compute, per sample b and head h (paper: Sec. 2 "The Transolver layer",
 * Eq. (1), App. F.1 "Kernel design", App. F.2 "Temperature gradients"):
 *
 *   logits   a[n, g] = (x[n, :] . W_s[:, g] + bias[g]) / tau[h]
 *   weights  w[n, :] = softmax over the G slices of a[n, :]      (never written to memory)
 *   slice    s[g] = sum_n w[n, g];  z[g, :] = (sum_n w[n, g] fx[n, :]) / (s[g] + eps)
 *   mix      zmix = Mix(z)   (identity, fixed G x G matrix, per-token channel map, or
 *                              single-head softmax self-attention among the G tokens)
 *   deslice  out[n, :] = sum_g w[n, g] zmix[g, :]
 *
 * and the exact backward of that composition. The N x G slice-weight tensor never exists in
 * device memory: every pass recomputes the weights from x and the saved per-point
 * normaliser `lse`.
 *
 * lse is stored in base 2, the unit the kernels compute in:
 *   lse[n] = log2( sum_g 2^(a[n, g] * log2(e)) ) = log(sum_g exp(a[n, g])) * log2(e),
 * so that w[n, g] = 2^(a[n, g] * log2(e) - lse[n]) with no unit conversion between passes.
 *
 * Conventions (all entry points):
 *   - Pointers are device pointers (hipMalloc / torch), owned by the caller. The library never
 *     allocates, frees, retains pointers or synchronises. All work is enqueued on `hip_stream`
 *     (a hipStream_t; NULL means the default stream); buffers must stay alive until it
 *     completes.
 *   - Layouts are row-major and contiguous:
 *       x (B,N,H,D), fx (B,N,H,V), out / dout / dfx (B,N,H,V), dx (B,N,H,D) in the storage
 *       dtype; z, zmix, dzmix (B,H,G,V), s (B,H,G), lse (B,H,N), attn_probs (B,H,G,G),
 *       W_s (D,G) [or (H,D,G) with ws_per_head], bias (G) [or (H,G)], tau (H): fp32.
 *   - Every device pointer must be 16-byte aligned.
 *   - Outputs are overwritten, never accumulated. Gradients of parameters shared by heads
 *     are summed over samples and heads. Inputs are never modified. An output that overlaps
 *     any input or another output is rejected (FS_ERR_ALIAS).
 *   - Errors: a negative fs_status is returned after host-side validation, before anything
 *     is enqueued; nothing is printed. A failed launch returns FS_ERR_HIP and records the
 *     hipError_t for fs_last_hip_error() (per thread).
 *   - tau > 0 is a precondition (tau lives in device memory and is not read by the host).
 *   - Results are deterministic: no atomics; every reduction has a fixed order, so repeated
 *     calls give bitwise identical outputs.
 *   - Supported shapes: D == V in {16, 32, 64}; G a multiple of 16 in [16, 1024], for every
 *     mix kind and storage type (slot counts between the kernels' tile sizes run padded up
 *     to the next one, the padding slots carrying zero weight); B * H <= 65535. Anything
 *     else returns FS_ERR_UNSUPPORTED.
 *   - Concurrent calls are safe as long as they do not share a workspace.
 */
#ifndef FLASHSLICE_H
#define FLASHSLICE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Storage dtype of x, fx, out, dout, dx, dfx. Arithmetic always accumulates in fp32. */
typedef enum { FS_F32 = 0, FS_BF16 = 1 } fs_dtype;

typedef enum {
  FS_OK = 0,
  FS_ERR_NULL = -1,        /* a required pointer is NULL                                  */
  FS_ERR_SHAPE = -2,       /* non-positive or inconsistent sizes                           */
  FS_ERR_DTYPE = -3,       /* unknown dtype                                                */
  FS_ERR_UNSUPPORTED = -4, /* valid problem outside the shapes this library implements     */
  FS_ERR_WORKSPACE = -5,   /* workspace missing or smaller than fs_workspace_bytes()       */
  FS_ERR_ARG = -6,         /* other invalid argument (eps < 0 or not finite, mix kind ...) */
  FS_ERR_ALIGN = -7,       /* a device pointer is not 16-byte aligned                      */
  FS_ERR_ALIAS = -8,       /* an output overlaps an input or another output                */
  FS_ERR_HIP = -9          /* the HIP runtime reported an error at launch                  */
} fs_status;

/* Problem description. B >= 1, N >= 0 points per sample (N = 0 is allowed: tokens are 0/eps),
 * H >= 1 heads, D = slice-projection width (dh), V = value width, G = number of slices.     */
typedef struct {
  int64_t B, N;
  int32_t H, D, V, G;
  int32_t dtype;        /* fs_dtype                                                        */
  float eps;            /* z = U / (s + eps); must be finite and >= 0 (paper: App. F.1)    */
  int32_t ws_per_head;  /* 0: W_s (D,G) and bias (G) shared by heads; 1: (H,D,G) and (H,G) */
} fs_problem;

typedef enum {
  FS_MIX_IDENTITY = 0, /* zmix = z                                                          */
  FS_MIX_LINEAR_G = 1, /* zmix[g, :] = sum_k A[g, k] z[k, :]   (constant core of Eq. (1))     */
  FS_MIX_LINEAR_C = 2, /* zmix = z Wc                          (per-token channel map)        */
  FS_MIX_ATTN = 3      /* q = z Wq, k = z Wk, v = z Wv; P = softmax_row(scale q k^T); zmix = P v */
} fs_mix_kind;

/* Token mix parameters (fp32 device pointers; only those of `kind` are read).
 * A: (G,G), or (H,G,G) when a_per_head = 1. Wc, Wq, Wk, Wv: (V,V), shared by heads.       */
typedef struct {
  int32_t kind;         /* fs_mix_kind                                                     */
  int32_t a_per_head;
  const float* A;
  const float* Wc;
  const float* Wq;
  const float* Wk;
  const float* Wv;
  float scale;          /* attention logit scale, e.g. 1/sqrt(V)                           */
} fs_mix_desc;

/* Bytes of device workspace needed by fs_slice_fwd (for_backward = 0), by fs_mix_bwd and
 * fs_slice_deslice_bwd (for_backward = 1), by fs_untied_bwd (for_backward = 2), by
 * fs_linearno_slice_fwd (for_backward = 3) or by fs_linearno_bwd (for_backward = 4), for
 * this problem. It holds per-workgroup partial sums (a bounded number of workgroups) and
 * token-sized buffers (G x V per sample and head). The slot-blocked kernels (G > 128 with
 * D <= 32, or G > 64 with D = 64 in bf16; tied path) add per-point state: 4 bytes per (point, head) in the forward (the
 * normaliser) and 16 in the backward (the softmax correction, the weighted mean logit and
 * the normaliser again, one record per point for the parameter pass),
 * plus per-head operand images (G x (2D + 3V) values). No size grows with N * G.
 * Returns FS_OK and writes *bytes, or a validation error (FS_ERR_ARG for another
 * for_backward). (A status return with an out-parameter, so that an invalid problem is an
 * error code rather than a size.)                                                         */
int fs_workspace_bytes(const fs_problem* prob, int for_backward, size_t* bytes);

/* Slice (paper: Sec. 2; App. F.1 single-tile equation): recompute the slice weights per
 * point tile and reduce them into s (B,H,G) and the normalised tokens z (B,H,G,V).
 * lse (B,H,N), nullable: receives the base-2 normaliser log2(sum_g 2^(a[n, g] log2 e)) per
 * point, needed by the deslice and the backward.
 * ws/ws_bytes: workspace of at least fs_workspace_bytes(prob, 0, .) bytes.                  */
int fs_slice_fwd(const fs_problem* prob, const void* x, const void* fx, const float* Ws,
                 const float* bias, const float* tau, float* z, float* s, float* lse,
                 void* ws, size_t ws_bytes, void* hip_stream);

/* fs_slice_fwd for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same computation and
 * the same outputs (z, s, optional lse), with the workspace taken from a static scratch
 * array of 64 MiB that the library holds on every GPU it runs on until the process ends. With
 * it the whole forward (this call, fs_mix, fs_deslice_fwd or fs_deslice_stats_fwd) needs no
 * caller workspace. It allocates nothing and calls no allocating routine. Returns
 * FS_ERR_WORKSPACE when the problem needs more than 64 MiB (fs_workspace_bytes(prob, 0, .)
 * tells), FS_ERR_ARG when hip_stream belongs to a device other than the current one. The
 * scratch is shared by every call on one GPU: calls that overlap on one GPU (other streams,
 * other threads) race on it and must be serialised by the caller.                          */
int fs_slice_fwd_noalloc(const fs_problem* prob, const void* x, const void* fx,
                         const float* Ws, const float* bias, const float* tau, float* z,
                         float* s, float* lse, void* hip_stream);

/* Token mix (paper: Sec. 2; Eq. (1); the attention-free variant). z, zmix: (B,H,G,V).
 * attn_probs: (B,H,G,G) output, required for FS_MIX_ATTN (saved for the backward),
 * ignored otherwise. Needs no workspace for any G (attention up to G = 1024 included).      */
int fs_mix(const fs_problem* prob, const fs_mix_desc* mix, const float* z, float* zmix,
           float* attn_probs, void* hip_stream);

/* Backward of the token mix (paper: the derivative of Eq. (1) and of the token
 * self-attention of Sec. 2 with respect to the tokens and the mix parameters):
 * dz = Mix^T(dzmix) and the mix-parameter gradient (summed over samples and heads; per head
 * for a per-head A): dmix_params is dA (G,G)/(H,G,G) for LINEAR_G, dWc (V,V) for LINEAR_C,
 * [dWq; dWk; dWv] (3,V,V) for ATTN; nullable (skipped). ws/ws_bytes: the backward workspace,
 * fs_workspace_bytes(prob, 1, .) bytes (the attention backward keeps q, k, v and dP there,
 * and the per-(sample, head) parameter partials are summed from it in a fixed order).     */
int fs_mix_bwd(const fs_problem* prob, const fs_mix_desc* mix, const float* z,
               const float* attn_probs, const float* dzmix, float* dz, float* dmix_params,
               void* ws, size_t ws_bytes, void* hip_stream);

/* Deslice (paper: Sec. 2, u_i = sum_g w_ig z'_g; App. F.1): recompute the weights from x and
 * write out (B,N,H,V) = w zmix in the storage dtype. lse (B,H,N) is the base-2 normaliser
 * saved by fs_slice_fwd; nullable: the kernel then recomputes each point's normaliser from its
 * logits (as fs_deslice_stats_fwd without the lse output).                                 */
int fs_deslice_fwd(const fs_problem* prob, const void* x, const float* Ws, const float* bias,
                   const float* tau, const float* zmix, const float* lse, void* out,
                   void* hip_stream);

/* Deslice with no saved normaliser, for a forward that runs no slice pass before it (forward
 * only inference; Sec. 2 and App. F.1, the per-point softmax over the G slots of Eq. (1)).
 * The maximum and the sum over the slots are formed per point inside the deslice kernel, the
 * weights normalised with them, and out (B,N,H,V) written as in fs_deslice_fwd.
 * lse_out (B,H,N) fp32, nullable: receives the base-2 normaliser of every point, the same
 * quantity fs_slice_fwd writes, for a later fs_slice_deslice_bwd. It must not overlap any
 * input or out (FS_ERR_ALIAS).                                                              */
int fs_deslice_stats_fwd(const fs_problem* prob, const void* x, const float* Ws,
                         const float* bias, const float* tau, const float* zmix, float* lse_out,
                         void* out, void* hip_stream);

/* Backward of slice -> mix -> deslice for the upstream gradient dout (B,N,H,V).
 * Inputs are the forward's inputs and saved z, s, zmix, attn_probs (ATTN only), lse.
 * Outputs: dx (B,N,H,D), dfx (B,N,H,V) in the storage dtype; dWs, dbias shaped like Ws,
 * bias; dtau (H); dmix_params as in fs_mix_bwd (nullable); dzmix_out (B,H,G,V) = w^T dout
 * (nullable). The temperature gradient follows App. F.2.                                    */
int fs_slice_deslice_bwd(const fs_problem* prob, const fs_mix_desc* mix, const void* x,
                         const void* fx, const float* Ws, const float* bias, const float* tau,
                         const float* z, const float* s, const float* zmix,
                         const float* attn_probs, const float* lse, const void* dout,
                         void* dx, void* dfx, float* dWs, float* dbias, float* dtau,
                         float* dmix_params, float* dzmix_out, void* ws, size_t ws_bytes,
                         void* hip_stream);

/* Backward of the untied variant (paper: Sec. 2 ablation suite, the deslice with its own
 * projection and temperature): the slice uses W_s (D,G), bias (G), tau (H) as everywhere
 * else, the deslice uses Wd, bd, taud of the same shapes (shared or per head with
 * ws_per_head), so its weights w_d = softmax_g((x Wd + bd) / taud) differ from the slice
 * weights w. The forward is fs_slice_fwd (W_s; lse), fs_mix, then fs_deslice_stats_fwd with
 * (Wd, bd, taud), which writes lse_d. Inputs as in fs_slice_deslice_bwd plus Wd, bd, taud
 * and lse_d. The deslice weights carry dw_d = dout zmix^T, the slice weights
 * dw = fx dU^T + 1 ds^T, each through its own softmax Jacobian and projection:
 * dx (B,N,H,D) = the sum of both projections' contributions; dfx (B,N,H,V) = w dU; dWs,
 * dbias, dtau from the slice weights and dWd, dbd, dtaud from the deslice weights (App. F.2
 * for both temperatures); dmix_params and dzmix_out (= w_d^T dout) as in
 * fs_slice_deslice_bwd. Workspace: fs_workspace_bytes(prob, 2, .). Every output is
 * overwritten; no output may overlap an input or another output.                          */
int fs_untied_bwd(const fs_problem* prob, const fs_mix_desc* mix, const void* x, const void* fx,
                  const float* Ws, const float* bias, const float* tau, const float* Wd,
                  const float* bd, const float* taud, const float* z, const float* s,
                  const float* zmix, const float* attn_probs, const float* lse,
                  const float* lse_d, const void* dout, void* dx, void* dfx, float* dWs,
                  float* dbias, float* dtau, float* dWd, float* dbd, float* dtaud,
                  float* dmix_params, float* dzmix_out, void* ws, size_t ws_bytes,
                  void* hip_stream);

/* LinearNO slice (paper: App. E and the Untied-LN row of the Sec. 2 ablation suite): the
 * slice weights are normalised by a softmax over the N points of each slot,
 * k[n, g] = exp(a[n, g]) / sum_n' exp(a[n', g]) with a = (x W_s + bias) / tau, and the tokens
 * are z_g = sum_n k[n, g] fx[n] (B,H,G,V), with no division by a weight sum. One streaming
 * pass with a running per-slot maximum; no N x G tensor is stored.
 * clse (B,H,G) fp32, nullable: the base-2 log normaliser of every slot over the points,
 * log2(sum_n 2^(a[n, g] log2 e)) (-inf for an empty point set, whose tokens are 0), needed by
 * fs_linearno_bwd. Workspace: fs_workspace_bytes(prob, 3, .).
 * The rest of the LinearNO forward is fs_mix (its layer uses FS_MIX_LINEAR_C) and
 * fs_deslice_stats_fwd with the deslice's own Wd, bd, taud (writing lse_d).                */
int fs_linearno_slice_fwd(const fs_problem* prob, const void* x, const void* fx,
                          const float* Ws, const float* bias, const float* tau, float* z,
                          float* clse, void* ws, size_t ws_bytes, void* hip_stream);

/* Backward of LinearNO. Inputs: the forward's inputs, Wd, bd, taud, and saved z, clse, zmix,
 * attn_probs (ATTN only), lse_d. The deslice weights carry dw_d = dout zmix^T (as in
 * fs_untied_bwd); the slice weights carry dk = fx dz^T through the softmax over the points,
 * da = k (dk - sum_n k dk) = k (fx dz^T - 1 (z . dz)^T). Outputs as in fs_untied_bwd: dx (both
 * projections' contributions), dfx = k dz, dWs, dbias (zero up to rounding: a constant added
 * to a slot's logits changes nothing), dtau, dWd, dbd, dtaud, dmix_params, dzmix_out.
 * Workspace: fs_workspace_bytes(prob, 4, .).                                               */
int fs_linearno_bwd(const fs_problem* prob, const fs_mix_desc* mix, const void* x, const void* fx,
                    const float* Ws, const float* bias, const float* tau, const float* Wd,
                    const float* bd, const float* taud, const float* z, const float* clse,
                    const float* zmix, const float* attn_probs, const float* lse_d,
                    const void* dout, void* dx, void* dfx, float* dWs, float* dbias,
                    float* dtau, float* dWd, float* dbd, float* dtaud, float* dmix_params,
                    float* dzmix_out, void* ws, size_t ws_bytes, void* hip_stream);

/* Measurement aid: for calls made later on this thread, record the caller's hipEvent_t
 * `before` immediately before, and `after` immediately after, the launch of the streaming
 * kernel of `pass` (0 slice, 1 deslice, 2 backward pass A, 3 backward pass B), on the stream
 * of that call. Each pass has its own pair; either event may be NULL; pass = -1 clears all
 * pairs. The events are only recorded (hipEventRecord), never synchronised or destroyed by
 * the library. Returns FS_ERR_ARG for an unknown pass.                                      */
int fs_set_pass_events(int pass, void* before, void* after);

/* Static text for a status code. */
const char* fs_status_string(int status);

/* hipError_t recorded by the last FS_ERR_HIP on this thread (0 if none). */
int fs_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FLASHSLICE_H */
