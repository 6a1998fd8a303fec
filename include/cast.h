/*
 * cast.h -- C ABI of libcast.so, the MI355X (gfx950) hot path of one
 * reconstruction-coupled DiT block step of CAST ("CAST: Reconstruction-Coupled
 * Acceleration of Interactive World Models").
 *
 * One block step at an eligible visual attention residual site is
 *
 *   cast_route_kv         pooled chunk scores and fixed-budget TopK over the
 *                         historical KV blocks                 (Sec. 4.4 eq:pooled, eq:topk)
 *   cast_anchor_attn      block-sparse attention of the anchor frames over the
 *                         routed blocks (plus an optional always-available
 *                         current/text segment)                 (Sec. 4.4, App. B.4)
 *   cast_par_reconstruct  Phase-Aware Reconstruction of every skipped frame's
 *                         residual from its two anchors         (Sec. 4.3 eq:cross,
 *                         eq:confidence, eq:gate, eq:fcpasm; App. A.2; eq:block)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.    Tensor arguments are DEVICE pointers owned by the caller; the library
 *            never allocates or frees device memory.  Scratch space is a caller-owned
 *            device `workspace` sized by the matching *_workspace_bytes() query
 *            (256-byte aligned).  `anchors` (PAR) is a small HOST array.
 * Layout.    Token-major, channel-fastest, densely packed, matching a DiT hidden
 *            state [frames, tokens, D] with D = H * dh head-major:
 *              Q       bf16 [n_a, S, H, dh]      (anchor frames only)
 *              K, V    bf16 [M, Bv, H, dh]       (M historical blocks of Bv tokens)
 *              resid   fp32 [n_frames, Hg, Wg, D]
 *            bf16 is IEEE binary32 truncated to its upper 16 bits (as torch.bfloat16).
 * Alignment. The bf16 tensors of the routing and attention calls (Q, K, V, the
 *            current segment, the attention output) and W_O / the Gram matrix are
 *            16-byte aligned; every other fp32 or int32 buffer is 4-byte aligned
 *            (the bf16 control inputs of cast_frame_select 2-byte aligned).  A
 *            misaligned buffer gives CAST_ERR_SHAPE.
 * Streams.   Every call only enqueues work on `stream` (NULL = the legacy default
 *            stream) and returns; nothing synchronises the host.  Asynchronous
 *            device faults surface at the caller's next stream synchronisation.
 * Errors.    Every call validates its arguments before enqueueing anything and
 *            returns a cast_status_t; it never throws or aborts across the ABI.
 *            cast_last_error_detail() gives a thread-local human-readable reason
 *            for the last non-OK status of the calling thread.
 * Threads.   Calls are re-entrant; the library holds no global mutable state other
 *            than the thread-local error detail and the per-GPU static scratch of
 *            cast_par_reconstruct_noalloc (see there).
 * Determinism. Results are bit-identical from run to run for identical inputs
 *            (fixed-order reductions, no floating-point atomics).
 */
#ifndef CAST_H_
#define CAST_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CAST_ABI_VERSION 2

typedef enum {
  CAST_OK = 0,
  CAST_ERR_NULL = 1,          /* a required pointer is NULL */
  CAST_ERR_SHAPE = 2,         /* a size is out of range or inconsistent */
  CAST_ERR_ANCHORS = 3,       /* anchors not strictly increasing in [0, n_frames), or K_f < 2 */
  CAST_ERR_UNSUPPORTED = 4,   /* valid request outside what the kernels implement */
  CAST_ERR_WORKSPACE = 5,     /* workspace NULL, misaligned or smaller than required */
  CAST_ERR_HIP = 6            /* a HIP launch or runtime call failed */
} cast_status_t;

/* Static string naming a status value. */
const char* cast_status_string(int status);

/* Thread-local detail of the calling thread's most recent non-OK status
 * (empty string if none).  Valid until the thread's next failing call. */
const char* cast_last_error_detail(void);

/* CAST_ABI_VERSION of the built library. */
int cast_abi_version(void);

/* ------------------------------------------------------------------------- */
/* Routing (Sec. 4.4 eq:pooled; eq:topk; App. B.3 budget rules)              */
/* ------------------------------------------------------------------------- */

/* Device scratch (bytes) needed by cast_route_kv for these sizes. */
size_t cast_route_kv_workspace_bytes(int n_a, int S, int H, int dh, int M, int Bv);

/*
 * Pooled chunk scores and TopK block selection, per (anchor frame i, head h):
 *
 *   q_bar[i,h,:] = mean over the S tokens of q[i,:,h,:]          (fp32 accumulation)
 *   k_bar[m,h,:] = mean over the Bv tokens of k_hist[m,:,h,:]   (fp32 accumulation)
 *   s[i,h,m]     = scale * dot(q_bar[i,h,:], k_bar[m,h,:])      (eq:pooled; the paper's
 *                                                                scale is 1/sqrt(dh))
 *   idx[i,h,:]   = the k_eff chunks with the largest s under the total order
 *                  (score descending, chunk index ascending), written in
 *                  ASCENDING chunk order; k_eff = min(topk, M) (App. B.3: with fewer
 *                  than topk blocks all are kept and the realised budget reported).
 *
 * q        bf16 [n_a, S, H, dh] device.      k_hist  bf16 [M, Bv, H, dh] device.
 * n_a>=1, S>=1, H>=1, dh in {32, 64, 128}, 0<=M<=4096, Bv>=1, topk>=1.
 * scores_out  fp32 [n_a, H, M] device, or NULL to skip.
 * idx_out     int32 [n_a, H, k_eff] device, densely packed (rows of k_eff entries,
 *             the layout cast_anchor_attn takes).  May be NULL only when M == 0.
 * k_eff_out   HOST int, receives k_eff (required).
 * M == 0: k_eff = 0 and nothing is enqueued (routing bypassed, App. B.3).
 * NaN scores give an unspecified but in-range selection.
 */
cast_status_t cast_route_kv(const void* q, const void* k_hist,
                            int n_a, int S, int H, int dh, int M, int Bv,
                            int topk, float scale,
                            float* scores_out, int32_t* idx_out, int* k_eff_out,
                            void* workspace, size_t workspace_bytes,
                            hipStream_t stream);

/* ------------------------------------------------------------------------- */
/* Reconstruction-coupled routing (Sec. 4.4 eq:omission..eq:topk; App. B:    */
/* eq:gain, eq:boundarygain, Algorithm 1; tab:config routing weights)        */
/* ------------------------------------------------------------------------- */

typedef struct {
  float l_anc, l_rec;   /* objective weights lambda_anc, lambda_rec (1, 1)          */
  int passes;           /* directional refinement passes L_s (2): forward, backward */
  float tol;            /* accept a change when J falls by > tol * max(J, 1e-8)
                           (1e-6)                                                   */
  float eps;            /* stabiliser of the omission proxy, eq:omission (1e-8)     */
} cast_coupled_params_t;

/* Fill *p with the defaults above.  NULL is ignored. */
void cast_coupled_params_default(cast_coupled_params_t* p);

/*
 * Gram matrices of the per-head output-projection slices, for the omission
 * proxy u = ||P_h delta||^2 = delta^T (P_h^T P_h) delta (eq:omission, P_h = the
 * head's slice of W_O).  They depend on the weights only: compute once per model.
 *   gram[h, a, b] = sum_r w_o[r, h*dh + a] * w_o[r, h*dh + b]   (fp32 accumulation)
 * w_o       bf16 [D, D] device, row-major, out = w_o @ concat_h(head outputs),
 *           D = H * dh.
 * gram_out  fp32 [H, dh, dh] device.
 * H>=1, dh in {32, 64, 128}, H*dh == D.
 */
cast_status_t cast_wo_gram(const void* w_o, int D, int H, int dh, float* gram_out,
                           hipStream_t stream);

/* Device scratch (bytes) needed by cast_route_coupled for these sizes. */
size_t cast_route_coupled_workspace_bytes(int n_a, int S, int H, int dh, int M, int Bv);

/*
 * Historical KV masks that couple neighbouring anchors through the frames they
 * reconstruct, per head h (masks of different heads never interact):
 *
 *   q_bar, k_bar, v_bar = token means (fp32) of q[i,:,h,:], k_hist[m,:,h,:],
 *                         v_hist[m,:,h,:];
 *   s[i,m] = scale q_bar[i].k_bar[m]; pi[i,:] = softmax over the M blocks;
 *   o_bar[i] = sum_m pi[i,m] v_bar[m];
 *   u[i,m] = (pi/(1-pi+eps))^2 (o_bar[i]-v_bar[m])^T gram[h] (o_bar[i]-v_bar[m])
 *                                                                (eq:omission)
 *   masks start as TopK_m(u[i,:]) and go through `passes` directional passes of
 *   Algorithm 1: anchor i's mask becomes TopK_m(G[i,:]) (eq:gain with the
 *   interval coefficients of eq:abc between adjacent anchors and the boundary
 *   coefficients of eq:boundarycoeff for frames before the first / after the
 *   last anchor, extrapolated from the first / last pair) when that lowers the
 *   head's objective J (eq:objective) by more than tol * max(J, 1e-8); a pass
 *   without a change ends the refinement.
 *
 * TopK orders (value descending, block index ascending); idx lists each mask in
 * ASCENDING block order, exactly k_eff = min(topk, M) blocks per (anchor, head),
 * the layout cast_anchor_attn takes.
 *
 * q        bf16 [n_a, S, H, dh] device (the anchor frames).
 * k_hist, v_hist  bf16 [M, Bv, H, dh] device.
 * gram     fp32 [H, dh, dh] device (cast_wo_gram).
 * anchors  HOST int [n_a], frame index of each row of q, strictly increasing,
 *          all in [0, n_frames); 1 <= n_a <= 512, n_a * M <= 32768.
 * u_out    fp32 [n_a, H, M] device, or NULL to skip.
 * idx_out  int32 [n_a, H, k_eff] device (may be NULL only when M == 0).
 * k_eff_out  HOST int, receives k_eff (required).
 * M == 0: k_eff = 0, nothing is enqueued.  topk >= M: every block is kept (the
 * refinement cannot change a full mask) but u is still computed.
 */
cast_status_t cast_route_coupled(const void* q, const void* k_hist, const void* v_hist,
                                 const float* gram, const int* anchors,
                                 int n_a, int n_frames, int S, int H, int dh, int M, int Bv,
                                 int topk, float scale, const cast_coupled_params_t* params,
                                 float* u_out, int32_t* idx_out, int* k_eff_out,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------- */
/* Routed block-sparse anchor attention (Sec. 4.4; App. B.4 complexity)      */
/* ------------------------------------------------------------------------- */

/*
 * For every anchor frame i and head h, with the key sequence
 *     [ k_cur[0..n0) ; k_hist[idx[i,h,0]] ; ... ; k_hist[idx[i,h,k_eff-1]] ]
 * of n0 + k_eff*Bv tokens (values likewise):
 *     out[i,s,h,:] = softmax_j(scale * q[i,s,h,:] . key_j) value_j
 * with fp32 logits, softmax and accumulation and bf16 output (the paper's BF16
 * QKV / FP32 softmax precision, tab:config).
 *
 * q        bf16 [n_a, S, H, dh] device.   k_hist, v_hist bf16 [M, Bv, H, dh] device.
 * idx      int32 [n_a, H, k_eff] device (as written by cast_route_kv); entries
 *          outside [0, M) are clamped into it so no access leaves k_hist/v_hist.
 * k_cur, v_cur  bf16 [n0, H, dh] device, the always-attended current/text segment;
 *          may be NULL when n0 == 0.
 * n0 >= 0, 0 <= k_eff <= min(M, 1024), n0 + k_eff*Bv >= 1; dh in {32, 64, 128};
 * scale finite and > 0; (n0 + k_eff*Bv) * Bv < 2^40 and n0 + k_eff*Bv < 2^24 * Bv;
 * k_hist, v_hist and k_cur, v_cur each smaller than 4 GiB.
 * out      bf16 [n_a, S, H, dh] device (must not alias the inputs).
 * lse_out  fp32 [n_a, H, S] device natural-log sum of exp of the scaled logits,
 *          or NULL to skip.
 * workspace  device scratch, or NULL.  The work is n_a * H * ceil(S / 256) units
 *          (anchor, head, 256-query tile).  With a workspace, the units of a last,
 *          at most half-full round on the device's compute units run as 2..8
 *          pieces over disjoint key ranges and are merged (the softmax of each
 *          piece renormalised by its log-sum-exp), which shortens that round;
 *          results agree with the unsplit run to fp32 rounding before the bf16
 *          output.  A non-NULL workspace must be 256-byte aligned and hold
 *          cast_anchor_attn_workspace_bytes(...) bytes (CAST_ERR_WORKSPACE
 *          otherwise); NULL runs every unit whole.  Owned by the caller; its
 *          contents need no initialisation and are garbage after the call.
 */
cast_status_t cast_anchor_attn(const void* q, const void* k_hist, const void* v_hist,
                               const int32_t* idx, int k_eff,
                               const void* k_cur, const void* v_cur, int n0,
                               int n_a, int S, int H, int dh, int M, int Bv,
                               float scale, void* out, float* lse_out,
                               void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes cast_anchor_attn uses for these sizes on the CURRENT device
 * (0: nothing is split, or the sizes are invalid, or no device is visible). */
size_t cast_anchor_attn_workspace_bytes(int n_a, int S, int H, int dh, int k_eff, int n0,
                                        int Bv);

/* ------------------------------------------------------------------------- */
/* Phase-Aware Reconstruction (Sec. 4.3; App. A.2; eq:block)                 */
/* ------------------------------------------------------------------------- */

typedef struct {
  int tile_h, tile_w;          /* disjoint spatial tiles, 1..8 each; default 8 x 8
                                  (tab:config_cast); edge tiles use their own size */
  float tau_low, tau_high;     /* eq:gate frequency prior, default 0.25, 0.75 */
  float q, T;                  /* eq:gate exponent and temperature, default 2, 0.10 */
  float eta_rel, eta_abs;      /* reliability threshold eta = eta_rel*max W + eta_abs,
                                  default 1e-6, 1e-8 (App. A.2) */
  float eps;                   /* eq:confidence stabiliser, default 1e-8 */
  int gate_mode;               /* 0: eq:gate; 1: g = 1 (full transport);
                                  2: g = 0 (linear interpolation / extrapolation) */
  int accumulate;              /* 0: out[t] = R_hat_t;  1: out[t] += R_hat_t, i.e.
                                  X_t <- X_t + R~_t of eq:block */
  int update_anchors;          /* 0: anchor slots of out are not touched;
                                  1: also the anchor case of eq:block, R~_a = R_a:
                                  out[a] = R_a (write) or out[a] += R_a (accumulate),
                                  fused into the reconstruction pass; out must then
                                  not overlap resid.  With accumulate = 1 one call
                                  is the whole update of one eligible residual site
                                  (visual attention or FFN) of a block. */
} cast_par_params_t;

/* Fill *p with the paper's settings (tab:config_cast, App. A.2), write mode,
   anchor slots untouched. */
void cast_par_params_default(cast_par_params_t* p);

/* Device scratch (bytes) needed by cast_par_reconstruct for these sizes. */
size_t cast_par_workspace_bytes(int n_frames, int n_anchor, int Hg, int Wg, int D,
                                const cast_par_params_t* params);

/*
 * Reconstruct the residual of every skipped frame t (t in [0, n_frames) not an
 * anchor) from its anchor pair per eq:block: interior t uses the bracketing
 * pair (a, b); t < a_0 uses (a_0, a_1); t > a_J uses (a_{J-1}, a_J);
 * alpha = (t - a)/(b - a), never clipped.  Per pair (a, b) and tile p:
 *   F = orthonormal 2-D real FFT of each channel of the tile (halved last axis),
 *   Z = sum_c F_b conj(F_a),  W = sum_c |F_b||F_a|          (eq:cross, all D channels)
 *   reliable: W > eta and |Z| > eta, eta = eta_rel * max_stored W + eta_abs;
 *   theta = Arg Z in (-pi, pi] on reliable representative bins, -theta on their
 *   mirrors, 0 on self-conjugate or unreliable bins;
 *   c_p = sum_{reliable, non-DC} kappa |Z| / (sum kappa W + eps), 0 if none
 *                                                        (eq:confidence);
 *   g = sigmoid((c_p - tau_low - (tau_high - tau_low) nu^q) / T)   (eq:gate);
 *   F_hat = (1-alpha) F_a e^{i g alpha theta} + alpha F_b e^{-i g (1-alpha) theta}
 *                                                        (eq:fcpasm);
 *   R_hat_t = inverse orthonormal real FFT, tiles assembled.
 *
 * resid    fp32 [n_frames, Hg, Wg, D] device; only the anchor frames are read.
 * anchors  HOST int[n_anchor], strictly increasing in [0, n_frames); n_anchor >= 2
 *          unless n_anchor == n_frames (K_f = N_cur: nothing to reconstruct, App.
 *          A.1; no work is enqueued unless update_anchors is set).  n_frames <= 4096, n_anchor <= 512.
 * out      fp32 [n_frames, Hg, Wg, D] device; only skipped-frame slots are
 *          written (or accumulated into); anchor slots are never touched.  `out`
 *          may be `resid` itself (write mode fills the skipped slots in place).
 * theta_out, gate_out  fp32 [n_anchor-1, n_tiles, tile_h*(tile_w/2+1)] device or
 *          NULL: per adjacent pair, tile and stored bin (ky*(tile_w/2+1)+kx) the
 *          transport phase and gate; entries past a smaller edge tile's bins are 0.
 *          n_tiles = ceil(Hg/tile_h) * ceil(Wg/tile_w), row-major.
 * conf_out fp32 [n_anchor-1, n_tiles] device or NULL: c_p per pair and tile.
 * Sizes: Hg, Wg >= 1; D >= 1; one frame Hg * Wg * D < 2^30 elements.
 */
cast_status_t cast_par_reconstruct(const float* resid, const int* anchors, int n_anchor,
                                   int n_frames, int Hg, int Wg, int D,
                                   const cast_par_params_t* params, float* out,
                                   float* theta_out, float* gate_out, float* conf_out,
                                   void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * cast_par_reconstruct for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same operation, arguments and results, with the scratch space taken from a
 * static array the library holds on each GPU (CAST_PAR_STATIC_SCRATCH_BYTES, 16
 * MiB, kept until the process ends) instead of a caller workspace.  The call
 * allocates and frees nothing; its device address is looked up once per device on
 * the first call made with that device current.
 * Sizes whose cast_par_workspace_bytes exceeds cast_par_static_scratch_bytes()
 * return CAST_ERR_WORKSPACE (enqueueing nothing).  Every call on one GPU shares
 * that GPU's array and overwrites it before reading it: calls that overlap on one
 * GPU (two streams, or two host threads without ordering) race and must be
 * serialised by the caller.
 */
#define CAST_PAR_STATIC_SCRATCH_BYTES (16u << 20)
cast_status_t cast_par_reconstruct_noalloc(const float* resid, const int* anchors, int n_anchor,
                                           int n_frames, int Hg, int Wg, int D,
                                           const cast_par_params_t* params, float* out,
                                           float* theta_out, float* gate_out, float* conf_out,
                                           hipStream_t stream);

/* Bytes of the static scratch of cast_par_reconstruct_noalloc on each GPU. */
size_t cast_par_static_scratch_bytes(void);

/* ------------------------------------------------------------------------
 * Control-aware frame selection (Sec. 3.1 eq:sensitivity; Sec. 4.2 eq:debt,
 * eq:score; App. A.1 eq:normalization and the scheduling rules)
 * ------------------------------------------------------------------------ */
typedef struct {
  float lambda_cov;   /* weight of the coverage debt: 0.5 (Sec. 4.2, tab:config_cast) */
  float eps;          /* stabiliser of the min-max normalisation: 1e-8 */
} cast_select_params_t;

/* Fill *p with the paper's settings. */
void cast_select_params_default(cast_select_params_t* p);

/* Device scratch (bytes) needed by cast_frame_select (0 when no branch is given). */
size_t cast_frame_select_workspace_bytes(int n_cur, int S, int D);

/*
 * Choose the anchors of the next transformer block after the current block ran
 * with anchors_prev and its control branches produced the feature updates
 * delta_cam and delta_act:
 *   r_{i,k} = RMS of delta_k[i] over the frame's tokens and channels;
 *   Norm_k = (r_k - min r_k) / (max r_k - min r_k + eps) over the N_cur frames;
 *   d_i = mean of Norm_k over the branches given (an absent branch is left out);
 *   ages: h_i = 0 for i in anchors_prev, h_i + 1 otherwise;
 *   D_i = h_i / ceil(N_cur / K_f);  S_i = d_i + lambda_cov D_i, or lambda_cov D_i
 *   when neither branch is given (no fresh control response);
 *   anchors = the K_f largest S_i, ties by increasing frame index.
 * Every step after r is fp32 with one rounding per operation (no contraction);
 * r is the fp32 rounding of the square root of the mean of squares.
 *
 * delta_cam, delta_act  device [n_cur, S, D] of dtype (0: fp32, 1: bf16), frame-
 *          major, channel-fastest; either or both may be NULL (absent branch).
 * n_cur    current frames, 1 .. 4096;  S, D >= 1.
 * anchors_prev  HOST int[n_prev], strictly increasing in [0, n_cur), n_prev >= 1:
 *          the anchors the block ran with (all frames after a dense block, which
 *          resets every age).
 * k_f      anchors to choose, 1 .. n_cur.
 * ages     device int32[n_cur], in/out: refresh ages before the block in, after
 *          it out (start from zeros; the dense first block resets them anyway).
 * r_out    device fp32[2, n_cur] or NULL: r per branch (row 0 camera, row 1
 *          action; the row of an absent branch is not written).
 * score_out  device fp32[n_cur] or NULL: S_i.
 * anchors_out  device int32[k_f]: the chosen frames, ascending.
 * workspace  device, 256-byte aligned, >= cast_frame_select_workspace_bytes.
 * Errors: CAST_ERR_NULL (ages, anchors_out, params or anchors_prev missing),
 * CAST_ERR_SHAPE (sizes, dtype, misaligned buffers, negative weights),
 * CAST_ERR_ANCHORS (anchors_prev not strictly increasing in range),
 * CAST_ERR_UNSUPPORTED (n_cur > 4096), CAST_ERR_WORKSPACE.
 */
cast_status_t cast_frame_select(const void* delta_cam, const void* delta_act, int dtype,
                                int n_cur, int S, int D, const int* anchors_prev, int n_prev,
                                int k_f, const cast_select_params_t* params, int32_t* ages,
                                float* r_out, float* score_out, int32_t* anchors_out,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Spectral diagnostics of reconstructed residuals (App. C eq:oracles,
 * eq:bandenergy, eq:phaseerror; the relative error e_t of Sec. 3.1
 * eq:sensitivity).  Reference-based: for validation, not for inference.
 * ------------------------------------------------------------------------ */
typedef struct {
  int tile_h, tile_w;       /* the PAR tiling (disjoint tiles, edge tiles at their own size): 8, 8 */
  int n_bands;              /* radial bands, 1 .. 8 */
  float band_edges[9];      /* ascending, band_edges[0] = 0, band_edges[n_bands] = 1: band k holds
                               the bins with band_edges[k] <= nu < band_edges[k+1] (nu = PAR's
                               normalised radius; nu = 1 falls in the last band) */
  float eps;                /* 1e-8 */
} cast_diag_params_t;

/* 8x8 tiles, three bands with edges (0, 1/3, 2/3, 1), eps = 1e-8. */
void cast_diag_params_default(cast_diag_params_t* p);

/* Device scratch (bytes) needed by cast_spectral_diagnostics. */
size_t cast_spectral_diagnostics_workspace_bytes(int n_frames, int Hg, int Wg, int D,
                                                 const cast_diag_params_t* params);

/*
 * For every skipped frame t of eq:block (pair (a, b), alpha = (t - a)/(b - a)):
 *   nrmse_out[t]  = ||R_t - R_hat_t|| / (||R_t|| + eps) over the frame;
 *   band_out[t,k] = sum_{tiles, channels, bins in band k} kappa |F_t - F_hat_t|^2
 *                   / (sum over all bins + eps)                        (eq:bandenergy);
 *   phase_err_out[t] = sum w |wrap_[-pi,pi)(Arg F_t - Arg F_a - alpha theta_p)| / (sum w + eps),
 *                   w = kappa |F_t|^2 on bins where F_t and F_a are nonzero    (eq:phaseerror);
 *   r_phase_out[t], r_mag_out[t] = inverse transforms of |F_lin| e^{i Arg F_t} and
 *                   |F_t| e^{i Arg F_lin}, F_lin = (1 - alpha) F_a + alpha F_b  (eq:oracles).
 * F is the orthonormal real 2-D DFT per tile and channel, kappa the real-FFT
 * multiplicity (1 on the columns that hold their own conjugates, 2 elsewhere).
 * Entries of anchor frames are 0; r_phase_out / r_mag_out slots of anchors are not
 * written.
 *
 * ref      fp32 [n_frames, Hg, Wg, D] device: reference residuals of every frame
 *          (anchors included).
 * approx   fp32 [n_frames, Hg, Wg, D] device: the reconstructions R_hat_t (skipped
 *          slots read; e.g. the output of cast_par_reconstruct in write mode).
 * theta    fp32 [n_anchor - 1, tiles, tile_h * (tile_w/2 + 1)] device: the transport
 *          phases of the pairs (theta_out of cast_par_reconstruct with the same
 *          tiling), or NULL: then phase_err_out is not written.
 * anchors  HOST int[n_anchor], strictly increasing in [0, n_frames), n_anchor >= 2.
 * nrmse_out [n_frames], band_out [n_frames, n_bands], phase_err_out [n_frames],
 *          r_phase_out, r_mag_out [n_frames, Hg, Wg, D]: device, each may be NULL.
 * Errors: CAST_ERR_NULL (ref, approx, anchors, params), CAST_ERR_SHAPE (sizes,
 * bands, misaligned buffers), CAST_ERR_ANCHORS, CAST_ERR_UNSUPPORTED (tile edges
 * above 8, n_frames > 4096, n_anchor > 512), CAST_ERR_WORKSPACE.
 */
cast_status_t cast_spectral_diagnostics(const float* ref, const float* approx, const float* theta,
                                        const int* anchors, int n_anchor, int n_frames, int Hg,
                                        int Wg, int D, const cast_diag_params_t* params,
                                        float* nrmse_out, float* band_out, float* phase_err_out,
                                        float* r_phase_out, float* r_mag_out, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream);

/*
 * Phase progress of every coefficient (App. C eq:phase_progress), for the interior
 * frames of each adjacent anchor pair (a, b): with F_t the orthonormal real 2-D
 * DFT of tile p and channel c of ref[t] (params->tile_h x tile_w tiles, edge tiles
 * at their own size) and, for each stored bin (ky, kx), the phase unwrapped along
 * the frames,
 *   u_a = 0,  u_t = u_{t-1} + wrap_[-pi,pi)(Arg F_t - Arg F_{t-1})  (t = a+1 .. b),
 *   p_out[t, p, ky * (tile_w/2 + 1) + kx, c] = u_t / u_b          (a < t < b).
 * Uniform progression gives alpha = (t - a)/(b - a) (eq:shift).  Entries of
 * anchor frames, of frames before the first or after the last anchor, and of slots
 * past a smaller edge tile's bins are not written; a vanishing displacement u_b
 * gives +-inf or NaN (IEEE division).
 *
 * ref      fp32 [n_frames, Hg, Wg, D] device: residuals of every frame.
 * anchors  HOST int[n_anchor], strictly increasing in [0, n_frames), n_anchor >= 2.
 * params   the tiling (tile_h, tile_w); the band fields must be valid but are unused.
 * p_out    fp32 [n_frames, n_tiles, tile_h * (tile_w/2 + 1), D] device,
 *          n_tiles = ceil(Hg/tile_h) * ceil(Wg/tile_w), row-major.
 * Errors: CAST_ERR_NULL (ref, anchors, params, p_out), CAST_ERR_SHAPE (sizes,
 * misaligned buffers), CAST_ERR_ANCHORS, CAST_ERR_UNSUPPORTED (tile edges above 8,
 * n_frames > 4096, n_anchor > 512).  Reference-based: for validation, not inference.
 */
cast_status_t cast_phase_progress(const float* ref, const int* anchors, int n_anchor, int n_frames,
                                  int Hg, int Wg, int D, const cast_diag_params_t* params,
                                  float* p_out, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* CAST_H_ */
