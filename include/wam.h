/*
 * libwam — MI355X (gfx950) hot path of training-free World Action Model
 * inference with adaptive intermediate states.
 *
 * The library runs the iterative flow-denoising step of a DiT-style joint
 * video-latent + action-token transformer, and the three state-adaptation
 * operators that let a replan continue from retained state instead of
 * re-denoising from noise:
 *
 *   Trajectory Remapping  (Sec. 3.1, Eq. direction and Eq. transport, with the
 *                          unit-RMS normalisation of Eq. app-transport-rms),
 *   Observation Rebinding (Sec. 3.2, Eq. bind-discrepancy and the kappa rule),
 *   Residual Rescaling    (Sec. 3.3, Eq. crr-reference, crr-alpha, crr-gate,
 *                          residual-injection and refresh on failure),
 *
 * coordinated as in Sec. 3.4 (joint runtime).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Ownership: the caller allocates every device buffer (packed weights,
 *    workspace, trajectories, conditions, noise, outputs) and keeps it alive
 *    while the handle uses it.  The library never allocates device memory; the
 *    retained-state cache lives inside the caller's workspace.  Host pointers
 *    are only read during the call.
 *  - Streams: all device work is enqueued on the hipStream_t given to
 *    wam_init.  Calls that need a host-side decision (Residual Rescaling gate,
 *    Observation Rebinding score) synchronise that stream before returning;
 *    the others are asynchronous.
 *  - Randomness: the library draws no random numbers.  Noise is an input.
 *  - Layouts (all row-major, all device float32 unless stated):
 *      trajectory  x [B][traj], traj = Nv*Cv + Na*A, per sample
 *                  [video tokens (Nv x Cv) | action tokens (Na x A)];
 *      condition   cond [B][No][Co] (observation-conditioning tokens);
 *      hidden      h [B][T][D] with T = Nv + Na + No rows ordered
 *                  [video | action | observation].
 *  - Errors: every int-returning call returns WAM_OK (0) or a negative status
 *    and, given a handle, stores a message for wam_last_error.  Nothing throws
 *    across the ABI.  A failing call leaves retained state unchanged unless
 *    documented otherwise.
 *  - Threading: a handle is used by one host thread at a time.
 */
#ifndef WAM_H
#define WAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------- */
#define WAM_OK 0
#define WAM_E_ARG (-1)         /* invalid scalar argument or null pointer     */
#define WAM_E_SHAPE (-2)       /* model dimensions not supported / mismatched */
#define WAM_E_STATE (-3)       /* call not valid in the handle's state        */
#define WAM_E_HIP (-4)         /* HIP runtime error                           */
#define WAM_E_WORKSPACE (-5)   /* weight or workspace buffer too small        */
#define WAM_E_UNSUPPORTED (-6) /* valid request the library does not implement */

/* ---- numeric modes --------------------------------------------------- */
#define WAM_FP32 0 /* all activations and contractions in float32            */
#define WAM_BF16 1 /* projection / attention operands bf16, fp32 accumulate;
                      residual stream, trajectory, layer state, norms and all
                      reductions stay float32 (or float64 for gate sums)      */

/* ---- Residual Rescaling modes ------------------------------------------ */
#define WAM_RR_OFF 0        /* plain full forward, no layer state kept        */
#define WAM_RR_AUTO 1       /* gate of Eq. crr-gate decides reuse or refresh  */
#define WAM_RR_FORCE_SKIP 2 /* reuse whenever a layer state exists            */
#define WAM_RR_FORCE_FULL 3 /* always compute the middle and refresh          */
/* wam_rr_profile.branches */
#define WAM_RR_JOINT 0  /* video (+ observation) and action rows: two checks */
#define WAM_RR_SINGLE 1 /* all rows: one check                                */

/* ---- wam_adapt_state operations ---------------------------------------- */
#define WAM_ADAPT_REMAP 1       /* args: const wam_remap_args*               */
#define WAM_ADAPT_RESET_LAYER 2 /* args: NULL; drop retained (p_a, R_a)      */
#define WAM_ADAPT_RESET_ALL 3   /* args: NULL; drop layer and replan state   */
#define WAM_ADAPT_SET_REPLAN 4  /* args: const wam_replan_state_args*        */
#define WAM_ADAPT_REBIND 5      /* args: const wam_rebind_args*              */

/* ---- replan paths (Sec. 3.4) ------------------------------------------- */
#define WAM_PATH_FIRST 0  /* first replan: K steps from fresh noise           */
#define WAM_PATH_ACCEPT 1 /* prefix under the predicted condition, rebound    */
#define WAM_PATH_REJECT 2 /* prefix failed the check: restart under c         */
#define WAM_PATH_FORCED 3 /* kappa reached kappa_max: refresh, no prefix      */
#define WAM_PATH_DIRECT 4 /* rebinding disabled: K-b0 steps under c           */

/* ---- wam_set_option ------------------------------------------------------ */
#define WAM_OPT_DEVICE_DECISION 1 /* 1: the Residual Rescaling decision stays on the
                                     device; the gate writes a flag that predicates
                                     the inject / middle / refresh launches, and step
                                     reports are read back once per call (default 0:
                                     the host reads the gate and launches one path) */
#define WAM_OPT_GRAPHS 2          /* 1: wam_replan replays one captured graph per
                                     (stage, RR variant); needs the device decision
                                     and a non-default stream; graphs are re-captured
                                     when the schedule or the RR profile changes */
#define WAM_OPT_ATTENTION 3       /* bf16 attention kernel (WAM_ATTN_*); every form
                                     gives the same result up to rounding */
#define WAM_ATTN_AUTO 0           /* default: a bounded form where the layer allows
                                     it (tile shape chosen by sequence length and
                                     grid size), else the running max */
#define WAM_ATTN_RUNNING_MAX 1    /* online softmax with a running maximum          */
#define WAM_ATTN_BOUNDED 2        /* QK-norm bounds every score by mref <= 60 (log2
                                     units, from the gains): mref is the fixed
                                     softmax reference, no running max; software-
                                     pipelined loop (QK of the next key tile
                                     issued before PV of this one)                 */
#define WAM_ATTN_PINGPONG 3       /* bounded, 8 waves in two groups that alternate
                                     MFMA and exp2 phases on each SIMD            */
#define WAM_ATTN_PLAIN 4          /* bounded, plain loop (one score buffer, more
                                     waves per SIMD); on grids too small to fill
                                     the chip, two wave groups split the keys and
                                     add their partial sums                      */
/* A bounded form asked for on a layer whose gains allow no bound (mref > 60)
   runs the running-max kernel. */

#define WAM_MAX_BATCH 16
#define WAM_MAX_COMPONENTS 8
#define WAM_MAX_STEPS 64

/* Kernel classes for wam_profile_* (per-launch timing from dispatch timestamps). */
#define WAM_KC_GEMM_QKV 0
#define WAM_KC_GEMM_PROJ 1
#define WAM_KC_GEMM_FC1 2
#define WAM_KC_GEMM_FC2 3
#define WAM_KC_ATTENTION 4
#define WAM_KC_RR_GATE 5
#define WAM_KC_RR_INJECT 6
#define WAM_KC_RR_REFRESH 7
#define WAM_KC_COUNT 8

typedef struct wam_handle *wam_t;

/* Model configuration.  D % 64 == 0 (D <= 2048), D % H == 0, head size D/H in
 * {32, 64}, Cv <= 16, A <= 16, Co <= 64; bf16 mode additionally needs
 * D/H == 64 and F % 128 == 0 (any head count, odd ones included).  Nv >= 0, Na >= 0, Nv + Na >= 1:
 * a model of an independently executed pair has only video (Na = 0) or only
 * action (Nv = 0) tokens; Cv and A stay >= 1 (their weights exist). */
typedef struct {
  int32_t B;       /* batch (samples denoised together), 1..WAM_MAX_BATCH */
  int32_t L;       /* DiT layers                                            */
  int32_t D;       /* hidden size                                           */
  int32_t H;       /* attention heads                                       */
  int32_t F;       /* MLP hidden size                                       */
  int32_t Nv, Cv;  /* video-latent tokens, channels per token               */
  int32_t Na, A;   /* action tokens (chunk length), action dimension        */
  int32_t No, Co;  /* observation tokens, channels per token                */
  int32_t dtype;   /* WAM_FP32 | WAM_BF16                                   */
  int32_t qk_norm; /* 1: RMS-normalise q and k per head (with gains)        */
  float ln_eps;    /* epsilon of LayerNorm and QK RMSNorm                   */
} wam_config;

/* Residual Rescaling profile (Sec. 3.3; thresholds as in Table app-guards).
 * Layer boundaries 0 < q < s < e < L partition the DiT into head [0,q),
 * probe [q,s), middle [s,e) and tail [e,L). */
typedef struct {
  int32_t q, s, e;
  int32_t mode; /* WAM_RR_* */
  float alpha_min, alpha_max, eps;
  float gamma_cos, gamma_fit;
  /* WAM_RR_JOINT: the jointly executed video (+ observation) and action
   * branches each get an alpha, and the middle is skipped only when both
   * pass (Sec. 3.3, joint execution).  WAM_RR_SINGLE: the model's whole token
   * set is one branch, as for each model of an independently executed video /
   * action pair (Sec. 3.3, independent execution; the branch-1 statistics of
   * wam_step_info are then NaN). */
  int32_t branches;
} wam_rr_profile;

/* Per-denoising-step report.  alpha/cos/fit are per sample and per branch
 * (branch 0 = video and observation rows, 1 = action rows; with
 * WAM_RR_SINGLE branch 0 = all rows and branch 1 = NaN); valid when
 * rr_attempted. */
typedef struct {
  int32_t rr_active;    /* RR mode was not OFF                              */
  int32_t rr_attempted; /* a retained state existed and the gate was run    */
  int32_t rr_accepted;  /* the middle layers were skipped                   */
  int32_t layers_evaluated;
  int32_t layers_skipped;
  int32_t reserved;
  double alpha[WAM_MAX_BATCH][2];
  double cos[WAM_MAX_BATCH][2];
  double fit[WAM_MAX_BATCH][2];
} wam_step_info;

/* Trajectory Remapping arguments (Eq. direction, Eq. transport). */
typedef struct {
  const float *x_bar; /* device [B][traj]: final output of the previous replan  */
  const float *x_r;   /* device [B][traj]: latent retained at stage r           */
  float sigma_r;      /* noise level of stage r, must be > 0                    */
  float sigma_b0;     /* noise level of the entry stage b0                      */
  int32_t shift_action; /* target action slot j takes source slot j+shift (>=0) */
  int32_t shift_video;  /* same for video tokens (>=0)                          */
  const float *noise; /* device [B][traj] N(0,1); unmapped slots get sigma_b0*noise */
  float *x_out;       /* device [B][traj]: remapped initialisation              */
} wam_remap_args;

/* Observation Rebinding's rebinding step (Sec. 3.2): the retained denoising
 * state (the working latent an anticipatory prefix produced under the
 * predicted condition c_hat, the latent captured at stage r, and the Residual
 * Rescaling layer state, which persists across the rebinding point, Sec. 3.3)
 * continues under the real condition c.  The library copies cond into its own
 * condition buffer (stream-ordered; the caller's buffer may be reused once the
 * stream passes this point) and from then on a NULL cond in wam_velocity,
 * wam_denoise_step, wam_continue and wam_hidden means that bound condition.
 * Nothing else of the retained state changes; the rebinding counter kappa
 * and the decision S < tau and kappa < kappa_max belong to wam_replan, which
 * performs the same step on its accept path (and leaves its real condition
 * bound after every replan).  cond: device [B][No][Co], may be NULL only when
 * No == 0.  WAM_E_ARG for a NULL cond otherwise. */
typedef struct {
  const float *cond;
} wam_rebind_args;

/* Adopt an externally held replan state (teacher forcing / resume). */
typedef struct {
  const float *x_bar; /* device [B][traj] */
  const float *x_r;   /* device [B][traj] */
  int32_t kappa;
} wam_replan_state_args;

/* One closed-loop replan (Sec. 3.4). */
typedef struct {
  const float *cond_real; /* device [B][No][Co]: real condition c_{t+1}          */
  const float *cond_pred; /* device [B][No][Co]: predicted condition (OR prefix) */
  /* consistency components compared before encoding (Eq. bind-discrepancy) */
  int32_t n_components;
  const float *u_hat[WAM_MAX_COMPONENTS]; /* device, n[m] floats each         */
  const float *u[WAM_MAX_COMPONENTS];
  int64_t n[WAM_MAX_COMPONENTS];
  double delta[WAM_MAX_COMPONENTS];
  double weight[WAM_MAX_COMPONENTS];
  const float *noise_first; /* device [B][traj] N(0,1): first replan's x at sigma_0 */
  const float *noise_remap; /* device [B][traj] N(0,1): unmapped slots / fresh init */
  float *x_out;             /* device [B][traj]: receives the new x_bar             */
  wam_rr_profile rr;
  int32_t b0, r;             /* entry stage and retained stage, b0 <= r < K    */
  int32_t shift_action, shift_video;
  int32_t k1;                /* anticipatory prefix steps, 0 < k1 < K-b0       */
  double tau;                /* accept iff S < tau and kappa < kappa_max       */
  int32_t kappa_max;
  int32_t tr_enabled, or_enabled;
  int32_t rr_first, rr_prefix, rr_refresh; /* RR allowed on each path       */
} wam_replan_args;

typedef struct {
  int32_t path;  /* WAM_PATH_* */
  int32_t kappa; /* after this replan */
  int32_t steps; /* denoising steps executed (prefix + continuation/restart) */
  int32_t n_start, n_bind; /* 0/1 for this replan (Eq. app-rebinding-rates) */
  int32_t rr_attempts, rr_reuses, layers_skipped, layers_dense;
  int32_t reserved;
  double S; /* consistency score, or -1 when no prefix was checked */
  int8_t decision[WAM_MAX_STEPS]; /* per step: -1 no attempt, 0 refresh, 1 reuse */
} wam_replan_info;

/* ---- sizes --------------------------------------------------------------- */
/* Number of float32 values of the canonical host weight buffer, which holds,
 * each row-major with Linear weights stored [in][out] (y = x W + b):
 *   t_w1[256][D] t_b1[D] t_w2[D][D] t_b2[D]
 *   in_wv[Cv][D] in_bv[D] in_wa[A][D] in_ba[D] in_wo[Co][D] in_bo[D]
 *   for each layer l: mod_w[D][6D] mod_b[6D] qkv_w[D][3D] qkv_b[3D]
 *                     q_g[dh] k_g[dh] proj_w[D][D] proj_b[D]
 *                     fc1_w[D][F] fc1_b[F] fc2_w[F][D] fc2_b[D]
 *   f_mod_w[D][2D] f_mod_b[2D] out_wv[D][Cv] out_bv[Cv] out_wa[D][A] out_ba[A]
 * Returns 0 for an invalid configuration. */
size_t wam_host_weight_count(const wam_config *cfg);
/* Device bytes of the packed weights (with the constant position-embedding
 * table) and of the workspace (0 if invalid). */
size_t wam_weight_bytes(const wam_config *cfg);
size_t wam_workspace_bytes(const wam_config *cfg);
/* Trajectory elements per sample, Nv*Cv + Na*A. */
int64_t wam_traj_elems(const wam_config *cfg);

/* ---- lifetime ------------------------------------------------------------ */
/* Validates cfg, converts and packs the host weights (bf16 mode: projection
 * and modulation matrices rounded to bf16, nearest-even) into dev_weights,
 * carves the workspace, and returns a handle.  Synchronous. */
int wam_init(const wam_config *cfg, const float *host_weights, size_t n_host_weights,
             void *dev_weights, size_t weight_bytes, void *dev_workspace,
             size_t workspace_bytes, void *hip_stream, wam_t *out);
void wam_destroy(wam_t h);
int wam_sync(wam_t h);
const char *wam_last_error(wam_t h);
const char *wam_status_string(int status);
/* Execution options (WAM_OPT_*); results are identical either way up to the
 * order of independent work.  Returns WAM_E_STATE for an invalid combination
 * and WAM_E_UNSUPPORTED for graphs on the default (null) stream. */
int wam_set_option(wam_t h, int option, int value);

/* Noise levels sigma_0 = 1 > ... > sigma_K = 0 of the flow schedule
 * (host float[K+1]); K <= WAM_MAX_STEPS.  Required before any step. */
int wam_set_schedule(wam_t h, const float *sigmas, int K);

/* ---- denoising ------------------------------------------------------------ */
/* Denoiser prediction v(x, sigma_k, cond) into v_out [B][traj]; runs the
 * embedding, the L DiT layers (with Residual Rescaling per rr, which may be
 * NULL = off), the final layer and the output heads.  Updates the retained
 * layer state as Sec. 3.3 prescribes. */
int wam_velocity(wam_t h, int k, const float *x, const float *cond, float *v_out,
                 const wam_rr_profile *rr, wam_step_info *info);
/* One Euler step of the flow ODE: x <- x + (sigma_{k+1} - sigma_k) v. */
int wam_denoise_step(wam_t h, int k, float *x, const float *cond,
                     const wam_rr_profile *rr, wam_step_info *info);
/* Steps k_from .. k_to-1 in place on x.  If k_from <= capture_stage <= k_to
 * the latent at that stage is copied to x_capture (device [B][traj]).
 * infos may be NULL or hold k_to - k_from entries. */
int wam_continue(wam_t h, int k_from, int k_to, float *x, const float *cond,
                 const wam_rr_profile *rr, int capture_stage, float *x_capture,
                 wam_step_info *infos);
/* Hidden state after the first n_layers layers (no RR) at stage k into
 * h_out [B][T][D]; for layer-level parity checks. */
int wam_hidden(wam_t h, int k, const float *x, const float *cond, int n_layers, float *h_out);

/* ---- state adaptation ------------------------------------------------------ */
int wam_adapt_state(wam_t h, int op, const void *args);
/* Observation Rebinding score (Eq. bind-discrepancy) over device arrays,
 * accumulated in float64: S = sqrt(sum w e^2 / sum w),
 * e_m = sqrt(mean(((u_hat_m - u_m)/delta_m)^2)).  u_hat[m], u[m]: device
 * float[n[m]], caller-owned; n_components in 1..WAM_MAX_COMPONENTS, n >= 1,
 * delta > 0, weight >= 0 with a positive sum (else WAM_E_ARG).  The squared
 * differences are summed on the device in runs (float64, fixed order) and the
 * run sums on the host.  Only this device form exists: the components are the
 * condition tensors, which already live on the device.  Uses the handle's
 * stream and workspace; synchronises. */
int wam_consistency_score(wam_t h, int n_components, const float *const *u_hat,
                          const float *const *u, const int64_t *n, const double *delta,
                          const double *weight, double *S_out);
/* Condition tokens of the action model of an independently executed video /
 * action pair (Sec. 3.3; the action model reads the observation and the video
 * model's latent): cond [B][No][Co] = the n_obs observation tokens obs
 * [B][n_obs][c_obs] followed by the n_ctx tokens of ctx (sample b, token j,
 * channel c at ctx[b * ctx_stride + j * c_ctx + c], e.g. the video part of
 * the video model's trajectory), each zero-padded to Co channels.  Needs
 * n_obs + n_ctx == No and c_obs, c_ctx <= Co.  Device pointers, caller-owned;
 * enqueued on the handle's stream (no synchronisation). */
int wam_pack_condition(wam_t h, const float *obs, int n_obs, int c_obs, const float *ctx, int n_ctx,
                       int c_ctx, int64_t ctx_stride, float *cond);
/* One replan of the joint runtime.  The first call (or after RESET_ALL) runs
 * the native K steps from noise_first; later calls apply Trajectory
 * Remapping, the anticipatory prefix under cond_pred, the consistency check
 * and rebinding or restart, with Residual Rescaling inside each step.  The
 * retained replan state (x_bar, x^r, kappa) lives in the workspace. */
int wam_replan(wam_t h, const wam_replan_args *args, wam_replan_info *info);
/* The same replan in two halves, so that the anticipatory prefix overlaps
 * action execution (Sec. 3.2).  wam_replan_begin applies Trajectory Remapping
 * and enqueues the prefix under cond_pred; with WAM_OPT_DEVICE_DECISION it
 * returns without waiting for the GPU.  wam_replan_end, called once the real
 * observation is available, computes the consistency score, rebinds or
 * restarts under cond_real, and fills info.  Both take the same args (the
 * buffers must stay valid until wam_replan_end returns); wam_replan_end
 * without a begin runs the whole replan.  A second begin before end is
 * WAM_E_STATE. */
int wam_replan_begin(wam_t h, const wam_replan_args *args);
/* While a replan is open (after wam_replan_begin, before wam_replan_end) the
 * other calls that touch the handle's state (wam_velocity, wam_denoise_step,
 * wam_continue, wam_hidden, wam_adapt_state except RESET_ALL,
 * wam_consistency_score, wam_get_replan_state, wam_set_schedule,
 * wam_set_option) return WAM_E_STATE; RESET_ALL abandons the open replan. */
int wam_replan_end(wam_t h, const wam_replan_args *args, wam_replan_info *info);
/* Copies of the retained replan state (device [B][traj] each; may be NULL). */
int wam_get_replan_state(wam_t h, float *x_bar, float *x_r, int32_t *kappa);

/* Trajectory Remapping that allocates nothing, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same computation and kernels as
 * wam_adapt_state(WAM_ADAPT_REMAP), without a handle.  From cfg only B, Nv,
 * Cv, Na and A are read (1 <= B <= WAM_MAX_BATCH, Nv, Na >= 0, Nv + Na >= 1,
 * Cv, A >= 1, B * traj < 2^31); args as for WAM_ADAPT_REMAP (device buffers,
 * caller-owned).  Enqueued on hip_stream (NULL: the default stream) with no
 * synchronisation.  The reduction scratch (at most WAM_MAX_BATCH x 2 x 1025
 * float64, 256.3 KiB) is a static array of the library on each GPU, held until
 * the process ends; every call on one GPU shares it, so calls that overlap on
 * one GPU (different streams or threads) race.  The call makes no device
 * allocation and no hipMalloc / hipFree.  Errors: WAM_E_SHAPE for sizes
 * beyond those limits, WAM_E_ARG for invalid arguments, WAM_E_HIP for a
 * runtime error; wam_noalloc_last_error() returns this thread's message of
 * the last failing call. */
int wam_remap_noalloc(const wam_config *cfg, const wam_remap_args *args, void *hip_stream);
const char *wam_noalloc_last_error(void);

/* ---- measurement ------------------------------------------------------------ */
/* Time every launch of kernel class kc (WAM_KC_*), up to max_launches
 * launches: a HIP event pair per launch, stamped by the dispatches themselves
 * (begin of the class's first kernel, end of its last; hipExtLaunchKernel), so
 * no event packets sit between the timed kernels.  Launches inside a graph
 * capture are not timed.  enable = 0 stops. */
int wam_profile_enable(wam_t h, int kc, int enable, int max_launches);
/* Sum of launch durations (ms), launch count and algorithmic work (FLOP for
 * contractions, bytes for streaming kernels) of the recorded launches.
 * Synchronises. */
int wam_profile_read(wam_t h, int kc, double *total_ms, int64_t *launches, double *work);

/* Achievable-peak probes (no handle; synchronous on hip_stream, which may be
 * NULL for the default stream).  They measure what the chip reaches in
 * practice, beside the vendor peaks that the roofline fractions use.
 *
 * wam_probe_mfma_bf16: n_blocks blocks of 256 threads each run iters rounds
 * of independent bf16 MFMA chains on register operands (shape 0:
 * v_mfma_f32_16x16x32_bf16, the instruction of the GEMM and attention
 * kernels; shape 1: v_mfma_f32_32x32x16_bf16), 131072 FLOP per wave per
 * round, after one untimed warm-up launch.  sink: device float[n_blocks *
 * 256], caller-owned, receives one value per thread.  Outputs the rate in
 * TFLOP/s and the timed launch in ms.  Size iters so that a launch lasts
 * tens of ms or more: the shader clock ramps up from idle over that time,
 * and launches of a few ms read up to ~20% low.
 *
 * wam_probe_copy: copies bytes (a multiple of 16, both pointers 16-byte
 * aligned, device, caller-owned, not overlapping) from src to dst reps times
 * after one warm-up; outputs the rate counting the bytes read plus written
 * (GB/s, 1e9) and the time per copy in ms.
 *
 * Both return WAM_E_ARG for invalid arguments and WAM_E_HIP for a runtime
 * error (no handle, so no message). */
int wam_probe_mfma_bf16(void *hip_stream, int shape, int n_blocks, int iters, float *sink, double *tflops,
                        double *ms);
int wam_probe_copy(void *hip_stream, const void *src, void *dst, size_t bytes, int reps, double *gbs,
                   double *ms);

#ifdef __cplusplus
}
#endif
#endif /* WAM_H */
