/*
 * dc.h -- C ABI of the DriveCache cache-aware denoising step on MI355X (gfx950).
 *
 * DriveCache (Sec. 3 of the paper) splits each denoising step of a frozen video
 * diffusion model into an expensive backbone r_k = F_k(u_k) and a cheap output
 * interface eps_k = H_k(x_k, r_k) (Eq. 1).  A host-side exact dynamic program
 * places cache reuse over the K steps under a response budget (Eq. 2-4, 8-11);
 * before every planned reuse a causal drift check (Eq. 12) may force a refresh
 * and a replan of the unexecuted suffix.  This library runs the whole step on
 * one GPU with hand-written HIP kernels, and the schedule on the host.
 *
 * Generator (a stand-in with the paper's structure; the paper treats it as
 * frozen): a video DiT over N = N_v + N_t tokens of width d -- N_v latent
 * patches of a [C, T, H, W] latent (patch p, token n = (t Hp + i) Wp + j) and
 * N_t text rows -- with L AdaLN-modulated blocks (joint self-attention, GELU-tanh
 * MLP), an AdaLN head and a flow-matching Euler sampler.  The cache boundary:
 * F_k is the block stack, r_k = h_out - h_in on the video rows, u_k = block 0's
 * modulated input on the video rows, H_k = head + Euler.
 *
 * Conventions
 *   Ownership   All device memory is owned by the caller; the library never
 *               allocates or frees device memory.  Host arrays passed in are
 *               read during the call only (dc_sampler_create copies what it keeps).
 *   Layouts     Row-major.  Weight matrices are [out, in] ("y = x W^T + b").
 *               Activations of a batch are [B, rows, d] with rows = N (h, h_in, g)
 *               or N_v (residual cache, reference input).
 *   dtype       DC_BF16: matrices (w_qkv, w_o, w_1, w_2, w_head, pos), the residual
 *               cache and the reference input are bf16; everything else f32.
 *               DC_F32: everything f32.  w_pe and the timestep MLP are always f32.
 *   Streams     Every device call is enqueued on the given stream (0 = null
 *               stream) and returns without waiting, except dc_denoise_step,
 *               which waits once per step when a drift check is due.
 *   Batches     idx/n select samples of the batch (host int32 array, n <= DC_MAX_BATCH,
 *               entries distinct and < B).  n = 0 is a no-op.
 *   Indexing    C arrays are 0-based: element i of a per-step array is step i+1;
 *               row j-1 / column h-1 of a table is refresh step j / cache age h.
 *   Errors      A negative status; dc_last_error() describes the most recent
 *               failure on the calling thread.  Outputs are unspecified on error.
 *               Shapes and arguments are checked before any launch.
 *   Threading   Entry points are reentrant; a dc_sampler is used by one thread.
 */
#ifndef DRIVECACHE_DC_H
#define DRIVECACHE_DC_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t dc_status;
enum {
  DC_OK = 0,
  DC_ERR_ARG = -1,        /* bad argument (null pointer, out of range value) */
  DC_ERR_SHAPE = -2,      /* model shape the kernels do not support */
  DC_ERR_DTYPE = -3,      /* unknown dtype */
  DC_ERR_HIP = -4,        /* a HIP runtime call failed; the message names it */
  DC_ERR_WORKSPACE = -5,  /* workspace smaller than dc_workspace_bytes() */
  DC_ERR_STATE = -6       /* sampler used out of order */
};

#define DC_MAX_BATCH 64

/* Text of the last error on this thread ("" if none).  Valid until the next
 * failing call on the same thread. */
const char* dc_last_error(void);

typedef enum { DC_F32 = 0, DC_BF16 = 1 } dc_dtype;

/* Model shape.  Requirements (else DC_ERR_SHAPE): heads * head_dim == hidden;
 * head_dim in {64, 72} for DC_BF16 and 64 for DC_F32; hidden a multiple of 128
 * and at most 3072; mlp_hidden a multiple of 128; lat_h, lat_w divisible by patch;
 * lat_c * patch^2 == 64. */
typedef struct {
  int32_t n_blocks, hidden, heads, head_dim, mlp_hidden;
  int32_t lat_c, lat_t, lat_h, lat_w, patch, n_txt;
  int32_t dtype;          /* dc_dtype */
  float ln_eps;           /* layer-norm epsilon (biased variance, no affine) */
} dc_model_cfg;

/* One block's parameters (device memory).  Matrices in the model dtype, biases f32. */
typedef struct {
  const void* w_qkv;  const float* b_qkv;   /* [3d, d], [3d]; Q | K | V, head-major within each */
  const void* w_o;    const float* b_o;     /* [d, d], [d] */
  const void* w_1;    const float* b_1;     /* [F, d], [F] */
  const void* w_2;    const float* b_2;     /* [d, F], [d] */
  const float* mod_offset;                  /* [6, d] per-block modulation offset M_l */
} dc_block_weights;

/* Whole-generator parameters (device memory, except the `blocks` host array). */
typedef struct {
  const float* w_pe;  const float* b_pe;    /* [d, 64], [d] f32 patch embedding */
  const void* pos;                          /* [N_v, d] position table, model dtype */
  const float* w_t1;  const float* b_t1;    /* [d, 256], [d] timestep MLP layer 1 */
  const float* w_t2;  const float* b_t2;    /* [d, d], [d]   timestep MLP layer 2 */
  const float* w_m;   const float* b_m;     /* [6d, d], [6d] shared modulation projection */
  const float* head_mod;                    /* [2, d] head modulation offset */
  const void* w_head; const float* b_head;  /* [64, d] model dtype, [64] */
  const dc_block_weights* blocks;           /* host array [n_blocks] */
} dc_model_weights;

/* ---------------------------------------------------------------------------
 * Device steps of the hot path.  All pointers are device memory unless noted,
 * 16-byte aligned (hipMalloc and PyTorch's allocator give 256; per-sample slices
 * of the [B, ...] buffers keep it because hidden is a multiple of 128).
 * ------------------------------------------------------------------------- */

/* Bytes of scratch device memory the calls below need for a batch of B. */
size_t dc_workspace_bytes(const dc_model_cfg* cfg, int32_t batch);

/* Timestep embedding and AdaLN modulation for steps 1..K (the conditioning of
 * F_k and H_k in Eq. 1).  sigmas: host f64 [K] noise levels; t = 1000 sigma.
 * mod out: f32 [K, L+1, 6, d]: entry [k, l] (l < L) = (shift1, scale1, gate1,
 * shift2, scale2, gate2) of block l; entry [k, L] rows 0, 1 = (shift_f, scale_f)
 * of the head, rows 2..5 zero. */
dc_status dc_time_modulation(const dc_model_cfg* cfg, const dc_model_weights* w,
                             const double* sigmas, int32_t K, float* mod,
                             void* ws, size_t ws_bytes, hipStream_t stream);

/* Backbone input of Eq. 1: h_in[b] = patchify(x[b]) w_pe^T + b_pe + pos on the
 * N_v video rows, then the N_t rows of txt[b].  x: f32 [B, C, T, H, W];
 * txt: f32 [B, N_t, d]; h_in: f32 [B, N, d]. */
dc_status dc_patch_embed(const dc_model_cfg* cfg, const dc_model_weights* w, const float* x,
                         const float* txt, float* h_in, const int32_t* idx, int32_t n,
                         void* ws, size_t ws_bytes, hipStream_t stream);

/* One transformer block, in place on h[b] (f32 [B, N, d]) for the selected samples.
 * mod: f32 [6, d] = this block's (shift1, scale1, gate1, shift2, scale2, gate2).
 * a = LN(h)(1+scale1)+shift1; h += gate1 (Attn(a W_qkv^T + b_qkv) W_o^T + b_o);
 * a2 = LN(h)(1+scale2)+shift2; h += gate2 (GELU_tanh(a2 W_1^T + b_1) W_2^T + b_2).
 * The refresh path runs this L times (F_k of Eq. 1). */
dc_status dc_block_forward(const dc_model_cfg* cfg, const dc_block_weights* blk,
                           const float* mod, float* h, const int32_t* idx, int32_t n,
                           void* ws, size_t ws_bytes, hipStream_t stream);

/* Refresh: store the cached backbone output r = h_out - h_in on the video rows
 * (Eq. 1; the reused value of Sec. 3).  h_out, h_in: f32 [B, N, d];
 * resid: [B, N_v, d] model dtype (bf16 rounds to nearest even). */
dc_status dc_cache_store(const dc_model_cfg* cfg, const float* h_out, const float* h_in,
                         void* resid, const int32_t* idx, int32_t n, hipStream_t stream);

/* Reuse: g = h_in + r on the video rows (Eq. 1, a reuse replaces r_k by the most
 * recent r_j).  h_in: f32 [B, N, d]; resid [B, N_v, d]; g: f32 [B, N, d], only the
 * video rows are written (g may alias a buffer other than h_in). */
dc_status dc_cache_apply(const dc_model_cfg* cfg, const float* h_in, const void* resid,
                         float* g, const int32_t* idx, int32_t n, hipStream_t stream);

/* Backbone input u = LN(h_in[:N_v])(1+scale1)+shift1 with mod0 = f32 [2, d]
 * (block 0's shift1, scale1).  snapshot != 0: u_ref[b] := u (model dtype).
 * snapshot == 0: sums[b] (f64 [B, 4]) = (sum|u-u_ref|, sum|u|, sum(u-u_ref)^2,
 * sum u^2) over the sample's N_v x d tensor, the ingredients of the observed
 * drift of Eq. 12.  Reductions are in a fixed order (bitwise reproducible). */
dc_status dc_drift_l1(const dc_model_cfg* cfg, const float* h_in, const float* mod0,
                      void* u_ref, int32_t snapshot, double* sums, const int32_t* idx,
                      int32_t n, void* ws, size_t ws_bytes, hipStream_t stream);

/* dc_drift_l1 for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same computation
 * and results, bit for bit, without a workspace argument.  The partial sums of the
 * reduction live in a fixed device array inside the library, one copy per GPU
 * (2 MiB, held until the process ends; its address is looked up on the first call on
 * each device).  Limit: n <= DC_MAX_BATCH samples (DC_ERR_ARG beyond); any model shape
 * dc_drift_l1 takes.  The call allocates nothing.  Calls that overlap on one GPU
 * (several streams or threads at once) share the array and race: serialise them. */
dc_status dc_drift_l1_noalloc(const dc_model_cfg* cfg, const float* h_in, const float* mod0,
                              void* u_ref, int32_t snapshot, double* sums, const int32_t* idx,
                              int32_t n, hipStream_t stream);

/* Output interface H_k and the sampler update (Eq. 1): y = LN(g)(1+scale_f)+shift_f
 * on the video rows of g (f32 [B, N, d]), v = unpatchify(y w_head^T + b_head),
 * x[b] += dsigma * v.  head_mod: f32 [2, d] (shift_f, scale_f); x: f32 [B, C, T, H, W].
 * bf16 models with hidden <= 2048 run one pass over g with the projection operand
 * split into two bf16 halves (about fp32 accuracy); wider bf16 models round y to
 * bf16 before the projection. */
dc_status dc_head_euler(const dc_model_cfg* cfg, const dc_model_weights* w,
                        const float* head_mod, const float* g, float* x, float dsigma,
                        const int32_t* idx, int32_t n, void* ws, size_t ws_bytes,
                        hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Host schedule (pure; no device access).
 * ------------------------------------------------------------------------- */

/* One scene's scheduling problem (host memory, read during the call).
 * Sec. 3.1: poses -> L, Theta (Eq. 2) -> z (Eq. 3, anchors (L0, Th0), (L1, Th1)) ->
 * support gate [0,1]^2 (outside: full inference) -> D (Eq. 4) -> one-sided
 * interpolation of q and d (Eq. 8) -> envelope Q and increments c (Eq. 9), costs in
 * integer units of 2^-40.  Sec. 3.2: exact DP (Eq. 10), B* (Eq. 11), backtracking. */
typedef struct {
  int32_t K, h_max, n_cap;      /* steps; max cache age; max total reuses (0..K-1) */
  const uint8_t* legal;         /* [K] 1 = reuse allowed at that step; entry 0 ignored */
  const int32_t* segment;       /* [K] or NULL; a run never crosses a segment change */
  int32_t n_pose;
  const double* pose_xy;        /* [n_pose, 2] planned positions (m) */
  const double* pose_yaw;       /* [n_pose] planned headings (rad) */
  double L0, Th0, L1, Th1;      /* low-motion and moving-turn anchors */
  double eps;                   /* the epsilon of Eq. 3 and of the veto */
  const double *q0, *q1;        /* [(K-1), h_max] anchor joint run responses */
  const double *d0, *d1;        /* [(K-1), h_max] anchor drift thresholds */
  int64_t tau_q;                /* budget tau (units 2^-40); INT64_MAX = no budget */
  int32_t start_step;           /* 1 = initial plan; s = replan after a forced refresh at s */
  int64_t spent_q;              /* charge C already accumulated (replans) */
  int32_t spent_n;              /* reuses already executed (replans) */
} dc_sched_problem;

typedef struct {
  uint8_t* reuse;               /* out [K]: 1 = reuse; steps <= start_step are 0 */
  int64_t* chat_q;              /* out [(K-1), h_max] scene costs, or NULL */
  double* dbar;                 /* out [(K-1), h_max] scene drift thresholds, or NULL */
  int32_t n_reuse;              /* out: B* (additional reuses on a replan) */
  int64_t cost_q;               /* out: the schedule's cost */
  double L, Theta, zL, zTh, D;  /* out: motion statistics and intensity */
  int32_t in_support;           /* out: 0 = outside the anchors' support (no reuse) */
} dc_schedule;

dc_status dc_schedule_dp(const dc_sched_problem* p, dc_schedule* out);

/* Response budget (Sec. 3.2 with the Sec. 4.1 protocol): the smallest candidate
 * threshold min_h J_K(n, h) at which the median B* over the n calibration problems
 * reaches ceil(rho (K-1)); the largest candidate if none does.  All problems
 * share K. */
dc_status dc_select_tau(const dc_sched_problem* problems, int32_t n, double rho, int64_t* tau_q);

/* Eq. 2 for one planned pose sequence: L = sum of ||p_t - p_{t-1}||_2 and Theta = sum of
 * |wrap(psi_t - psi_{t-1})| (wrap to [-pi, pi)), one IEEE double operation at a time (the
 * values dc_schedule_dp reports).  pose_xy: host f64 [n_pose, 2]; pose_yaw: host f64
 * [n_pose]; L, Theta: host out.  n_pose < 2 gives 0, 0.  Errors: DC_ERR_ARG on NULL. */
dc_status dc_motion_statistics(const double* pose_xy, const double* pose_yaw, int32_t n_pose,
                               double* L, double* Theta);

/* Anchor selection of Sec. 3.1 over n calibration clips with motion statistics L[i],
 * Theta[i] (host f64 [n], e.g. from dc_motion_statistics).  Both are standardised with the
 * set's mean and population standard deviation (max(sd, eps) as the denominator).  The
 * low-motion anchor minimises z^L + z^Theta.  Among clips whose Theta is above the set's
 * median (mean of the two middle values for even n) and whose L and Theta are above the
 * low-motion anchor's, the moving-turn anchor maximises z^L z^Theta.  Ties keep the lower
 * clip index.  Out: anchors [4] = (L0, Theta0, L1, Theta1) for dc_sched_problem, index [2]
 * = the two clip indices.  No qualifying clip: index[1] = -1, (L1, Theta1) = (L0, Theta0),
 * DC_OK; the paper then falls back to full inference (the caller's decision).
 * Errors: DC_ERR_ARG for n < 1, eps <= 0, non-finite statistics or NULL pointers. */
dc_status dc_select_anchors(const double* L, const double* Theta, int32_t n, double eps,
                            double* anchors, int32_t* index);

/* ---------------------------------------------------------------------------
 * Anchor calibration of the run tables (Sec. 3.1 after Eq. 4; Eq. 5-7).
 * ------------------------------------------------------------------------- */

/* Bytes of device workspace dc_calibrate_tables needs for K steps (the full trace of
 * x_k, u_k, r_k plus the tangent-mode activations of one network pass). */
size_t dc_calibrate_workspace_bytes(const dc_model_cfg* cfg, int32_t K);

/* The response and drift tables of one anchor clip, from its full (uncached) denoising
 * trace: for a run refreshed at step j and reused for h steps (row j-1, column h-1),
 *   d[j,h] = ||u_{j+h} - u_j||_2 / (||u_{j+h}||_2 + eps)                      (Eq. 5)
 *   e_{j,l} = H_{j+l}(x_{j+l}, r_j) - H_{j+l}(x_{j+l}, r_{j+l})               (Eq. 6)
 *   q[j,h] = ||sum_{l<=h} P_{j+l} e_{j,l}||_2 / (||x_out||_2 + eps)            (Eq. 7)
 * where u, r, x are the trace's backbone inputs, backbone outputs and latents, H_k(x, r)
 * the head's denoiser output for g = h_in(x)[video] + r, x_out the terminal latent, and
 * P_t e the terminal-latent tangent when the denoiser output of step t moves by e (a
 * Jacobian-vector product of the network at every later step of the trace).  Entries
 * with j + h > K are 0.  x1: device f32 [C, T, H, W] (the clip's initial noise); txt:
 * device f32 [N_t, d]; sigmas: host f64 [K+1]; q, d: host f64 [(K-1), h_max] out, the
 * q0/d0 (or q1/d1) of dc_sched_problem.  The trace runs the library's kernels of the
 * model's dtype; r, u, the perturbations and the tangents are fp32 (bf16 weights are
 * widened exactly).  head_dim 64 (else DC_ERR_SHAPE).  Waits on `stream` (the table
 * entries are read back). */
dc_status dc_calibrate_tables(const dc_model_cfg* cfg, const dc_model_weights* w, const float* x1,
                              const float* txt, const double* sigmas, int32_t K, int32_t h_max,
                              double eps, double* q, double* d, void* ws, size_t ws_bytes,
                              hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Sampler: the causal controller of Sec. 3.2 around the device steps.
 * ------------------------------------------------------------------------- */
typedef struct dc_sampler dc_sampler;

/* Caller-owned device buffers of a batch of B scenes. */
typedef struct {
  float* x;          /* [B, C, T, H, W] latent x_k, updated in place */
  const float* txt;  /* [B, N_t, d] text embeddings */
  float* h_in;       /* [B, N, d] backbone input */
  float* h;          /* [B, N, d] residual stream; the head input on refresh steps (on reuse
                        steps bf16 models with hidden <= 2048 form g = h_in + r inside the
                        head kernel and leave h as it was; other models write g here) */
  void* resid;       /* [B, N_v, d] residual cache r_j (model dtype) */
  void* u_ref;       /* [B, N_v, d] refresh input u_j (model dtype) */
  float* mod;        /* [K, L+1, 6, d] modulation table (filled at creation) */
  double* sums;      /* [B, 4] drift sums */
  void* ws;          /* workspace of dc_workspace_bytes(cfg, B) bytes */
  size_t ws_bytes;
} dc_buffers;

/* problems: host [B] (start_step 1, nothing spent); sigmas: host f64 [K+1].
 * drift_metric 0 = relative L1 (sum|u-u_j| / (sum|u| + eps)), 1 = relative L2 (Eq. 12).
 * Fills buf->mod (enqueued on `stream`) and computes the initial schedules. */
dc_status dc_sampler_create(const dc_model_cfg* cfg, const dc_model_weights* w, int32_t B,
                            const dc_sched_problem* problems, const double* sigmas,
                            const dc_buffers* buf, int32_t drift_metric, hipStream_t stream,
                            dc_sampler** out);

/* Options of dc_sampler_create_ex; zero-initialise, then set what is used.
 * Model-specific legality (Sec. 3.2, last paragraph; Table 4):
 *  - Two experts: steps k >= k_switch run w_low (its own patch embedding,
 *    conditioning, blocks and head) with the modulation table mod_low
 *    (f32 [K, L+1, 6, d], filled at creation); earlier steps run the weights
 *    passed to the create call.  No cached entry crosses the switch: every
 *    scene's problem must change segment at k_switch (else DC_ERR_ARG).
 *    w_low NULL: one backbone.
 *  - Guidance branches: cfg = 1 adds to every scene an unconditional branch on
 *    txt_null (f32 [B, N_t, d]) with its own residual cache, and x moves along
 *    v_u + guidance (v_c - v_u).  Then h_in, h and resid of dc_buffers hold
 *    2B entries (entry B + b is scene b's unconditional branch), ws must hold
 *    dc_workspace_bytes(cfg, 2B) bytes and B <= 32; u_ref and sums keep B.
 *    Both branches share every step's decision; the drift check (on the video
 *    rows, which do not depend on the text) runs once per scene. */
typedef struct {
  int32_t drift_metric;                /* as in dc_sampler_create */
  const dc_model_weights* w_low;       /* low-noise expert, or NULL */
  int32_t k_switch;                    /* first step of w_low, in 2..K */
  float* mod_low;                      /* [K, L+1, 6, d] modulation table of w_low */
  int32_t cfg;                         /* 1: guidance branches */
  float guidance;                      /* guidance scale w */
  const float* txt_null;               /* [B, N_t, d] unconditional text */
} dc_sampler_opts;

/* dc_sampler_create with the options above (NULL opts = drift_metric 0, one
 * backbone, no guidance). */
dc_status dc_sampler_create_ex(const dc_model_cfg* cfg, const dc_model_weights* w, int32_t B,
                               const dc_sched_problem* problems, const double* sigmas,
                               const dc_buffers* buf, const dc_sampler_opts* opts,
                               hipStream_t stream, dc_sampler** out);

/* Denoising step k (1-based, called for k = 1..K in order) of every scene.
 * realized: host uint8 [B] out (1 = reused, 0 = backbone evaluated); drift: host f64
 * [B] out (observed drift, NaN where no check ran).  Waits on `stream` once if any
 * scene has a planned reuse at k; otherwise returns with work enqueued. */
dc_status dc_denoise_step(dc_sampler* s, int32_t k, hipStream_t stream, uint8_t* realized,
                          double* drift);

/* Current plan of scene b (host uint8 [K] out), vetoes so far and charge C. */
dc_status dc_sampler_plan(const dc_sampler* s, int32_t b, uint8_t* reuse, int32_t* n_veto,
                          int64_t* charge_q);

void dc_sampler_destroy(dc_sampler* s);

/* ---------------------------------------------------------------------------
 * Kernel timing (a measurement aid; off by default).
 * Classes: 0 attention, 1 QKV GEMM, 2 output-projection GEMM, 3 MLP-up GEMM,
 * 4 MLP-down GEMM, 5 AdaLN modulation, 6 patch embedding, 7 drift reduction,
 * 8 cache store, 9 cache apply, 10 head + Euler, 11 head + Euler on a reuse step of a
 * bf16 model (its input g = h_in + r formed in the kernel).
 * ------------------------------------------------------------------------- */

/* Bit c of mask enables timing of class c: each launch is bracketed by two
 * hipEvents on its stream (adds a few microseconds of host work per launch). */
dc_status dc_profile_enable(uint32_t mask);
/* Launch count and summed device time (ms) of class cls since the last reset;
 * waits for the recorded events.  DC_ERR_ARG for an unknown class. */
dc_status dc_profile_read(int32_t cls, int64_t* launches, double* total_ms);
/* Forget recorded launches (their events return to a reuse pool). */
dc_status dc_profile_reset(void);

#ifdef __cplusplus
}
#endif
#endif /* DRIVECACHE_DC_H */
