/*
 * instantmimic.h -- C ABI of the MI355X environment-plus-policy step.
 *
 * The library implements, for a batch of independent environments, the part
 * of a DeepMimic-style PPO rollout step that runs outside the physics solver
 * (InstantMimic, arXiv 2609.09821): Sec. 3 / Fig. 3 gives the loop
 *     action = policy(obs); <physics>; reward, terminated, truncated =
 *     eval_reward_and_dones(); reset_envs(terminated | truncated);
 *     obs = build_obs()
 * and Sec. 4 makes every post-physics stage a fused GPU kernel that reads
 * the simulator's arrays in place (Sec. 4.2) with an unconditional reset
 * restricted by a device-side mask (Sec. 4.2).
 *
 * Entry points:
 *   im_env_step_fused  reward + termination + masked reset + observation
 *                      (Sec. 4.1 Fig. 5 reward and dones, Sec. 4.2 reset,
 *                      Sec. 6.1 observation), one kernel launch;
 *   im_policy_act      Gaussian MLP policy forward and action sampling
 *                      (Fig. 3 "policy(obs)", Sec. 6.1 / backflip table:
 *                      state-independent log-std);
 *   im_reset_envs      forced reset of the envs selected by a device mask
 *                      (start of a rollout, host-requested resets).
 *
 * Conventions.  Quaternions are (w, x, y, z), Hamilton product (Fig. 4a
 * converts the simulator's quaternions to wxyz).  World up is +z; a root's
 * local +x axis is its forward direction.  Body 0 is the root (free joint);
 * parent[b] < b.
 *
 * Memory.  Every per-env buffer is device memory owned by the caller; the
 * library never keeps caller pointers between calls.  Per-env arrays are
 * structure-of-arrays with a leading dimension `ld` (>= n_envs): component
 * c of body b of env e is at  base[(b * NC + c) * ld + e].  A context owns
 * its device copies of the skeleton, clip and weight tables and a policy
 * workspace sized for `max_envs` at creation.
 *
 * Hot calls (im_env_step_fused, im_policy_act, im_reset_envs,
 * im_standin_physics) allocate nothing, read no device memory on the host
 * and never synchronise: they validate their arguments on the host in O(1),
 * enqueue kernels on `stream` (a hipStream_t; NULL = the default stream) and
 * return.  Device faults surface at the caller's next synchronisation.
 * They may be captured into a HIP graph.
 *
 * Errors.  Every function returns an im_status and never throws;
 * im_last_error() returns a message for the calling thread's last failure.
 */
#ifndef INSTANTMIMIC_H
#define INSTANTMIMIC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    IM_OK = 0,
    IM_ERR_INVALID_ARG = 1,  /* NULL pointer, bad size, inconsistent description */
    IM_ERR_UNSUPPORTED = 2,  /* valid but beyond this build's limits (e.g. > 64 bodies) */
    IM_ERR_OOM = 3,          /* device allocation failed at creation */
    IM_ERR_HIP = 4           /* a HIP runtime call or kernel launch failed */
} im_status;

enum {
    IM_JOINT_FREE = 0,       /* the root only */
    IM_JOINT_SPHERICAL = 1,  /* 3 rotational DoF */
    IM_JOINT_REVOLUTE = 2,   /* 1 DoF about `axis` */
    IM_JOINT_FIXED = 3       /* no DoF; its clip rotations must be identity */
};

enum { IM_DTYPE_F32 = 0, IM_DTYPE_BF16 = 1 };

#define IM_MAX_BODIES 64
#define IM_MAX_DEPTH 16

typedef struct im_ctx im_ctx;

/*
 * Step configuration.  Reward (Sec. 4.1, Fig. 5, with the end-effector
 * position term of the DeepMimic reward that Sec. 6.1 builds on):
 *   r = c_pose exp(-(w_pos e_pos + w_ee e_ee)) + c_vel exp(-w_vel e_vel)
 *       + c_com exp(-w_com e_com)
 * with e_pos / e_vel the sums over bodies of squared position / linear
 * velocity errors, e_ee the position errors summed over leaf bodies and
 * e_com the squared error of the mass-weighted centre of the body origins.
 * Fig. 5's printed form is c = (0.60, 0.25, 0.15), w = (4, 0.25, 8), w_ee = 0.
 * Termination (Fig. 5, strict "<"; grace steps from the backflip table):
 *   terminated = (t + 1 > grace) && (root_z < h_term || !(r >= r_min)).
 * Truncation: the clip phase reaches 1.
 *
 * Training terms (Sec. 6.1 and the backflip configuration table):
 *   reward_form = IM_REWARD_MULTIPLICATIVE replaces the reward above by
 *     r = exp(-m_jrot e_jrot) exp(-m_jvel e_jvel) exp(-m_com e_com)
 *         exp(-m_eepos e_eepos) exp(-m_eerot e_eerot)
 *   with e_jrot = sum_b angle(qr_b^-1 q_b)^2 over the joint rotations in the
 *   parent frame (the root's world orientation for b = 0), e_jvel = sum_b
 *   |w_b - wr_b|^2 over the joint angular velocities in the parent frame
 *   (R(Q_p)^T (W_b - W_p); the root's world angular velocity), e_com as above,
 *   e_eepos = sum over end effectors (leaf bodies) of squared position errors,
 *   e_eerot = sum over end effectors of squared world-orientation angles.
 *   obs_future = K (0..4) appends, for the next K control steps, the reference
 *   frames of the root and the end effectors; obs_prev_action appends the
 *   action applied in this step (see im_env_bufs).
 */
typedef struct {
    double dt;        /* control step in seconds (> 0) */
    float h_term;     /* root-height termination threshold (m) */
    float r_min;      /* reward termination threshold */
    int32_t grace;    /* steps after a reset during which no env terminates (>= 0) */
    float c_pose, w_pos, w_ee;
    float c_vel, w_vel;
    float c_com, w_com;
    uint64_t seed;    /* Philox4x32-10 key (low word, high word) */
    int32_t reward_form;      /* IM_REWARD_GROUPED (the form above) or IM_REWARD_MULTIPLICATIVE */
    float m_jrot, m_jvel, m_com, m_eepos, m_eerot;  /* multiplicative weights (finite) */
    int32_t obs_future;       /* future reference frames in the observation, 0..4 */
    int32_t obs_prev_action;  /* 1: the previous action ends the observation */
    int32_t env_split;        /* threads per env of im_env_step_fused: IM_SPLIT_AUTO (by
                                 batch size), IM_SPLIT_ONE, IM_SPLIT_HALVES (two walks),
                                 IM_SPLIT_PATHS (one walk per root-to-leaf path; needs
                                 2..8 leaves, else IM_ERR_UNSUPPORTED at im_create).  The
                                 results are the same up to the order of the reward's
                                 fp32 sums over bodies. */
} im_config;

enum { IM_REWARD_GROUPED = 0, IM_REWARD_MULTIPLICATIVE = 1 };
enum { IM_SPLIT_AUTO = 0, IM_SPLIT_ONE = 1, IM_SPLIT_HALVES = 2, IM_SPLIT_PATHS = 3 };

/* Host arrays; copied at creation. */
typedef struct {
    int32_t n_bodies;        /* B, 1..IM_MAX_BODIES */
    const int32_t *parent;   /* [B]; parent[0] = -1, 0 <= parent[b] < b */
    const int32_t *jtype;    /* [B]; jtype[0] = FREE, others SPHERICAL/REVOLUTE/FIXED */
    const float *axis;       /* [B][3]; unit revolute axis in the parent frame */
    const float *offset;     /* [B][3]; joint (= body origin) in the parent frame, m */
    const float *mass;       /* [B]; > 0, kg (point mass at the body origin) */
} im_skeleton;

/* One reference clip, host arrays; copied at creation. */
typedef struct {
    int32_t n_frames;        /* F >= 2 */
    float fps;               /* frames per second (> 0) */
    const float *root_pos;   /* [F][3] world root position */
    const float *root_quat;  /* [F][4] world root orientation, unit (|q| within 1e-3) */
    const float *local_quat; /* [F][B-1][4] rotation of body b = 1..B-1 in its parent frame */
} im_clip;

/*
 * Gaussian MLP policy.  dims[0] must be the observation width D (im_env_bufs) and
 * dims[L] is the action width A.  Hidden layers: ReLU; last layer linear
 * (the mean).  BF16: observation and hidden activations are rounded to bf16
 * (nearest even), weights are bf16, products accumulate in fp32.  Actions:
 * a = mean + exp(log_std) * z, z ~ N(0, 1) from Philox4x32-10 with counter
 * (env, env_n, j, 0) for the four actions 4j..4j+3 (Box-Muller on the two
 * word pairs); logp = -sum_a (z_a^2/2 + log_std_a + ln(2 pi)/2).
 */
typedef struct {
    int32_t n_layers;              /* L >= 1 */
    const int32_t *dims;           /* [L+1] */
    int32_t dtype;                 /* IM_DTYPE_F32 or IM_DTYPE_BF16 */
    const void *const *weight;     /* [L] host pointers, W_l [dims[l+1]][dims[l]] row-major:
                                      float for F32, uint16 bf16 bit patterns for BF16 */
    const float *const *bias;      /* [L] host pointers, b_l [dims[l+1]] */
    const float *log_std;          /* [A] */
} im_policy;

/*
 * Per-env device buffers (caller-owned), ld >= n_envs.
 *   body_pos    [B][3][ld]  world body-origin position (m); read by the step,
 *                           written for reset envs (reference state)
 *   body_quat   [B][4][ld]  world orientation (w,x,y,z)
 *   body_linvel [B][3][ld]  world linear velocity of the body origin (m/s)
 *   body_angvel [B][3][ld]  world angular velocity (rad/s)
 *   env_clip    [ld] int32  reference clip of the env          (read/write)
 *   env_phase   [ld] float  clip phase in [0, 1]               (read/write)
 *   env_t       [ld] int32  steps since the last reset         (read/write)
 *   env_n       [ld] uint32 step counter of the env's random streams
 *   reward      [ld] float, terminated [ld] uint8, truncated [ld] uint8
 *   obs         [D][ld] float: per body b at rows 15b..15b+14 heading-frame
 *               position (3), first two columns of the heading-frame rotation
 *               matrix (6), heading-frame linear (3) and angular (3) velocity;
 *               row 15B = phase (Sec. 6.1).  With obs_future = K, for j = 1..K
 *               the reference of the env's clip at the phase of the j-th next
 *               control step (phase_j = phase_{j-1} + dphi, fp32, evaluated at
 *               min(phase_j, 1)): the root, then each end effector in body order,
 *               9 rows each (heading-frame position and the two columns); then,
 *               with obs_prev_action, A rows of the previous action (zero for an
 *               env reset in this call).  D = 15B + 1 + 9 K (1 + n_ee) + A?
 *   ref_frame   [ld] int32 or NULL: reference frame index used this step
 *   prev_action [n_envs][A] float, read when obs_prev_action (else may be
 *               NULL): the action applied in this step (the im_policy_act
 *               output of the step).  Appended after ld.
 */
typedef struct {
    float *body_pos;
    float *body_quat;
    float *body_linvel;
    float *body_angvel;
    int32_t *env_clip;
    float *env_phase;
    int32_t *env_t;
    uint32_t *env_n;
    float *reward;
    uint8_t *terminated;
    uint8_t *truncated;
    float *obs;
    int32_t *ref_frame;
    int64_t n_envs;
    int64_t ld;
    const float *prev_action;
} im_env_bufs;

typedef struct {
    int32_t n_bodies, obs_dim, action_dim, n_clips, n_layers, policy_dtype, max_depth;
    int64_t max_envs;
    int64_t device_bytes;    /* device memory held by the context */
} im_info;

/*
 * Create a context on the current HIP device.  Validates everything
 * (topology, joint types, unit quaternions, clip lengths, layer widths) and
 * uploads/packs the tables; max_envs bounds n_envs of im_policy_act.
 * On failure *out is NULL and nothing is leaked.
 */
im_status im_create(const im_config *cfg, const im_skeleton *skel, const im_clip *clips,
                    int32_t n_clips, const im_policy *policy, int64_t max_envs, im_ctx **out);

im_status im_destroy(im_ctx *ctx);

im_status im_get_info(const im_ctx *ctx, im_info *info);

/*
 * Fused environment step (Fig. 3 post-physics phase, Sec. 4).  For each env
 * e < n_envs, on the sim state the physics left in the buffers:
 *  1. phase' = phase + dphi_k (fp32, dphi_k = float(dt * fps_k / (F_k - 1)));
 *     t' = t + 1; n' = n + 1; truncated = phase' >= 1;
 *  2. reference at min(phase', 1): s = phase * (F-1), i0 = min(floor(s), F-2),
 *     alpha = s - i0; root position lerp, root and joint rotations slerp
 *     between frames i0 and i0+1, forward kinematics over the tree, reference
 *     velocities = exact time derivatives of that path;
 *  3. reward and terminated (im_config) against the sim state;
 *  4. envs with terminated | truncated are reset: Philox counter
 *     (e, n', 0, 1) gives clip = (x0 * n_clips) >> 32 and phase =
 *     (x1 >> 8) * 2^-24, t = 0, and the sim state of every body is set to
 *     the reference state there (reference state initialisation);
 *     other envs keep clip and sim state and take phase', t';
 *  5. obs is built from the post-reset sim state; env_n = n' for all envs.
 * reward/terminated/truncated describe the pre-reset state.
 */
im_status im_env_step_fused(im_ctx *ctx, const im_env_bufs *bufs, void *stream);

/*
 * Policy forward and sampling for envs e < n_envs.
 *   obs    [D][ld_obs] float (device), env_n [ld_obs] uint32 (device: the
 *          counter before the step that will consume the action)
 *   mean, action [n_envs][A] float (device), logp [n_envs] float or NULL.
 * n_envs <= max_envs.  Uses the context's workspace: calls on one context
 * must be ordered (same stream or synchronised).
 */
im_status im_policy_act(im_ctx *ctx, const float *obs, int64_t ld_obs, const uint32_t *env_n,
                        int64_t n_envs, float *mean, float *action, float *logp, void *stream);

/*
 * Forced reset of the envs whose mask byte is non-zero (all envs when mask
 * is NULL; mask is a device array [n_envs]).  Draws clip and phase with the
 * Philox counter (e, env_n, 0, 4), sets t = 0, writes the reference state to
 * the sim buffers and the observation.  env_n is not advanced.
 */
im_status im_reset_envs(im_ctx *ctx, const im_env_bufs *bufs, const uint8_t *mask, void *stream);

/*
 * Benchmark/test harness, not part of the step: a kinematic stand-in for
 * the physics solver.  Writes to the sim buffers the reference state at each
 * env's next phase (phase + dphi) with Gaussian rotation noise (std
 * sigma_joint rad per DoF) composed on the right of the root orientation and
 * of every non-fixed joint, and velocities = reference + N(0, sigma_vel^2)
 * per component.  Normals: Philox counter (e, env_n, j/4, 3), lane j%4 of
 * the Box-Muller block; j runs over the root rotation (3), then each body
 * 1..B-1's DoFs in index order, then each body's linear (3) and angular (3)
 * velocity in index order.
 */
im_status im_standin_physics(im_ctx *ctx, const im_env_bufs *bufs, float sigma_joint,
                             float sigma_vel, void *stream);

/*
 * Value head for the PPO rollout (Fig. 3: the rollout storage feeds the
 * policy update): a critic MLP laid out like im_policy with dims[0] = D,
 * dims[L] = 1, ReLU hidden layers, linear output and the policy's dtype (the
 * same bf16 rounding points); log_std is not used and may be NULL.  Copied
 * to the device; a second call replaces the critic.  Not hot: allocates, and
 * synchronises the device; no call on the context may be in flight.
 */
im_status im_set_critic(im_ctx *ctx, const im_policy *critic);

/*
 * value[e] = V(obs[:, e]) for e < n_envs: obs [D][ld_obs] float (device),
 * value [n_envs] float (device).  Needs im_set_critic.  Shares the policy's
 * workspace: calls on one context must be ordered (same stream or
 * synchronised).
 */
im_status im_value(im_ctx *ctx, const float *obs, int64_t ld_obs, int64_t n_envs, float *value,
                   void *stream);

/*
 * im_policy_act followed by im_value on the same observation, as one rollout
 * step needs them (Fig. 3: action, logp and value of every observation go to
 * the storage).  Arguments as in the two calls; the outputs equal theirs bit
 * for bit.  A bf16 network of at most 8 layers, hidden widths and input up to
 * 1024 and an output up to 128 runs as one kernel that reads the float
 * observation itself; when both networks are beyond that, a large batch rounds
 * and transposes the observation into the staging buffer once for both
 * instead of once per call.  Needs im_set_critic.  Errors: those of the two
 * calls, before any launch.
 */
im_status im_policy_act_value(im_ctx *ctx, const float *obs, int64_t ld_obs,
                              const uint32_t *env_n, int64_t n_envs, float *mean, float *action,
                              float *logp, float *value, void *stream);

/* Fields of the rollout summary (float64, device). */
enum {
    IM_SUM_REWARD = 0,          /* sum of rewards over steps and envs */
    IM_SUM_TERMINATED,          /* terminated steps */
    IM_SUM_TRUNCATED,           /* truncated steps */
    IM_SUM_EPISODES,            /* episodes ended (terminated or truncated) */
    IM_SUM_EPISODE_RETURN,      /* sum of the returns of the ended episodes */
    IM_SUM_EPISODE_LENGTH,      /* sum of their lengths in steps */
    IM_SUM_ADVANTAGE,           /* sum of the stored advantages */
    IM_SUM_ADVANTAGE_SQ,        /* sum of their squares */
    IM_SUM_VALUE,               /* sum of V_t, t < T */
    IM_SUM_RETURN,              /* sum of the stored returns */
    IM_SUMMARY_FIELDS
};

/*
 * Rollout storage (device, caller-owned).  The step writes into it in place:
 * step t reads obs slot t and writes action/logp/value slot t, and the fused
 * env step writes reward/terminated/truncated slot t and obs slot t+1, so
 * storing a step copies nothing (Fig. 3 storage write).  [T][ld] arrays have
 * the env fastest.
 *   reward [T][ld] float, terminated / truncated [T][ld] uint8
 *   value [T+1][ld] float: V of the observation of each step, slot T the
 *         observation after the last step
 *   advantage, ret [T][ld] float: written
 *   ep_return [ld] float, ep_length [ld] int32: return and length of the
 *         episode each env is in, carried across rollouts (read/write; used
 *         with summary only)
 *   summary [IM_SUMMARY_FIELDS] double or NULL: written
 */
typedef struct {
    int32_t T;
    int64_t n_envs, ld;
    float gamma, lambda;
    const float *reward;
    const uint8_t *terminated;
    const uint8_t *truncated;
    const float *value;
    float *advantage;
    float *ret;
    float *ep_return;
    int32_t *ep_length;
    double *summary;
} im_rollout;

/*
 * Generalized advantage estimation over the rollout storage (Schulman et al.
 * 2016; gamma and lambda from the configuration table of the Appendix):
 *   delta_t = r_t + gamma * next_t - V_t, next_t = 0 if terminated, V_t if
 *             truncated only (cut off, not failed: the next observation is
 *             already the reset one, so the step's own value stands in),
 *             V_{t+1} otherwise;
 *   A_t = delta_t + gamma * lambda * A_{t+1}, the sum stopping at an episode
 *         end (terminated or truncated) and after step T-1; R_t = A_t + V_t.
 * Computed in float64, stored as float32.  With summary: the rollout
 * summaries (IM_SUM_*); at every step the reward is added to ep_return
 * (float32) and ep_length grows by one, an ended episode enters the sums and
 * restarts at 0.  Sums are in float64 in a fixed order (results do not depend
 * on timing).  1 <= T, 0 <= n_envs <= max_envs, ld >= n_envs.
 */
im_status im_gae(im_ctx *ctx, const im_rollout *r, void *stream);

/*
 * im_gae for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * kernels and results, without a context.  The per-block summary sums go to
 * a fixed array of the library on the current device (IM_GAE_NOALLOC_MAX_ENVS
 * / 256 blocks x IM_SUMMARY_FIELDS doubles = 320 KiB, held until the process
 * ends), whose address is looked up on the first call on each device (or at
 * im_create on the context's device).  Every call on a device shares that
 * array: calls that overlap on one GPU (different streams, no ordering) race
 * and must be ordered by the caller.  The call allocates nothing.
 * Errors: those of im_gae; n_envs above IM_GAE_NOALLOC_MAX_ENVS is
 * IM_ERR_UNSUPPORTED.
 */
#define IM_GAE_NOALLOC_MAX_ENVS (1 << 20)
im_status im_gae_noalloc(const im_rollout *r, void *stream);

/*
 * PPO update (Fig. 3 update_policy; objective of Schulman et al. 2017, the
 * paper's configuration table gives its coefficients).  bf16 policies only.
 * Per minibatch: advantages normalised with the rollout's mean and unbiased
 * std (from the im_gae summary), ratio = exp(logp - logp_old),
 *   L_pi = mean max(-A ratio, -A clip(ratio, 1 - clip, 1 + clip)),
 *   L_V  = mean max((V - R)^2, (V_old + clip(V - V_old, -clip, clip) - R)^2)
 *          (clipped_value_loss; else mean (V - R)^2),
 *   H    = sum_a (log_std_a + (1 + ln 2 pi) / 2),
 *   loss = L_pi + value_coef L_V - entropy_coef H;
 * KL to the rollout policy (mean_old, log_std at the start of the update),
 * averaged over the minibatch, adapts the learning rate when desired_kl > 0
 * (/1.5 above 2 desired_kl, not below lr_min; x1.5 below desired_kl / 2,
 * not above lr_max); the gradient of all parameters is clipped to the
 * global norm max_grad_norm (> 0), then one Adam step updates the float32
 * master weights, and the policy and critic copies the rollout calls use are
 * refreshed from them.  The forward rounds input, weights and hidden
 * activations to bf16 like im_policy_act; the backward stores the gradient
 * of every layer's pre-activation as bf16 and accumulates in float32.
 */
typedef struct {
    float clip;                /* ratio clip, also the value clip */
    float value_coef, entropy_coef;
    int32_t clipped_value_loss;
    float max_grad_norm;       /* <= 0: no clipping */
    float beta1, beta2, eps;   /* Adam */
    float desired_kl;          /* <= 0: fixed learning rate */
    float lr_min, lr_max;
    int32_t epochs, minibatches;
} im_ppo_params;

/*
 * The rollout to learn from (device, the im_rollout storage after im_gae):
 *   obs [T+1][D][ld] (slots 0..T-1), action and mean [T][n_envs][A] (the
 *   actions and means im_policy_act returned), logp [T][ld], value [T+1][ld],
 *   advantage and ret [T][ld], summary: the im_gae summary of this rollout.
 *   perm [epochs][T * n_envs / 64] int32: the order of the rollout's 64-env
 *   chunks in each epoch (chunk q = envs 64 (q % (n_envs/64)) .. +63 of step
 *   q / (n_envs/64)); the chunks of an epoch are split into `minibatches`
 *   consecutive groups, the first (count % minibatches) one chunk longer
 *   (entries outside [0, count) are clamped into it).
 *   lr: device float, the learning rate (adapted in place).
 *   stats: device double [IM_PPO_STATS] (sums over minibatches, added to) or
 *   NULL.  n_envs must be a multiple of 64.
 */
typedef struct {
    int32_t T;
    int64_t n_envs, ld;
    const float *obs, *action, *mean, *logp, *value, *advantage, *ret;
    const double *summary;
    const int32_t *perm;
    float *lr;
    double *stats;
} im_ppo_batch;

enum {
    IM_PPO_LOSS_PI = 0,   /* surrogate loss (sum of minibatch means) */
    IM_PPO_LOSS_V,        /* value loss */
    IM_PPO_KL,            /* KL to the rollout policy */
    IM_PPO_CLIP_FRAC,     /* fraction of clipped ratios */
    IM_PPO_GRAD_NORM,     /* gradient norm before clipping */
    IM_PPO_MINIBATCHES,   /* minibatches counted */
    IM_PPO_LR,            /* learning rate after the last step (not a sum) */
    IM_PPO_STATS
};

/*
 * Allocate the training state for minibatches of up to max_minibatch
 * samples: float32 master weights (from the current policy and critic),
 * Adam moments, activation and gradient buffers.  Not hot: allocates and
 * synchronises.  Needs a critic; a second call resets the optimizer.
 * Parameter vector order: actor W_0 [out][in], b_0, ..., log_std, critic
 * W_0, b_0, ..., the critic's output layer W [1][in], b [1].
 */
im_status im_ppo_setup(im_ctx *ctx, int64_t max_minibatch);

/* The whole update (epochs x minibatches); enqueued on the stream, no host
 * synchronisation, allocates nothing. */
im_status im_ppo_update(im_ctx *ctx, const im_ppo_batch *b, const im_ppo_params *p, void *stream);

/* The float32 gradient (parameter vector order, before clipping) of one
 * minibatch of one epoch at the current weights, no step; stats (device
 * double [IM_PPO_STATS] or NULL) receives that minibatch's loss terms. */
im_status im_ppo_grad(im_ctx *ctx, const im_ppo_batch *b, const im_ppo_params *p, int32_t epoch,
                      int32_t minibatch, float *grad, double *stats, void *stream);

/* Number of parameters and, when params != NULL, a copy of the master
 * weights (device float [n]). */
im_status im_ppo_params_get(im_ctx *ctx, float *params, int64_t *n, void *stream);

/*
 * Buffers of the update's last minibatch (the one im_ppo_grad or
 * im_ppo_update ran last), for checking its stages one at a time.  Columns
 * are that minibatch's samples in gather order, padded to a multiple of 256
 * (padding columns hold the zero-input forward and zero gradients); rows of a
 * layer are its width padded to 128.
 *   IM_PPO_BUF_INPUT          bf16 [D128][cols]  observation as the forward reads it
 *   IM_PPO_BUF_ACTOR_HIDDEN   bf16 [W128][cols]  output of the actor's hidden layer `layer`
 *                                                (bias, ReLU, rounded to bf16)
 *   IM_PPO_BUF_CRITIC_HIDDEN  bf16 [W128][cols]  the same for the critic
 *   IM_PPO_BUF_MEAN           float [A][cols]    policy mean
 *   IM_PPO_BUF_VALUE          float [1][cols]    value
 *   IM_PPO_BUF_DMEAN          bf16 [A128][cols]  gradient of the loss with respect to the
 *                                                mean, as the backward reads it
 *   IM_PPO_BUF_DVALUE         float [1][cols]    gradient of the loss with respect to the value
 */
enum {
    IM_PPO_BUF_INPUT = 0,
    IM_PPO_BUF_ACTOR_HIDDEN,
    IM_PPO_BUF_CRITIC_HIDDEN,
    IM_PPO_BUF_MEAN,
    IM_PPO_BUF_VALUE,
    IM_PPO_BUF_DMEAN,
    IM_PPO_BUF_DVALUE,
    IM_PPO_BUFFERS
};

/* Shape of buffer `buffer` (layer: hidden layer index, else 0) in *rows,
 * *cols, *elem_bytes (any may be NULL) and, when dst != NULL, a device copy
 * of it into dst (rows * cols * elem_bytes bytes, enqueued on the stream).
 * Errors: no training state, no minibatch run yet, buffer or layer out of
 * range. */
im_status im_ppo_read(im_ctx *ctx, int32_t buffer, int32_t layer, void *dst, int64_t *rows,
                      int64_t *cols, int64_t *elem_bytes, void *stream);

const char *im_status_str(im_status s);
const char *im_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* INSTANTMIMIC_H */
