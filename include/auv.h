/*
 * auv.h - C interface of libauv, the batched 6-DOF underwater-vehicle rollout on one
 * AMD Instinct MI355X (gfx950).
 *
 * What is computed: many independent copies of one vehicle model stepped in a single
 * batch, each with its own random initial conditions and randomisation parameters
 * (paper Sec. IV-A), observed through body-frame errors (Sec. IV-B) and driven by a
 * policy network (Sec. III-A, V).  One control step of one environment:
 *   1. action a (caller's, Philox-uniform, or the policy MLP's mean / Gaussian sample);
 *      u = clip(a, -1, 1); thrust f = f_max u; body wrench tau = T f (6x8 allocation)
 *   2. `substeps` classic RK4 substeps of the Fossen 6-DOF equations of motion (the model
 *      of Sec. IV-D, Eq. 8) with added mass, Coriolis, linear + quadratic damping, restoring
 *      forces with the buoyancy centre offset (Sec. VI-A) and a constant ocean current
 *   3. episode step + 1; reference pose (episode goal, or Lissajous + yaw ramp)
 *   4. observation [R^T(p_ref - p), R_err[:,0], R_err[:,1], v, omega, u], R_err = R^T R_ref
 *   5. reward -|R^T(p_ref - p)| - 0.5 theta_err - 0.01 |u|^2 (shape of Sec. IV-B, Eqs. 2-5)
 *   6. at the episode length: automatic reset with fresh Philox draws (Sec. V-A)
 *
 * Conventions: world NED, body forward-right-down with origin at the centre of gravity,
 * Hamilton quaternion (w, x, y, z) body -> world.  State rows: p(3) q(4) v(3) omega(3).
 *
 * Memory: every device buffer is allocated and owned by the caller; the library keeps
 * non-owning pointers and never allocates device memory.  Layouts are structure of
 * arrays with the environment index fastest: [k][N] or [k][T][N].  Device pointers must
 * be 16-byte aligned.  All fp32 unless stated.
 *
 * Errors: every function returns AUV_OK (0) or a negative code; nothing throws or aborts
 * across the interface.  Arguments are checked before anything is enqueued; a failed
 * check returns AUV_EINVAL and enqueues nothing.  auv_last_error() gives a message for
 * the calling thread's last failure.  Launch failures return AUV_ELAUNCH.
 *
 * Streams: `stream` is a hipStream_t passed as void* (NULL = the null stream).  Every
 * call is asynchronous on that stream unless stated.  A handle is not thread-safe.
 */
#ifndef AUV_H
#define AUV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  AUV_OK = 0,
  AUV_EINVAL = -1,   /* bad argument: nothing was enqueued */
  AUV_ENODEV = -2,   /* no usable HIP device */
  AUV_ELAUNCH = -3,  /* kernel launch failed */
  AUV_ERUNTIME = -4, /* other HIP runtime error */
  AUV_ENONFINITE = -5 /* auv_get_status: non-finite state (or an abandoned wait) was seen */
};

/* Action sources. */
enum {
  AUV_ACT_EXTERNAL = 0,     /* caller's actions */
  AUV_ACT_RANDOM = 1,       /* Philox uniform in [-1, 1), counter (env, global step, 1, b) */
  AUV_ACT_POLICY_MEAN = 2,  /* policy MLP output mu */
  AUV_ACT_POLICY_SAMPLE = 3 /* mu + exp(log_std) eps, eps Box-Muller from (env, step, 2, b) */
};

/* Configuration flags. */
enum {
  AUV_F_DR = 1,        /* mass (and inertia), added mass, damping scaled by U[0.8, 1.2] */
  AUV_F_CURRENT = 2,   /* constant world-frame current, U[-0.3, 0.3] m/s per axis */
  AUV_F_LISSAJOUS = 4, /* Lissajous position reference and level yaw ramp */
  AUV_F_STAGGER = 8    /* at auv_reset, ep_step of env i starts at (global id) mod H */
};

#define AUV_OBS_DIM 23
#define AUV_ACT_DIM 8
#define AUV_STATE_DIM 13
#define AUV_PARAM_DIM 24
#define AUV_HIDDEN 256
#define AUV_ENVS_PER_GROUP 64 /* environments per workgroup; stats partials per group */

typedef struct auv_env auv_env; /* opaque; host memory owned by the library */

typedef struct {
  int32_t n_envs;      /* N >= 1 */
  int32_t substeps;    /* S >= 1 RK4 substeps per control step */
  int32_t episode_len; /* H >= 1 control steps per episode */
  float dt_control;    /* control period in seconds, > 0 */
  uint64_t seed;       /* Philox key = (seed & 0xffffffff, seed >> 32) */
  uint32_t flags;      /* AUV_F_* */
  uint32_t env_offset; /* global id of local env 0 (Philox counter word 0 = global id) */
} auv_config;

/* Vehicle constants, copied by value into every launch.  Diagonal matrices are given by
 * their diagonals in the order (surge, sway, heave, roll, pitch, yaw). */
typedef struct {
  float m;              /* rigid-body mass, kg */
  float inertia[3];     /* rigid-body inertia diagonal about the CoG, kg m^2 */
  float added_mass[6];  /* diagonal added mass M_A */
  float lin_damp[6];    /* diagonal linear damping D_L */
  float quad_damp[6];   /* diagonal quadratic damping D_Q (force = D_Q |nu| nu) */
  float W, B;           /* weight and buoyancy, N */
  float r_b[3];         /* centre of buoyancy in body axes, m */
  float f_max;          /* thrust per thruster at |u| = 1, N */
  float alloc[48];      /* 6x8 allocation table T, row-major: tau = T f */
} auv_vehicle;

/* Environment state buffers (device, caller-owned, each N-strided). */
typedef struct {
  float* state;       /* [13][N] p, q, v, omega */
  float* params;      /* [24][N] s_m s_a s_d, c_w(3), p_goal(3), q_goal(4), A(3), f(3),
                         phase(3), yaw_rate, yaw0 */
  int32_t* ep_step;   /* [N] control steps taken in the current episode */
  uint32_t* episode;  /* [N] episode index (Philox counter word 1 of the reset draws) */
  float* obs;         /* [23][N] current observation; rows 15..22 = previous clipped action */
  uint32_t* status;   /* [2] or NULL: failure counters read (and cleared) by auv_get_status;
                         zero them before the first launch.  [0] non-finite state components
                         seen, [1] abandoned inter-wave waits of policy rollouts */
} auv_env_buffers;

/* MLP n_in=23 -> 256 -> 256 -> n_out, tanh hidden layers, linear output.  Every layer's
 * input is rounded to bf16 (nearest even); accumulation is fp32; biases fp32. */
typedef struct {
  const uint16_t* w;     /* device bf16 bits: W1[256][23], W2[256][256], W3[n_out][256],
                            contiguous, row-major (out, in) */
  const float* b;        /* device: b1[256], b2[256], b3[n_out] contiguous */
  const float* log_std;  /* device [8]; needed for AUV_ACT_POLICY_SAMPLE, else may be NULL */
  int32_t n_out;         /* 8 for the policy, 1 for a value net */
} auv_mlp;

/* Optional per-step outputs of auv_rollout (device, caller-owned; any may be NULL). */
typedef struct {
  float* obs;        /* [23][T][N] observation o_t each action was chosen on */
  float* act;        /* [8][T][N] action a_t before clipping */
  float* logp;       /* [T][N] Gaussian log-prob of a_t (AUV_ACT_POLICY_SAMPLE only) */
  float* value;      /* [T][N] V(o_t) (needs a value net) */
  float* reward;     /* [T][N] */
  float* done;       /* [T][N] 1.0 where the episode ended at step t, else 0.0 */
  float* last_value; /* [N] V(o_T) bootstrap value (needs a value net) */
  float* traj_state; /* [13][T+1][N] state before step 0 and after every step */
  float* stats;      /* [3][T] per step: sum of reward, sum of done, sum of |dp| */
  float* stats_work; /* workspace for stats: auv_stats_work_floats(N, T) floats */
} auv_rollout_buffers;

/* Number of floats of the stats workspace for N envs and T steps (3 T 4 ceil(N/64)). */
int64_t auv_stats_work_floats(int32_t n_envs, int32_t T);

/* Validates the configuration and buffers and creates a handle.  Makes no GPU call and
 * allocates no device memory.  global_step starts at 0. */
int auv_create(const auv_config* cfg, const auv_vehicle* veh, const auv_env_buffers* bufs,
               auv_env** out);
int auv_destroy(auv_env* env);

/* Resets every environment: episode 0, ep_step 0 (or staggered), Philox reset draws
 * (counter (global id, episode, 0, 0..7)), velocities 0, previous action 0, observation;
 * global_step back to 0. */
int auv_reset(auv_env* env, void* stream);

/* One control step of every environment.  Modes: AUV_ACT_EXTERNAL (actions [8][N] device),
 * AUV_ACT_RANDOM (actions ignored), AUV_ACT_POLICY_MEAN / AUV_ACT_POLICY_SAMPLE (policy
 * required, actions ignored; the step is the first step of auv_rollout with T = 1, bit for
 * bit, and k such steps equal one rollout of k steps).  reward [N] fp32, done [N] uint8 and
 * stats [3] (sums over envs) are optional outputs; stats needs stats_work
 * (auv_stats_work_floats(N, 1) floats).  global_step += 1.  AUV_EINVAL, nothing enqueued:
 * unknown mode, a policy in a non-policy mode or none in a policy mode, external mode
 * without actions, misaligned buffers, stats without stats_work. */
int auv_step(auv_env* env, int mode, const float* actions, const auv_mlp* policy, float* reward,
             uint8_t* done, float* stats, float* stats_work, void* stream);

/* T control steps of every environment in one launch.  Modes: AUV_ACT_RANDOM (actions
 * from Philox), AUV_ACT_EXTERNAL (actions from rbufs->act, read as [8][T][N]),
 * AUV_ACT_POLICY_MEAN / AUV_ACT_POLICY_SAMPLE (policy required; value optional).
 * global_step += T.  In the policy modes the waves of a workgroup order their work through
 * bounded waits; should one never complete (a defect, not an input condition), the launch
 * still ends and the affected environments' state is NaN. */
int auv_rollout(auv_env* env, int32_t T, int mode, const auv_mlp* policy,
                const auv_mlp* value, const auv_rollout_buffers* rbufs, void* stream);

/* auv_rollout for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same launches and
 * results, with the batch-statistics partials held in a device array of the library's own
 * (AUV_STATIC_STATS_FLOATS floats, 8 MiB, on every GPU the library runs on, kept until the
 * process ends) instead of rbufs->stats_work, which must be NULL.  Statistics of T steps need
 * 3 T G floats of it, G = the launch's partial groups: ceil(N / 16) for the random / external
 * modes up to 32768 envs, else ceil(N / 64); in the policy modes ceil(N / 16) below 8192 envs,
 * ceil(N / 32) below 16384, else ceil(N / 64) (on a 256-CU device).  Every call on a GPU shares
 * its array; each call rewrites the partials it reads, so nothing needs clearing, but calls
 * that overlap on one GPU (any handle, stream or thread) race and must be ordered by the
 * caller.  Calls no hipMalloc, hipFree or allocating library routine; the array's device
 * address is looked up once per device on the first call there.  AUV_EINVAL, nothing
 * enqueued: stats_work given, 3 T G beyond AUV_STATIC_STATS_FLOATS, or what auv_rollout
 * rejects. */
#define AUV_STATIC_STATS_FLOATS (2 * 1024 * 1024)
int auv_rollout_static(auv_env* env, int32_t T, int mode, const auv_mlp* policy,
                       const auv_mlp* value, const auv_rollout_buffers* rbufs, void* stream);

/* Generalised advantage estimation over a [T][N] rollout (backward scan per env):
 * delta_t = r_t + gamma (1 - d_t) V_{t+1} - V_t, V_T = last_value;
 * A_t = delta_t + gamma lambda (1 - d_t) A_{t+1}, A_T = 0; ret_t = A_t + V_t. */
int auv_gae(int32_t T, int32_t n_envs, const float* reward, const float* value,
            const float* done, const float* last_value, float gamma, float lambda,
            float* adv, float* ret, void* stream);

/* Stand-alone MLP forward: obs [23][N] -> out [n_out][N] (same bf16 quantisation points
 * as inside auv_rollout; the output layer's split-K partials are added in a different
 * grouping, so the two agree to fp32 rounding). */
int auv_mlp_forward(const auv_mlp* net, int32_t n_envs, const float* obs, float* out,
                    void* stream);

/* Failure detection (synchronises the stream).  Every environment kernel (step, rollout,
 * SHAC window) counts the non-finite components of each environment's 13 state values
 * where an episode ends (before the reset replaces them) and where the launch ends, and
 * adds the count to status[0] of the handle's buffers; a policy rollout whose inter-wave
 * wait gave up (see auv_rollout) adds 1 per affected tile to status[1].  This call waits for
 * the work enqueued on `stream`, copies both counters to the host, clears them and returns
 * AUV_ENONFINITE if either was nonzero, else AUV_OK.  nonfinite_count and abandoned_waits
 * (host, either may be NULL) receive the counts since the previous call.  AUV_EINVAL: the
 * handle has no status buffer.  AUV_ERUNTIME: the copy or the synchronisation failed.
 * Environments are not reset on a non-finite state (their episode ends stay on schedule). */
int auv_get_status(auv_env* env, uint32_t* nonfinite_count, uint32_t* abandoned_waits, void* stream);

/* The kernels' own number conversions applied to n 32-bit words (device, caller-owned,
 * 16-byte aligned), one output float per word, for checking them bit for bit against their
 * definitions:
 *   AUV_CONV_UNIFORM        (w >> 8) 2^-24, in [0, 1)            (every uniform draw)
 *   AUV_CONV_UNIFORM_OPEN0  ((w >> 8) + 1) 2^-24, in (0, 1]     (the Box-Muller radius input)
 *   AUV_CONV_AFFINE         lo + span (w >> 8) 2^-24 rounded once to fp32 (fused multiply-add;
 *                           the randomisation draws, with their fp32 (lo, span))
 *   AUV_CONV_BF16           the fp32 value with bits w rounded to bf16, nearest even (the
 *                           conversion of every MLP layer input), widened back to fp32
 * AUV_EINVAL, nothing enqueued: unknown kind, n outside [1, 2^31], NULL or misaligned buffers. */
enum { AUV_CONV_UNIFORM = 0, AUV_CONV_UNIFORM_OPEN0 = 1, AUV_CONV_AFFINE = 2, AUV_CONV_BF16 = 3 };
int auv_convert(int kind, int64_t n, const uint32_t* in, float lo, float span, float* out, void* stream);

/* Throughput probe of the units that bound the fused rollout: `blocks` workgroups of 256
 * threads, each lane running `iters` iterations of 8 independent chains of one instruction
 * (AUV_PROBE_EXP: v_exp_f32, AUV_PROBE_RCP: v_rcp_f32, AUV_PROBE_FMA: v_fma_f32;
 * AUV_PROBE_MFMA_BF16: v_mfma_f32_16x16x32_bf16, per wave).  The caller times the launch:
 * lane operations = 256 blocks iters 8 (MFMA: blocks 4 iters 8 instructions of 16384 FLOP).
 * sink: 256 blocks floats (device) that keep the results live.  AUV_EINVAL for an unknown
 * kind, blocks outside [1, 2^20], iters < 1, a NULL or misaligned sink. */
enum { AUV_PROBE_EXP = 0, AUV_PROBE_RCP = 1, AUV_PROBE_FMA = 2, AUV_PROBE_MFMA_BF16 = 3 };
int auv_probe_rate(int kind, int32_t blocks, int32_t iters, float* sink, void* stream);

/* Host-side step counter (Philox counter word 1 of action and noise draws); set it to
 * resume a saved run bit-exactly together with the state buffers. */
int64_t auv_get_global_step(const auv_env* env);
int auv_set_global_step(auv_env* env, int64_t step);

/* Bound on the number of polls of one wait between the waves of a policy-rollout
 * workgroup (0 restores the default, about one second of polling).  Only for exercising the
 * abandonment path described under auv_rollout: with a tiny bound the launch gives up early,
 * ends normally and leaves NaN state. */
int auv_set_sync_poll_limit(auv_env* env, uint32_t polls);

/* ---- The paper's own training task ------------------------------------------------------
 * By default an environment runs the workload task described at the top.  AUV_TASK_PAPER
 * switches it to the task the paper trains on (Sec. IV-B observation / action / reward,
 * Sec. IV-C randomisation, Sec. V-A references):
 *   action a in R^6 (rows 0-2 forces, 3-5 torques), u = clip(a, -1, 1),
 *     body wrench [f_max u_0:3, tau_max u_3:6] (no thruster allocation)
 *   observation (rows 0-11 of the obs buffers): body-frame position error R^T(p_goal - p),
 *     rotation vector of q^* (x) q_goal (shortest rotation), v, omega; rows 12-17 of the env
 *     obs buffer hold the moving average of past clipped actions (state), rows 18-22 are 0;
 *     recorded rollout observations have zeros in rows 12-22
 *   reward -w_pos |D dp|^2 - w_att |dtheta|^2 - w_act |u_3:6|^2 - w_vel |omega|^2
 *     - w_mavg |u - abar|^2, then abar <- beta abar + (1 - beta) u (abar = 0 at an episode start)
 *   reset: at rest at the origin, level; goal position U[-2, 2]^3 (reset words 12-14); goal
 *     attitude q_z(yaw) q_y(pitch) q_x(roll), each angle U[-euler_max, euler_max] (words
 *     15-17); weight gamma W with gamma U[gamma_lo, gamma_lo + gamma_span] (word 0, kept in
 *     params row 13); buoyancy centre at the centre of gravity (r_b ignored); no other
 *     randomisation, no current, goal pose constant over the episode
 *   random actions: action c <- word 2c, action 3 + c <- word 2c + 1 of the random-action
 *   counter; sampled actions: the Box-Muller pair of words (2c, 2c + 1) gives the noise of
 *   actions c and 3 + c.  The policy is a 23-256-256-8 network whose W1 columns 12-22 and
 *   W3 rows 6-7 are zero (a 12-256-256-6 network).  Batches of any size use the quad-layout
 *   loop.  Set the task before auv_reset. */
enum { AUV_TASK_WORKLOAD = 0, AUV_TASK_PAPER = 1 };

/* Hydrodynamics of the paper task.  AUV_FLUID_FOSSEN: the vehicle's added mass and linear +
 * quadratic damping (auv_vehicle).  AUV_FLUID_INERTIA_BOX: the inertia-based fluid model of the
 * paper's MJX simulation (Sec. IV-B): the vehicle is replaced by the uniform solid box with its
 * mass and principal inertia, s_i = sqrt(6 (I_j + I_k - I_i) / m); no added mass; viscous
 * drag -3 pi mu d v and torque -pi mu d^3 w (d = mean side); quadratic drag
 * -rho/2 s_j s_k |v_i| v_i and torque -rho s_i (s_j^4 + s_k^4) / 64 |w_i| w_i.  The constants are
 * derived on the host by auv_set_task; the kernels are the same. */
enum { AUV_FLUID_FOSSEN = 0, AUV_FLUID_INERTIA_BOX = 1 };

typedef struct {
  int32_t kind;          /* AUV_TASK_* */
  float f_max, tau_max;  /* N, N m at |u| = 1 (> 0) */
  float w_pos, d_pos[3], w_att, w_act, w_vel, w_mavg;   /* reward weights (>= 0) */
  float beta;            /* moving-average factor, 0 <= beta < 1 */
  float gamma_lo, gamma_span;   /* gravity factor range, gamma_lo > 0, span >= 0 */
  float euler_max;       /* goal Euler angle bound, rad, 0 <= euler_max <= pi */
  int32_t fluid;         /* AUV_FLUID_* */
  float density;         /* kg/m^3 (> 0), AUV_FLUID_INERTIA_BOX only */
  float viscosity;       /* Pa s (>= 0), AUV_FLUID_INERTIA_BOX only */
} auv_task;

/* Selects the task of a handle (no GPU call).  AUV_EINVAL for values out of range, for
 * AUV_TASK_PAPER with AUV_F_DR, AUV_F_CURRENT or AUV_F_LISSAJOUS set (not part of that task), or
 * for AUV_FLUID_INERTIA_BOX with an inertia no solid box has (I_i >= I_j + I_k). */
int auv_set_task(auv_env* env, const auv_task* task);

/* ---- PPO update of the policy and value MLPs on one minibatch ------------------------
 * The clipped-surrogate objective of PPO (Schulman et al. 2017; the on-policy learner of
 * paper Sec. III-A1, which gives no hyperparameters), over minibatch samples b:
 *   logp_b = sum_j [-((a_jb - mu_jb) / sigma_j)^2 / 2 - log sigma_j - log(2 pi) / 2],
 *            sigma = exp(log_std), mu = policy(o_b)
 *   rho_b  = exp(logp_b - logp_old_b)
 *   A^_b   = (A_b - mean A) / (std A + 1e-8) over the minibatch (population std) when
 *            normalize_adv, else A_b
 *   L = -(1/B) sum_b min(rho_b A^_b, clip(rho_b, 1 - eps, 1 + eps) A^_b)
 *       + (c_v / 2) (1/B) sum_b (V(o_b) - R_b)^2 - c_e sum_j (log sigma_j + (1 + log 2 pi) / 2)
 * The gradient of min() flows through the unclipped term where it is the smaller (ties
 * included).  The forward uses the bf16 weights and quantisation points of auv_mlp; the
 * backward rounds dL/dy, dz2 and dz1 to bf16 before each product (bf16 MFMA, fp32
 * accumulation); bias gradients and the tanh derivatives use the unrounded fp32 values.
 *
 * A network's parameters are one fp32 vector packed W1[256][23] | W2[256][256] |
 * W3[n_out][256] | b1[256] | b2[256] | b3[n_out] | log_std[8] (policy only), row-major;
 * gradients and Adam moments use the same packing.  The auv_mlp a rollout or auv_ppo_grad
 * reads is a view of it: w = the bf16 copy of W1 | W2 | W3 (auv_ppo_net.w_bf16),
 * b = theta + AUV_PPO_NW(n_out), log_std = theta + AUV_PPO_NW(n_out) + 512 + n_out. */
#define AUV_PPO_NW(n_out) (256 * 23 + 256 * 256 + (n_out) * 256)
#define AUV_PPO_NPARAM(n_out) (AUV_PPO_NW(n_out) + 512 + (n_out) + ((n_out) == 8 ? 8 : 0))

typedef struct {
  float clip_eps;      /* eps of the clipped surrogate, > 0 */
  float vf_coef;       /* c_v >= 0 */
  float ent_coef;      /* c_e (entropy bonus) */
  float max_grad_norm; /* global-norm clipping over both networks' gradients; <= 0: off */
  float lr, beta1, beta2, adam_eps; /* Adam (Kingma and Ba, Algorithm 1): lr > 0, 0 <= beta < 1, eps > 0 */
  int32_t normalize_adv;            /* nonzero: normalise advantages over the minibatch */
  int32_t n_actions;                /* actions of the policy, 1..8 (0 means 8): the loss uses
                                       outputs 0..n_actions-1; the others (zero padding) get zero
                                       gradients, so a padded 6-action policy stays padded */
} auv_ppo_config;

/* The rollout buffer a minibatch is drawn from (device, fp32, M = T N samples; sample
 * s = t N + i is column s of every row, as auv_rollout and auv_gae write them). */
typedef struct {
  const float* obs;  /* [23][M] */
  const float* act;  /* [8][M] actions before clipping */
  const float* logp; /* [M] log-prob of the action under the policy that acted */
  const float* adv;  /* [M] advantages */
  const float* ret;  /* [M] returns (value targets) */
  int64_t M;         /* 1 <= M < 2^31 */
} auv_ppo_batch;

/* One trainable network (device, caller-owned). */
typedef struct {
  float* theta;     /* fp32 parameters, packed as above */
  float* adam_m;    /* Adam first moments, same packing */
  float* adam_v;    /* Adam second moments */
  uint16_t* w_bf16; /* bf16 copy of W1 | W2 | W3 (what the auv_mlp view's w points at) */
  int32_t n_out;    /* 8 (policy) or 1 (value) */
} auv_ppo_net;

/* Bytes of device workspace auv_ppo_grad needs for a minibatch of B samples (-1 for B
 * outside [1, 2^24]); about 1.1 KB per sample from B = 131072 up, 1.6 KB below, plus 80 MB. */
int64_t auv_ppo_work_bytes(int32_t B);

/* Loss and gradients of one minibatch: entries idx[0..B-1] (int32 sample indices into the
 * batch; values outside [0, M) are clamped into it).  policy may be NULL: then only the value
 * loss and its gradient are computed (grad_policy, act, logp and adv are not read; stats[0],
 * [3], [4], [5] are 0 and the entropy term is absent), e.g. for a critic's regression.  Overwrites grad_policy
 * [AUV_PPO_NPARAM(8)], grad_value [AUV_PPO_NPARAM(1)] and stats [8]: surrogate loss, value
 * loss, entropy, approximate KL (mean of logp_old - logp), fraction of samples whose
 * gradient the clip removes, squared gradient norms of policy and value, and the clipping
 * factor auv_ppo_adam applies.  work: auv_ppo_work_bytes(B) bytes, 16-byte aligned.  Reads
 * of obs / act are coalesced when idx runs in blocks of 16 consecutive samples.  The
 * result is deterministic (same inputs, same bits).  AUV_EINVAL, nothing enqueued: B
 * outside [1, 2^24], NULL or misaligned pointers, a network other than 23-256-256-8 (with
 * log_std) / 23-256-256-1, or a config out of range. */
int auv_ppo_grad(const auv_ppo_config* cfg, const auv_mlp* policy, const auv_mlp* value,
                 const auv_ppo_batch* batch, const int32_t* idx, int32_t B, float* grad_policy,
                 float* grad_value, float* stats, void* work, void* stream);

/* One Adam step (t >= 1: steps so far, this one included) of both networks on the
 * gradients of auv_ppo_grad times stats[7]: rewrites theta, adam_m, adam_v and the bf16
 * weight copies (round to nearest even).  Either network may be NULL (it is then left
 * alone; its gradient is not read), not both.  AUV_EINVAL, nothing enqueued, for t < 1,
 * NULL or misaligned pointers, wrong n_out, or a config out of range. */
int auv_ppo_adam(const auv_ppo_config* cfg, int64_t t, const auv_ppo_net* policy,
                 const auv_ppo_net* value, const float* grad_policy, const float* grad_value,
                 const float* stats, void* stream);

/* A value net's regression over a batch in one call (SHAC's critic update, paper Sec. III-A3;
 * the value loss of auv_ppo_grad): `iterations` passes, each shuffling the M / 16 blocks of
 * 16 consecutive samples (Fisher-Yates, Knuth TAOCP Vol. 2 Algorithm P, driven by a
 * SplitMix64 stream started at `seed`) and taking `batches` minibatches of B = 16 floor(M / 16
 * / batches) samples from the front of that order; each minibatch is one auv_ppo_grad with the
 * policy left out and one auv_ppo_adam step of value_net (steps t0 + 1, t0 + 2, ...); without
 * gradient clipping (max_grad_norm <= 0) the Adam step runs inside the gradient's last kernel,
 * with the same bits as the separate calls.  value
 * is value_net's auv_mlp view; batch: obs and ret are read (M = batch->M).  The host
 * shuffles the next pass while the device runs the current one: a pass's indices are
 * written into one half of host_stage (int32 [2][16 floor(M / 16)], pinned host memory
 * owned by the caller) and copied asynchronously into the workspace, on a copy stream of the
 * library's own (one per device, created on first use, default priority) that events order
 * against `stream`, so that the copy runs beside the previous pass's kernels.  The call returns when
 * every copy has been made (the device may still run the last minibatches); grad_value
 * [AUV_PPO_NPARAM(1)] and stats [8] then hold the last minibatch's results.  work:
 * auv_ppo_fit_work_bytes(M, batches) bytes (-1 unless 16 <= M <= 2^28 and 1 <= batches <=
 * M / 16), 16-byte aligned.  Deterministic for a given seed.  AUV_EINVAL, nothing
 * enqueued: sizes out of range, NULL or misaligned pointers, iterations < 1, t0 < 0, or what
 * auv_ppo_grad / auv_ppo_adam reject. */
int64_t auv_ppo_fit_work_bytes(int64_t M, int32_t batches);
int auv_ppo_fit_value(const auv_ppo_config* cfg, const auv_mlp* value, const auv_ppo_net* value_net,
                      const auv_ppo_batch* batch, int32_t iterations, int32_t batches, uint64_t seed,
                      int64_t t0, int32_t* host_stage, float* grad_value, float* stats, void* work,
                      void* stream);

/* ---- SHAC: the actor gradient of one short window on the paper task -------------------
 * Short-Horizon Actor-Critic (Xu et al. 2022; the differentiable-simulation learner of
 * paper Sec. III-A3, trained on the paper task of auv_set_task).  One window of h control
 * steps of all N environments from their current state, with the policy in the loop:
 *   a_t = mu(o_t) (+ exp(log_std) eps_t in sample mode, the noise stream of auv_rollout),
 *   u_t = clip(a_t, -1, 1), s_{t+1} = the paper task's RK4 step, r_t its reward,
 *   L = -(1 / (N h)) sum_i [ sum_{t<h} gamma^t r_t + gamma^h V(o(s_h)) ]
 * and the gradient of L with respect to the policy parameters by reverse-mode
 * differentiation through the reward, the observation, RK4 + Fossen (relative-velocity form
 * without current; d|x|/dx = sign x), the clip (derivative 1 on [-1, 1], else 0) and the
 * policy network (the terminal value is differentiated with respect to s_h; the value
 * net is not trained here).  bf16 points: the forward's as auv_mlp; in the backward the
 * cotangent of each layer's pre-activation is rounded to bf16 before it reaches the layer's
 * weights, bias and input (bf16 MFMA, fp32 accumulation); tanh derivatives use fp32
 * activations.  The state adjoint is carried in fp32.
 *
 * The window may end the episode only at its last step (the environments must not have
 * staggered episodes, and (global_step mod H) + h <= H): there the terminal value is taken
 * on the final state before the reset, and the environment then resets as in a rollout.
 * Afterwards the environment buffers hold the window's end (or reset) state and
 * global_step += h. */
typedef struct {
  int32_t h;            /* window length, 1 <= h <= min(64, H) control steps */
  int32_t mode;         /* AUV_ACT_POLICY_SAMPLE, AUV_ACT_POLICY_MEAN or AUV_ACT_EXTERNAL */
  float gamma;          /* discount, 0 < gamma <= 1 */
  float max_grad_norm;  /* clipping factor stats[7] = min(1, c / (|grad| + 1e-6)); <= 0: 1 */
} auv_shac_config;

/* Window inputs and optional per-step outputs (device, caller-owned, [k][h][N] layouts). */
typedef struct {
  const float* actions; /* AUV_ACT_EXTERNAL: [8][h][N] actions before clipping (rows 0-5
                           used); the objective is then a function of these actions */
  float* obs;           /* [23][h][N] observation o_t each action was taken on (rows 12-22 0) */
  float* act;           /* [8][h][N] a_t before clipping (rows 6-7 0) */
  float* reward;        /* [h][N] r_t */
  float* done;          /* [h][N] 1.0 where the episode ended (only possible at t = h - 1) */
  float* grad_act;      /* [8][h][N] dL/da_t, the total derivative with respect to the action
                           before the clip (rows 6-7 0); in policy modes also dL/dmu_t */
  float* value_last;    /* [N] V(o(s_h)) on the final state before any reset (0 without a
                           value net) */
  float* grad_state0;   /* [13][N] dL/ds_0 */
} auv_shac_buffers;

/* Bytes of device workspace auv_shac_window needs for N environments and windows of h
 * steps (-1 outside N in [1, 2^22], h in [1, 64]); about 3.4 KB per environment-step plus
 * 81 MB. */
int64_t auv_shac_work_bytes(int32_t n_envs, int32_t h);

/* One SHAC window.  policy: the 23-256-256-8 network (a padded 12-256-256-6 net; log_std
 * for sample mode), required except in external mode.  value: a 23-256-256-1 network or
 * NULL (V = 0).  grad_policy: NULL or AUV_PPO_NPARAM(8) floats, overwritten with dL/dtheta
 * in the packed layout of auv_ppo_grad (entries of padding rows and columns are 0); not
 * allowed in external mode.  stats [8]: L, mean over envs of sum_t gamma^t r_t, mean V(o(s_h)),
 * 0, 0, |grad|^2, 0, clipping factor (the input of auv_ppo_adam).  work:
 * auv_shac_work_bytes(N, h) bytes, 16-byte aligned.  Deterministic (same inputs, same bits).
 * AUV_EINVAL, nothing enqueued: a handle without the paper task, staggered episodes, more
 * than 4 substeps, a window crossing an episode end, h out of range, wrong networks, NULL
 * or misaligned pointers. */
int auv_shac_window(auv_env* env, const auv_shac_config* cfg, const auv_mlp* policy, const auv_mlp* value,
                    const auv_shac_buffers* out, float* grad_policy, float* stats, void* work, void* stream);

/* Message for the calling thread's last error ("" if none). */
const char* auv_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* AUV_H */
