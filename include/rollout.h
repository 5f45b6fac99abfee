/* rollout.h -- C ABI of the MI355X batched multi-agent rollout library.
 *
 * The library steps thousands of independent gridworld episodes and runs each
 * agent's policy network forward to sample its next action, entirely on one
 * GPU.  One rollout step of one env is the Dec-POMDP step of the paper's
 * problem setting (Section 3): state s, joint action a = (a_1..a_N) drawn
 * from the decentralised policies pi_i(a_i | o_i), transition P(s' | s, a),
 * shared team reward r(s, a), per-agent observations o_i of s', and a fresh
 * episode from the initial-state distribution rho when one ends.  The
 * environments are those of Section 4 (environment table): Level-Based
 * Foraging (LBF), an Overcooked-style two-agent kitchen and two-player
 * Hanabi are implemented.
 *
 * Conventions for every entry point
 *   - Tensor pointers are DEVICE pointers (gfx950 global memory), owned by the
 *     caller, laid out densely in row-major order with the shapes given below.
 *     The library allocates no device memory and keeps no pointer after a call
 *     returns.  Struct arguments are HOST pointers, read during the call only.
 *   - `stream` is a hipStream_t passed as an opaque pointer (NULL = the null
 *     stream).  Work is enqueued on it and the call returns without waiting;
 *     results are ready when the stream is synchronised.
 *   - Arguments are validated on the host before anything is enqueued.  On a
 *     non-zero status nothing was launched; rollout_last_error() describes
 *     the failure.  A device-side fault surfaces at the caller's next stream
 *     synchronisation, not as a status.
 *   - Step indices t are absolute: t = 0 is the step rollout_init prepares.
 *     Every random decision of env e at step t is a pure function of
 *     (seed, env_base + e, t): a run of 128 steps equals a run of 64 steps
 *     followed by a run of 64 steps from t0 = 64, bit for bit, and env e of a
 *     batch equals the same global env id in any other batch.
 *   - Random draws: Philox4x64-10 (Salmon et al., SC'11), key (seed, 0),
 *     counter (global env id, t, sub-stream, tag).  Actions are sampled by
 *     the Gumbel-max rule; see policy/sampling below.
 */
#ifndef MI355X_ROLLOUT_H
#define MI355X_ROLLOUT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t rl_status;
enum {
  RL_OK = 0,
  RL_EINVAL = -1,       /* a required pointer is NULL, a size is <= 0 or out of range */
  RL_EUNSUPPORTED = -2, /* env kind, dtype or size with no compiled kernel */
  RL_ESHAPE = -3,       /* policy dims disagree with the env's obs size / action count */
  RL_EDEVICE = -4       /* the HIP runtime reported an error when launching */
};

enum { RL_ENV_LBF = 0, RL_ENV_OVERCOOKED = 1, RL_ENV_HANABI = 2 };
enum { RL_F32 = 0, RL_BF16 = 1 };

/* Environment configuration (host struct).
 *
 * LBF (Level-Based Foraging): grid_h x grid_w cells (each 3..16, at most 256
 * cells), n_agents in 1..4 agents with levels 1..max_agent_level, n_food in
 * 1..8 foods with levels 1..max_food_level placed on interior cells, episodes
 * truncated after max_steps steps (>= 1).  Observations have
 * 3 * grid_h * grid_w features per agent; there are 6 actions
 * (0 noop, 1 north, 2 south, 3 west, 4 east, 5 load).  The exact rules are in
 * the LBF section below.
 *
 * Overcooked: n_agents == 2, oc_cook_time in 1..255, oc_soup_reward in
 * 0..2^20, max_steps >= 1; grid_h, grid_w, n_food and the level fields must
 * be 0.  Observations have 26 * 45 = 1170 features per agent and there are
 * 6 actions (0 noop, 1 north, 2 south, 3 west, 4 east, 5 interact).  Rules in
 * the Overcooked section below.
 *
 * Hanabi: n_agents == 2, hn_hand_size 5, hn_info_tokens 8, hn_life_tokens 3,
 * and either the standard game (hn_colors 5, hn_ranks 5: 658 features (0/1)
 * per agent, 20 actions) or the mini game of the paper's environment table
 * (hn_colors 3, hn_ranks 3: 18 cards with 3, 2, 1 copies of ranks 1..3 per
 * colour, 278 features, 16 actions: 5 discards, 5 plays, 3 colour and 3 rank
 * hints); any other positive sizes give RL_EUNSUPPORTED.  max_steps >= 1
 * (truncation; a game cannot last 100 moves, so 1000 never truncates).  Rules
 * in the Hanabi section below (written for 5 x 5; the mini game sizes every
 * section by its colours and ranks).
 * Fields of another kind must be 0 (RL_EINVAL otherwise). */
typedef struct {
  int32_t kind;            /* RL_ENV_* */
  int32_t n_envs;          /* E >= 1 envs in this batch */
  int32_t n_agents;        /* A */
  int32_t grid_h, grid_w;  /* LBF grid */
  int32_t n_food;          /* LBF foods per episode */
  int32_t max_agent_level; /* LBF agent levels are 1..max_agent_level (1..15) */
  int32_t max_food_level;  /* LBF food levels are 1..max_food_level (1..15) */
  int32_t max_steps;       /* episode step limit (truncation) */
  int32_t oc_cook_time;    /* Overcooked: steps a full pot cooks (0 for LBF) */
  int32_t oc_soup_reward;  /* Overcooked: reward of a served soup (0 for LBF) */
  int32_t hn_colors, hn_ranks, hn_hand_size, hn_info_tokens, hn_life_tokens; /* Hanabi (0 otherwise) */
  int32_t lbf_const_levels; /* LBF, 0 or 1: 1 is the constant-levels variant (the paper's LBF task table):
                               every agent at max_agent_level and every food at max_food_level, which
                               must not exceed n_agents * max_agent_level; the level draws of a reset are
                               still made and ignored, so cells are those of the drawn-levels game.
                               0 (and for other kinds) = levels drawn at each reset */
  int64_t env_base;        /* global id of env 0 of this batch (>= 0) */
  uint64_t seed;           /* Philox key word 0 */
} rl_env_config;

/* Policy: x -> tanh(x W1^T + b1) -> tanh(. W2^T + b2) -> . W3^T + b3, one
 * network shared by every agent (host struct holding device pointers).
 * W_l is [dims[l+1], dims[l]] row-major (the nn.Linear layout) and b_l is
 * [dims[l+1]], both of `dtype`.  Observations fed to the network have the
 * same dtype; logits are always float32.  In RL_BF16 the hidden activations
 * are rounded to bfloat16 (nearest even) before the next layer and every
 * product is accumulated in float32.
 * Limits: n_layers == 3; dims[0] (D) in 1..2048; dims[1], dims[2] multiples of
 * 16 in 16..512; dims[3] (nA) in 1..32. */
typedef struct {
  int32_t dtype;    /* RL_F32 or RL_BF16 */
  int32_t n_layers; /* must be 3 */
  int32_t dims[4];  /* D, H1, H2, nA */
  const void* W[3];
  const void* b[3];
  /* Optional (RL_BF16 only): a copy of W[0..2] in the fragment-major layout
   * written by rl_policy_pack, or NULL.  When set, the streamed-weight
   * kernels (the kitchen and Hanabi rollouts, the wide-layer policy_forward)
   * read their operands from it, 1 KB contiguous per load instead of 16 rows
   * x 64 bytes; results are bit-identical to reading W.  Must be 16-byte aligned and stay valid and
   * unchanged while calls that use the policy run. */
  const void* packed;
} rl_policy;

/* Trajectory outputs of rollout_run (host struct of device pointers).  Any
 * pointer may be NULL ("do not write").  T = n_steps of the call. */
typedef struct {
  void* obs;         /* [T, E, A, D] policy dtype: o_t, the observation a_t was sampled from */
  int32_t* actions;  /* [T, E, A] a_t */
  float* logits;     /* [T, E, A, nA] policy logits at o_t (illegal actions are -inf) */
  float* reward;     /* [T, E] shared team reward of the transition at t */
  uint8_t* done;     /* [T, E] bit 0 terminated, bit 1 truncated; an env with done != 0
                        starts a fresh episode at t + 1 */
  void* obs_last;    /* [E, A, D] policy dtype: o_{t0+T}, the observation after the last step */
} rl_traj;

/* Actor-critic outputs of rollout_run_ac (host struct of device pointers).
 * Any pointer may be NULL ("do not write"). */
typedef struct {
  float* value;       /* [T, E, A] V(o_t): the critic's value of the observation a_t was sampled from */
  float* logp;        /* [T, E, A] log pi(a_t | o_t) under the float32 logits a_t was sampled from */
  float* value_last;  /* [E, A] V(o_{t0+T}), for bootstrapping the next advantage estimate */
} rl_ac_traj;

/* ---- host-only queries (no device work) ---- */

/* Bytes of the env state buffer for `cfg` (0 if cfg is invalid). */
size_t rl_state_bytes(const rl_env_config* cfg);
/* Features per agent observation, D (<= 0 if cfg is invalid). */
int32_t rl_obs_dim(const rl_env_config* cfg);
/* Actions per agent, nA (<= 0 if cfg is invalid). */
int32_t rl_num_actions(const rl_env_config* cfg);
/* Description of the last failure on the calling thread; valid until the
 * thread's next call into the library. */
const char* rollout_last_error(void);

/* ---- entry points ---- */

/* rho: draw the first episode of every env at t = 0 (Section 3, initial-state
 * distribution) and write its observation.
 *   state     [rl_state_bytes(cfg)] bytes, written (layout below).
 *   obs       [E, A, D] of obs_dtype, written; may be NULL.
 *   legal     [E, A, nA] uint8 legal-action mask (1 = legal), written; may be NULL. */
rl_status rollout_init(const rl_env_config* cfg, void* state, void* obs, int32_t obs_dtype,
                       uint8_t* legal, void* stream);

/* P, r, Omega with injected actions: advance every env n_steps steps from
 * absolute step t0 (Section 3 transition and reward), auto-resetting ended
 * episodes.  Step k (0 <= k < n_steps) applies actions[k] at t = t0 + k.
 *   actions   [n_steps, E, A] int32, read.  An action outside 0..nA-1 (or,
 *             for envs with a legality mask, an illegal one) acts as the
 *             lowest-index legal action (LBF: noop).
 *   obs_out   [n_steps, E, A, D] of obs_dtype: o_{t+1}, after any reset; may be NULL.
 *   reward    [n_steps, E] float32; done [n_steps, E] uint8; either may be NULL.
 *   legal_out [n_steps, E, A, nA] uint8 masks for o_{t+1}; may be NULL. */
rl_status rollout_step(const rl_env_config* cfg, void* state, uint64_t t0, int32_t n_steps,
                       const int32_t* actions, void* obs_out, int32_t obs_dtype, float* reward,
                       uint8_t* done, uint8_t* legal_out, void* stream);

/* Bytes of the fragment-major weight copy of an RL_BF16 policy (host query;
 * 0 when the policy is invalid or float32).  Layer l (W_l of N = dims[l+1]
 * rows and K = dims[l] columns) takes ceil(N/16) * ceil(K/32) KB, starting at
 * a 256-byte boundary after the previous layer; for each 16-row tile t and
 * 32-wide K step s the 1 KB block at ((t * ceil(K/32) + s) * 1024) holds, for
 * lane l = 0..63, the 8 bf16 W_l[16t + l%16][32s + 8(l/16) + j], j = 0..7
 * (zero outside W_l), i.e. the MFMA B operands of that tile and step. */
size_t rl_policy_packed_bytes(const rl_policy* policy);

/* Writes that copy of policy->W into `packed` (device, 16-byte aligned, at
 * least rl_policy_packed_bytes bytes, caller-owned), enqueued on `stream`.
 * policy->packed is ignored.  RL_EUNSUPPORTED for a float32 policy. */
rl_status rl_policy_pack(const rl_policy* policy, void* packed, void* stream);

/* pi(. | o): the logits of the decentralised policy pi_i(a_i | o_i) of
 * Section 3 (problem setting: each agent acts on its own observation) for
 * `rows` observations, i.e. the policy network of the step on its own.
 *   obs    [rows, D] of policy->dtype, read.
 *   legal  [rows, nA] uint8 or NULL (all legal); an illegal action's logit is -inf.
 *   logits [rows, nA] float32, written. */
rl_status policy_forward(const rl_policy* policy, const void* obs, const uint8_t* legal,
                         int64_t rows, float* logits, void* stream);

/* The full rollout loop of the Dec-POMDP step of Section 3 (problem
 * setting): for t = t0 .. t0+n_steps-1, every env observes (o_i of s), every
 * agent samples a_i from pi(. | o_i) by Gumbel-max, the joint action moves
 * the env through P and yields the shared reward r(s, a), and an ended
 * episode restarts from rho; results go to `out` (any field NULL = skipped).
 * Runs as one persistent kernel; `state` is left at step t0 + n_steps. */
rl_status rollout_run(const rl_env_config* cfg, const rl_policy* policy, void* state,
                      uint64_t t0, int32_t n_steps, const rl_traj* out, void* stream);

/* rollout_run for an actor-critic network: the policy's last layer has
 * nA + 1 outputs, the first nA being the action logits (sampled as in
 * rollout_run) and the last the critic's value V(o) of the same observation
 * (a value head on the shared trunk).  Besides `out` it writes `ac`: V(o_t),
 * log pi(a_t | o_t) = l_a - (m + log sum_i exp(l_i - m)) over the nA float32
 * logits l (m their maximum), and V of the observation after the last step.
 * These are what a PPO-style learner consumes after a rollout (the learners
 * the paper benchmarks build on PPO, appendix "Algorithms Overview").  LBF
 * envs only (RL_EUNSUPPORTED otherwise); dims[3] must be nA + 1 (RL_ESHAPE). */
rl_status rollout_run_ac(const rl_env_config* cfg, const rl_policy* policy, void* state, uint64_t t0,
                         int32_t n_steps, const rl_traj* out, const rl_ac_traj* ac, void* stream);

/* Generalised advantage estimation over a stored trajectory (float32), a
 * backward scan per (env, agent):
 *   delta_t = r_t + gamma (1 - d_t) V_{t+1} - V_t,  A_t = delta_t + gamma lambda (1 - d_t) A_{t+1},
 *   A_T = 0, V_T = value_last, R_t = A_t + V_t,
 * with d_t = 1 where done[t] != 0: an episode end (terminated or truncated)
 * cuts the recurrence, as the next observation starts a fresh episode.
 *   reward [T, E] float32, done [T, E] uint8, value [T, E, A] float32 and
 *   value_last [E, A] float32 read; adv [T, E, A] written; ret [T, E, A]
 *   written, may be NULL.  gamma and lambda in [0, 1]. */
rl_status rl_gae(const float* reward, const uint8_t* done, const float* value, const float* value_last,
                 int32_t n_steps, int32_t n_envs, int32_t n_agents, float gamma, float lambda, float* adv,
                 float* ret, void* stream);

/* The rollout of rollout_run with one policy per agent slot, drawn from a
 * population: the ego agent and its teammates of the ad hoc teamwork objective
 * (Section 3, the J_AHT equation: the ego policy paired with teammate
 * policies from a held-out set), e.g. the cross-play matrix of a population
 * evaluated as one batch.  LBF envs only (RL_EUNSUPPORTED otherwise).
 *   pop           one policy's dtype and dims, with W[l] pointing at
 *                 n_policies matrices [dims[l+1], dims[l]] stacked
 *                 ([n_policies, dims[l+1], dims[l]] row-major) and b[l] at
 *                 [n_policies, dims[l+1]]; device memory, read.
 *   n_policies    1..4096.
 *                 pop->packed (optional, bf16): n_policies packed copies
 *                 (rl_policy_pack of each policy), policy q at
 *                 q * rl_policy_packed_bytes(pop) bytes.
 *   policy_index  [E, A] int32 device, read: agent a of env e acts with policy
 *                 policy_index[e * A + a]; an index outside 0..n_policies-1
 *                 selects policy 0.
 * Everything else as rollout_run.  A workgroup's 16 envs run each layer once
 * per distinct policy among their agents, so the cost grows with that count
 * (assigning teammates to blocks of envs keeps it at two). */
rl_status rollout_run_pop(const rl_env_config* cfg, const rl_policy* pop, int32_t n_policies,
                          const int32_t* policy_index, void* state, uint64_t t0, int32_t n_steps,
                          const rl_traj* out, void* stream);

/* rollout_run with heuristic teammates in the loop (LBF only): agent a of
 * env e acts with the heuristic teammates[e * A + a] when it is in 0..10, and
 * with `policy` otherwise.  The heuristics are the paper's Greedy and
 * Sequential LBF teammates (Appendix, the table of heuristic teammates), read
 * as deterministic policies of the env state: kinds 0-2 Greedy toward the
 * uneaten food closest to the agent / to agent (a + 1) mod A / to both (sum of
 * Manhattan distances); 3-4 Greedy toward the lowest / highest food level
 * (then the closest); 5-8 Sequential in row-major, reverse row-major,
 * column-major, reverse column-major order of the food cells; 9-10
 * Sequential nearest / farthest first by Manhattan distance from the agent's
 * cell at the start of its episode (for an episode already running at t0,
 * the cell the reset of step t0 - steps placed it on, i.e. where that
 * episode began).  Ties go to the lowest food index.  Next to its target the agent loads; otherwise it
 * steps along the axis with more distance left (rows on ties), or along the
 * other axis when that cell holds an uneaten food or another agent and the
 * other axis also closes in.  A heuristic agent's logits are 0 for its
 * action and -inf for the others (so the sampler returns that action).
 *   teammates [E, A] int32, read.  Everything else as rollout_run. */
rl_status rollout_run_teams(const rl_env_config* cfg, const rl_policy* policy, const int32_t* teammates,
                            void* state, uint64_t t0, int32_t n_steps, const rl_traj* out, void* stream);

/* ---- recurrent S5 actor-critic (the paper's ego agent, Appendix on agent
 * architectures: dense encoder, S5 of model width 128 and state 128, actor
 * and critic heads of three 1024-unit layers) ----
 *
 * Network, per agent row and step:  u = tanh(W_enc o + b_enc)       [H]
 *   x_t = Lambda_bar x_{t-1} + B_bar u    (complex [P]; x_{t-1} := 0 when o
 *                                          is the first of its episode)
 *   y = Re(C x_t) + d * u                 [H]
 *   actor:  three tanh layers of width F, then nA logits;
 *   critic: three tanh layers of width F, then one value.
 * S5 is Smith et al., ICLR 2023; the reset at episode starts follows Lu et
 * al., NeurIPS 2023.  Dense layers are bfloat16 (nn.Linear layout [out, in]),
 * every product accumulates in float32 and u, y and the head activations are
 * rounded to bfloat16; the S5 parameters and state are float32.  Every
 * pointer is device memory, 16-byte aligned.
 * Limits: dtype RL_BF16; H a multiple of 64 in 64..256; P a multiple of 16 in
 * 16..128; F a multiple of 128 in 128..4096; nA in 1..16; D (the env's
 * observation size) at most 1024, and the encoder/S5 tile within 160 KiB of
 * LDS (RL_EUNSUPPORTED otherwise; D 192, H 128, P 128 takes 128 KiB). */
typedef struct {
  int32_t dtype;       /* RL_BF16 */
  int32_t obs_dim;     /* D, must equal rl_obs_dim(cfg) */
  int32_t d_model;     /* H */
  int32_t d_state;     /* P */
  int32_t head_width;  /* F */
  int32_t n_actions;   /* nA, must equal rl_num_actions(cfg) */
  const void* w_enc;   /* [H, D] */
  const void* b_enc;   /* [H] */
  const float* lambda_bar; /* [2, P]: real parts, then imaginary parts (from rl_s5_discretize) */
  const float* b_bar;      /* [2, P, H] */
  const float* c;          /* [2, H, P] */
  const float* d;          /* [H] */
  const void* actor_w[4];  /* [F, H], [F, F], [F, F], [nA, F] */
  const void* actor_b[4];
  const void* critic_w[4]; /* [F, H], [F, F], [F, F], [1, F] */
  const void* critic_b[4];
} rl_s5_policy;

/* Zero-order hold of the continuous S5 parameters (Smith et al., Section 2):
 * lambda_bar = exp(lambda dt), b_bar = (lambda_bar - 1) / lambda * b with
 * dt = exp(log_dt), evaluated in double precision and rounded to float32.
 *   lambda [2, P] (real parts < 0), log_dt [P], b [2, P, H] read;
 *   lambda_bar [2, P], b_bar [2, P, H] written.  P, H >= 1. */
rl_status rl_s5_discretize(int32_t d_state, int32_t d_model, const float* lambda, const float* log_dt,
                           const float* b, float* lambda_bar, float* b_bar, void* stream);

/* Bytes of the device workspace rollout_run_s5 needs for cfg and policy
 * (hidden activations of both heads, y, two observation tiles, actions);
 * 0 if either is invalid. */
size_t rl_s5_workspace_bytes(const rl_env_config* cfg, const rl_s5_policy* policy);

/* The rollout loop of rollout_run_ac with the recurrent S5 actor-critic
 * (LBF only).  Each step runs the policy on o_t (the carried state zeroed
 * for rows whose episode starts at o_t, i.e. whose env step counter is 0),
 * samples a_t by Gumbel-max from the logits, and steps the envs.
 *   carry      [E * A, 2, P] float32 (rows env-major; real then imaginary
 *              parts): the S5 state of every agent, read and left at step
 *              t0 + n_steps; its content is irrelevant for rows that start an
 *              episode at t0 (zeros are a valid start).
 *   out, ac    as rollout_run_ac; value_last is V(o_{t0+T}) computed without
 *              advancing carry.
 *   workspace  rl_s5_workspace_bytes(cfg, policy) bytes of device memory,
 *              owned by the caller, not read across calls.
 * The call is a sequence of kernels on `stream` (per step: encoder and S5,
 * three head layers, output layers and sampling, env step). */
rl_status rollout_run_s5(const rl_env_config* cfg, const rl_s5_policy* policy, void* state, float* carry,
                         uint64_t t0, int32_t n_steps, const rl_traj* out, const rl_ac_traj* ac, void* workspace,
                         size_t workspace_bytes, void* stream);

/* rollout_run_s5 without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc).  The workspace is a file-scope device
 * array of the library, 80 MiB (83,886,080 bytes) on every GPU the library
 * runs on, held until the process ends; its address on the current GPU is
 * resolved on the first call there.  Calls whose rl_s5_workspace_bytes
 * exceeds 80 MiB fail with RL_EINVAL before anything is launched (4096 LBF
 * 8x8 envs of 2 agents at D 192, H 128, P 128, F 1024 need 75.7 MB).  No
 * call allocates memory.  Nothing in the array needs to start at zero: every
 * call writes each workspace region before reading it.  Every call on one GPU
 * shares that GPU's array, so calls that overlap in time on one GPU (on
 * different streams or host threads) race and must be serialised by the
 * caller.  Arguments, results and errors otherwise as rollout_run_s5. */
rl_status rollout_run_s5_noalloc(const rl_env_config* cfg, const rl_s5_policy* policy, void* state, float* carry,
                                 uint64_t t0, int32_t n_steps, const rl_traj* out, const rl_ac_traj* ac,
                                 void* stream);

/* Gumbel-max sampling of the actions of step t from given logits (the
 * sampling stage of rollout_run on its own).
 *   logits  [E, A, nA] float32 read;  legal [E, A, nA] uint8 or NULL;
 *   actions [E, A] int32 written. */
rl_status rollout_sample(const rl_env_config* cfg, uint64_t t, const float* logits,
                         const uint8_t* legal, int32_t* actions, void* stream);

/* The sampler's noise function on its own: g[i] = float32(-ln(-ln((u[i] + 1/2) / 2^24)))
 * evaluated in double precision, for 24-bit inputs u[i] (higher bits ignored).
 *   u [n] uint32 read, g [n] float32 written. */
rl_status rl_gumbel_noise(const uint32_t* u, int64_t n, float* g, void* stream);

/* ---- sampling ----
 * Action a of agent i of env e at step t uses Philox block
 * (seed; env_base + e, t, i * 256 + a / 8, TAG_ACTION = 2), word (a % 8) / 2,
 * its high 32-bit half for even a and low half for odd a; u = half >> 8 and
 * g = noise(u).  The action is argmax_a float32(logit_a + g_a) with illegal
 * actions and NaN scores counted as -inf, ties to the lowest index, and
 * action 0 when every score is -inf.
 *
 * ---- LBF ----
 * State buffer: int32 planes of E entries each, plane p of env e at
 * state[p * E + e]:
 *   p = i            (0 <= i < A)  agent i cell, row * grid_w + col
 *   p = A + i                       agent i level
 *   p = 2A + j       (0 <= j < F)  food j cell
 *   p = 2A + F + j                  food j level
 *   p = 2A + 2F                     eaten-food bitmask (bit j = food j eaten)
 *   p = 2A + 2F + 1                 steps taken in the current episode
 *   p = 2A + 2F + 2                 sum of the episode's food levels
 * Reset at step t draws 32-bit words k = 0.. from blocks
 * (seed; env, t, k / 8, TAG_RESET = 1), word (k % 8) / 2, high half first,
 * and maps word k to 0..n-1 as (k_word * n) >> 32: A agent levels
 * 1..max_agent_level, then F food levels 1..min(max_food_level, sum of agent
 * levels), then F food cells (the drawn index among the interior cells free
 * of food, row-major), then A agent cells (the drawn index among cells free of
 * food and earlier agents, row-major).
 * Step: a move (1..4) succeeds iff the target is on the grid, holds no uneaten
 * food and no agent before the step, and no other agent moves to the same
 * target; food j is eaten iff the agents choosing load that are 4-adjacent to
 * it have levels summing to >= its level (a loader counts for every adjacent
 * food); reward = float32(eaten levels) / float32(sum of food levels);
 * done bit 0 when every food is eaten, bit 1 when the episode reaches
 * max_steps; a done env is reset with the draws of step t + 1.
 * Observation of agent i, 3 planes of grid_h x grid_w (plane-major): agent
 * levels at agent cells, uneaten food levels at food cells, 1 at agent i's
 * own cell.  Every action is always legal.
 *
 * ---- Overcooked ----
 * A kitchen of W x H cells (W in 5..9, H in 4..5) at the top-left of a fixed
 * 5 x 9 canvas, cell id = row * 9 + col; canvas cells outside the kitchen are
 * counters.  Cell kinds: floor, counter, onion dispenser, plate dispenser,
 * pot (one or two), serving cell.  Each env keeps one kitchen for the whole
 * launch sequence; it is drawn from the stream (seed; env, attempt, k / 8,
 * TAG_LAYOUT = 3) with 32-bit draws k = 0.. taken as for LBF resets and
 * u(n) = (draw * n) >> 32: W = 5 + u(5), H = 4 + u(2); u(((H-2)(W-2)) / 4 + 1)
 * interior counters, each on the u(n)-th remaining interior floor cell
 * (row-major); n_onion = 1 + u(2), n_pot = 1 + u(2); then n_onion onion
 * dispensers, n_pot pots, one plate dispenser and one serving cell, each on
 * the u(n)-th candidate, a border counter that is not a kitchen corner and has
 * a floor 4-neighbour (row-major).  An attempt is kept iff the floor is
 * 4-connected with >= 2 cells and no station ran out of candidates; attempts
 * 0..63 are tried in order, then attempt 64 with no interior counters.
 * Reset at step t (stream TAG_RESET): agent 0 on the u(n_floor)-th floor
 * cell, agent 1 on the u(n_floor - 1)-th of the others, both facing north,
 * empty hands, pots and counters, step count 0.
 * Step: a move (1..4) turns the agent that way even when blocked, and
 * succeeds iff the faced cell is floor and held no agent before the step and
 * the other agent does not move there too.  Then interact (5), agent 0 first,
 * on the faced cell: take an onion / a plate from a dispenser with an empty
 * hand; put an onion in a pot with < 3 onions (the third sets the timer to
 * cook_time); take soup from a pot with 3 onions and timer 0 with a plate
 * (the pot empties); deliver soup on the serving cell (reward += soup_reward);
 * place a held item on an empty counter or pick one up with an empty hand.
 * Pots that were cooking (3 onions, timer > 0) before the step count down by
 * one.  done = 2 (truncated) when the episode reaches max_steps; a done env
 * is reset (kitchen kept) with the draws of step t + 1.  Out-of-range actions
 * act as noop; every action is always legal.
 * State buffer: 32 int32 planes of E entries (plane p of env e at
 * state[p * E + e]): 0-17 nine 45-bit cell masks as (low, high) word pairs --
 * floor, counter, onion dispenser, plate dispenser, pot, serving cell, onion /
 * plate / soup lying on a counter; 18 W | H << 8; 19-20 agent cells; 21-22
 * facings (0 N, 1 S, 2 W, 3 E); 23-24 held items (0 none, 1 onion, 2 plate,
 * 3 soup); 25-26 the pot cells in row-major order (-1: no second pot); 27-28
 * onions in those pots; 29-30 their timers; 31 steps taken in the episode.
 * Observation of agent i, 26 planes of 45 canvas cells (plane-major): 0 own
 * cell, 1 other agent's cell, 2-5 own facing and 6-9 the other's (at the
 * agent's cell), 10-14 counter / onion / plate / pot / serving cells, 15-17
 * onion / plate / soup on a counter, 18-20 own held onion / plate / soup and
 * 21-23 the other's (at the holder's cell), 24 onions in each pot and 25 its
 * remaining cook timer (at the pot cell).
 *
 * ---- Hanabi ----
 * Cards: id = colour * 5 + rank - 1; per colour, rank 1 has 3 copies, ranks
 * 2-4 two, rank 5 one (50 cards).  Reset at step t: the ordered deck (colours
 * in order, ranks ascending with their copies) is shuffled by Fisher-Yates,
 * for i = 49 down to 1 swapping cards i and j = u(i + 1), with draw k = 0..48
 * of the TAG_RESET stream taken as for LBF; player 0 holds deck[0..4] in slots
 * 0..4, player 1 deck[5..9], deck[10] is drawn next; player 0 moves first
 * with 8 info tokens and 3 lives.
 * Actions of the player to move: 0-4 discard slot, 5-9 play slot, 10-14
 * hint colour c to the partner, 15-19 hint rank r.  Legal: play a held slot;
 * discard a held slot when tokens < 8; hint when tokens > 0 and the partner
 * holds a matching card.  The other player has no legal action: its mask row
 * is all zero, its logits all -inf, and its sampled / injected action (0)
 * is ignored.  An illegal injected action of the mover acts as its lowest
 * legal action.
 * Step: a play that is one above its colour's firework extends it (reward
 * +1; a completed firework returns a token if below 8), otherwise the card
 * is discarded and a life lost; a discard returns a token.  The hand then
 * closes up and the next deck card, if any, enters the last slot with blank
 * knowledge.  A hint costs a token: matching partner cards learn that value
 * exactly, the others lose it from their possible set.  The game ends (done
 * bit 0) when the last life is lost (that step's reward is minus the
 * fireworks total, so the game scores 0), when every firework is complete,
 * or on the second move after the move that drew the last card.
 * State buffer: 35 int32 planes of E entries (plane p of env e at
 * state[p * E + e]): 0-12 the deck, card k in byte k % 4 of plane k / 4;
 * 13-14 the hands (5-bit card ids, slot s at bit 5s); 15-16 cards held;
 * 17-18 possible colours and 19-20 possible ranks (5-bit masks, slot s at bit
 * 5s); 21-22 hinted colour + 1 and 23-24 hinted rank (3 bits per slot, 0 =
 * none); 25 firework heights (3 bits per colour); 26-27 discarded copies
 * (2 bits per card id, ids 0-15 then 16-24); 28 info tokens; 29 lives; 30
 * player to move; 31 moves left after the deck ran out (-1 before); 32 index
 * of the next deck card; 33 steps taken; 34 the last move (bit 0 present, 1
 * actor, 2-3 kind: play, discard, hint colour, hint rank; 4 hint target; 5-7
 * hinted colour + 1; 8-10 hinted rank; 11-15 revealed slots; 16-18 acted slot
 * + 1; 19-23 acted card + 1; 24 play succeeded; 25 token gained).
 * Observation of agent i, 658 features (0/1): the partner's hand (5 slots x
 * 25 card one-hot), 2 bits for a short hand (own, partner), a 40-bit
 * thermometer of the cards left in the deck, per colour a one-hot of its
 * firework height (25), token (8) and life (3) thermometers, per card id a
 * thermometer of its discarded copies (50), the last move (55: actor relative
 * to i, kind, hint target relative to i, hinted colour, hinted rank, revealed
 * slots, acted slot, acted card, play succeeded, token gained), and the
 * knowledge of agent i's then the partner's hand (5 slots x (25 plausible
 * cards, hinted colour, hinted rank)). */

#ifdef __cplusplus
}
#endif
#endif /* MI355X_ROLLOUT_H */
