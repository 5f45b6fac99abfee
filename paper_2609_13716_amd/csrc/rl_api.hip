// C-ABI entry points: host-side validation, then one kernel launch on the
// caller's stream.  No device memory is allocated and no call waits on the
// device.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "rollout.h"
#include "rl_internal.h"

namespace {

thread_local char g_err[512] = "";

rl_status fail(rl_status code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

rl_status ok() {
  g_err[0] = '\0';
  return RL_OK;
}

rl_status launched(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(RL_EDEVICE, "%s: launch failed: %s", what, hipGetErrorString(e));
  return ok();
}

bool valid_dtype(int32_t dt) { return dt == RL_F32 || dt == RL_BF16; }

// A validated env configuration: its kind and the kernel parameters of that kind.
struct EnvSpec {
  int kind;
  rl::LbfParams lbf;
  rl::OcParams oc;
  rl::HnParams hn;
  int E, A, D, NA;
  size_t state_bytes;
};

rl_status check_lbf(const rl_env_config* cfg, EnvSpec* es) {
  if (cfg->n_agents < 1 || cfg->n_agents > rl::LBF_MAXA)
    return fail(RL_EINVAL, "LBF n_agents %d outside 1..%d", cfg->n_agents, rl::LBF_MAXA);
  if (cfg->n_food < 1 || cfg->n_food > rl::LBF_MAXF)
    return fail(RL_EINVAL, "LBF n_food %d outside 1..%d", cfg->n_food, rl::LBF_MAXF);
  if (cfg->grid_h < 3 || cfg->grid_h > 16 || cfg->grid_w < 3 || cfg->grid_w > 16)
    return fail(RL_EINVAL, "LBF grid %dx%d outside 3..16", cfg->grid_h, cfg->grid_w);
  const int hw = cfg->grid_h * cfg->grid_w;
  if (cfg->n_food > (cfg->grid_h - 2) * (cfg->grid_w - 2))
    return fail(RL_EINVAL, "LBF n_food %d exceeds the %d interior cells", cfg->n_food,
                (cfg->grid_h - 2) * (cfg->grid_w - 2));
  if (cfg->n_food + cfg->n_agents > hw) return fail(RL_EINVAL, "LBF grid too small for agents and food");
  if (cfg->max_agent_level < 1 || cfg->max_agent_level > 15 || cfg->max_food_level < 1 || cfg->max_food_level > 15)
    return fail(RL_EINVAL, "LBF levels must be in 1..15");
  if (cfg->lbf_const_levels != 0 && cfg->lbf_const_levels != 1)
    return fail(RL_EINVAL, "lbf_const_levels must be 0 or 1");
  if (cfg->lbf_const_levels && cfg->max_food_level > cfg->n_agents * cfg->max_agent_level)
    return fail(RL_EINVAL, "constant food level %d exceeds the agents' total level %d", cfg->max_food_level,
                cfg->n_agents * cfg->max_agent_level);
  if (cfg->oc_cook_time || cfg->oc_soup_reward || cfg->hn_colors || cfg->hn_ranks || cfg->hn_hand_size ||
      cfg->hn_info_tokens || cfg->hn_life_tokens)
    return fail(RL_EINVAL, "Overcooked/Hanabi fields must be 0 for LBF");
  rl::LbfParams& p = es->lbf;
  p.E = cfg->n_envs;
  p.A = cfg->n_agents;
  p.F = cfg->n_food;
  p.H = cfg->grid_h;
  p.W = cfg->grid_w;
  p.HW = hw;
  p.D = 3 * hw;
  p.Lmax = cfg->max_agent_level;
  p.Fmax = cfg->max_food_level;
  p.max_steps = cfg->max_steps;
  p.const_levels = cfg->lbf_const_levels;
  p.wmagic = rl::div_magic((uint32_t)cfg->grid_w);
  p.env_base = cfg->env_base;
  p.seed = cfg->seed;
  es->A = p.A;
  es->D = p.D;
  es->NA = rl::LBF_NACT;
  es->state_bytes = (size_t)rl::lbf_planes(p.A, p.F) * (size_t)p.E * sizeof(int32_t);
  return RL_OK;
}

rl_status check_overcooked(const rl_env_config* cfg, EnvSpec* es) {
  if (cfg->n_agents != 2) return fail(RL_EINVAL, "Overcooked has 2 agents, got %d", cfg->n_agents);
  if (cfg->oc_cook_time < 1 || cfg->oc_cook_time > 255)
    return fail(RL_EINVAL, "Overcooked cook_time %d outside 1..255", cfg->oc_cook_time);
  if (cfg->oc_soup_reward < 0 || cfg->oc_soup_reward > (1 << 20))
    return fail(RL_EINVAL, "Overcooked soup_reward %d outside 0..2^20", cfg->oc_soup_reward);
  if (cfg->grid_h || cfg->grid_w || cfg->n_food || cfg->max_agent_level || cfg->max_food_level ||
      cfg->lbf_const_levels || cfg->hn_colors || cfg->hn_ranks || cfg->hn_hand_size || cfg->hn_info_tokens || cfg->hn_life_tokens)
    return fail(RL_EINVAL, "LBF/Hanabi fields must be 0 for Overcooked");
  rl::OcParams& p = es->oc;
  p.E = cfg->n_envs;
  p.cook_time = cfg->oc_cook_time;
  p.soup_reward = cfg->oc_soup_reward;
  p.max_steps = cfg->max_steps;
  p.env_base = cfg->env_base;
  p.seed = cfg->seed;
  es->A = 2;
  es->D = rl::OC_D;
  es->NA = rl::OC_NACT;
  es->state_bytes = (size_t)rl::OC_PLANES_STATE * (size_t)p.E * sizeof(int32_t);
  return RL_OK;
}

rl_status check_hanabi(const rl_env_config* cfg, EnvSpec* es) {
  if (cfg->n_agents != 2) return fail(RL_EINVAL, "Hanabi is built for 2 players, got %d", cfg->n_agents);
  if (cfg->hn_colors < 1 || cfg->hn_ranks < 1 || cfg->hn_hand_size < 1 || cfg->hn_info_tokens < 1 ||
      cfg->hn_life_tokens < 1)
    return fail(RL_EINVAL, "Hanabi colours, ranks, hand size, info and life tokens must be >= 1");
  const bool std_game = cfg->hn_colors == rl::HnStd::C && cfg->hn_ranks == rl::HnStd::R &&
                        cfg->hn_hand_size == rl::HnStd::H;
  const bool mini_game = cfg->hn_colors == rl::HnMini::C && cfg->hn_ranks == rl::HnMini::R &&
                         cfg->hn_hand_size == rl::HnMini::H;
  if (!(std_game || mini_game) || cfg->hn_info_tokens != rl::HN_INFO || cfg->hn_life_tokens != rl::HN_LIVES)
    return fail(RL_EUNSUPPORTED,
                "Hanabi is built for 5 colours x 5 ranks or 3 colours x 3 ranks, hands of 5, 8 info tokens, 3 lives");
  if (cfg->grid_h || cfg->grid_w || cfg->n_food || cfg->max_agent_level || cfg->max_food_level ||
      cfg->lbf_const_levels || cfg->oc_cook_time || cfg->oc_soup_reward)
    return fail(RL_EINVAL, "LBF/Overcooked fields must be 0 for Hanabi");
  rl::HnParams& p = es->hn;
  p.E = cfg->n_envs;
  p.max_steps = cfg->max_steps;
  p.mini = mini_game ? 1 : 0;
  p.env_base = cfg->env_base;
  p.seed = cfg->seed;
  es->A = 2;
  es->D = mini_game ? rl::HnMini::OBS : rl::HnStd::OBS;
  es->NA = mini_game ? rl::HnMini::NACT : rl::HnStd::NACT;
  es->state_bytes = (size_t)rl::HN_PLANES_STATE * (size_t)p.E * sizeof(int32_t);
  return RL_OK;
}

// Checks cfg and fills the kernel parameters of its kind.
rl_status check_cfg(const rl_env_config* cfg, EnvSpec* es) {
  EnvSpec local;
  if (!es) es = &local;
  if (!cfg) return fail(RL_EINVAL, "cfg is NULL");
  if (cfg->kind != RL_ENV_LBF && cfg->kind != RL_ENV_OVERCOOKED && cfg->kind != RL_ENV_HANABI)
    return fail(RL_EINVAL, "unknown env kind %d", cfg->kind);
  if (cfg->n_envs < 1 || cfg->n_envs > (1 << 26)) return fail(RL_EINVAL, "n_envs %d outside 1..2^26", cfg->n_envs);
  if (cfg->env_base < 0) return fail(RL_EINVAL, "env_base must be >= 0");
  if (cfg->max_steps < 1) return fail(RL_EINVAL, "max_steps must be >= 1");
  es->kind = cfg->kind;
  es->E = cfg->n_envs;
  return cfg->kind == RL_ENV_LBF ? check_lbf(cfg, es)
         : cfg->kind == RL_ENV_OVERCOOKED ? check_overcooked(cfg, es)
                                          : check_hanabi(cfg, es);
}

rl_status check_policy(const rl_policy* pol, rl::PolicyArgs* a) {
  if (!pol) return fail(RL_EINVAL, "policy is NULL");
  if (!valid_dtype(pol->dtype)) return fail(RL_EUNSUPPORTED, "policy dtype %d unsupported", pol->dtype);
  if (pol->n_layers != 3) return fail(RL_EUNSUPPORTED, "policy must have 3 layers, got %d", pol->n_layers);
  const int D = pol->dims[0], H1 = pol->dims[1], H2 = pol->dims[2], NA = pol->dims[3];
  if (D < 1 || D > 2048) return fail(RL_EUNSUPPORTED, "policy input size %d outside 1..2048", D);
  if (H1 < 16 || H1 > 512 || H1 % 16 || H2 < 16 || H2 > 512 || H2 % 16)
    return fail(RL_EUNSUPPORTED, "hidden sizes %d, %d must be multiples of 16 in 16..512", H1, H2);
  if (NA < 1 || NA > rl::MAX_NA) return fail(RL_EUNSUPPORTED, "action count %d outside 1..%d", NA, rl::MAX_NA);
  for (int l = 0; l < 3; ++l)
    if (!pol->W[l] || !pol->b[l]) return fail(RL_EINVAL, "policy weight or bias %d is NULL", l);
  if (pol->packed) {
    if (pol->dtype != RL_BF16) return fail(RL_EUNSUPPORTED, "packed weights are for bf16 policies only");
    if ((uintptr_t)pol->packed % 16) return fail(RL_EINVAL, "packed weights must be 16-byte aligned");
  }
  if (a) {
    a->dt = pol->dtype == RL_F32 ? rl::DT_F32 : rl::DT_BF16;
    a->D = D;
    a->H1 = H1;
    a->H2 = H2;
    a->NA = NA;
    const int dims[4] = {D, H1, H2, NA};
    for (int l = 0; l < 3; ++l) {
      a->W[l] = pol->W[l];
      a->b[l] = pol->b[l];
      a->Wp[l] = pol->packed ? static_cast<const uint8_t*>(pol->packed) + rl::packed_layer_offset(dims, l) : nullptr;
    }
  }
  return RL_OK;
}

}  // namespace

extern "C" {

size_t rl_state_bytes(const rl_env_config* cfg) {
  EnvSpec es;
  if (check_cfg(cfg, &es) != RL_OK) return 0;
  return es.state_bytes;
}

int32_t rl_obs_dim(const rl_env_config* cfg) {
  EnvSpec es;
  const rl_status s = check_cfg(cfg, &es);
  return s != RL_OK ? s : es.D;
}

int32_t rl_num_actions(const rl_env_config* cfg) {
  EnvSpec es;
  const rl_status s = check_cfg(cfg, &es);
  return s != RL_OK ? s : es.NA;
}

const char* rollout_last_error(void) { return g_err; }

rl_status rollout_init(const rl_env_config* cfg, void* state, void* obs, int32_t obs_dtype, uint8_t* legal,
                       void* stream) {
  EnvSpec es;
  rl_status s = check_cfg(cfg, &es);
  if (s != RL_OK) return s;
  if (!state) return fail(RL_EINVAL, "state is NULL");
  if (obs && !valid_dtype(obs_dtype)) return fail(RL_EUNSUPPORTED, "obs dtype %d unsupported", obs_dtype);
  const int dt = obs_dtype == RL_F32 ? rl::DT_F32 : rl::DT_BF16;
  int32_t* st = static_cast<int32_t*>(state);
  const hipStream_t hs = (hipStream_t)stream;
  return launched(es.kind == RL_ENV_LBF          ? rl::launch_lbf_init(es.lbf, st, obs, dt, legal, hs)
                  : es.kind == RL_ENV_OVERCOOKED ? rl::launch_oc_init(es.oc, st, obs, dt, legal, hs)
                                                 : rl::launch_hn_init(es.hn, st, obs, dt, legal, hs),
                  "rollout_init");
}

rl_status rollout_step(const rl_env_config* cfg, void* state, uint64_t t0, int32_t n_steps, const int32_t* actions,
                       void* obs_out, int32_t obs_dtype, float* reward, uint8_t* done, uint8_t* legal_out,
                       void* stream) {
  EnvSpec es;
  rl_status s = check_cfg(cfg, &es);
  if (s != RL_OK) return s;
  if (!state) return fail(RL_EINVAL, "state is NULL");
  if (!actions) return fail(RL_EINVAL, "actions is NULL");
  if (n_steps < 1) return fail(RL_EINVAL, "n_steps %d must be >= 1", n_steps);
  if (t0 > UINT64_MAX - (uint64_t)n_steps) return fail(RL_EINVAL, "t0 + n_steps overflows");
  if (obs_out && !valid_dtype(obs_dtype)) return fail(RL_EUNSUPPORTED, "obs dtype %d unsupported", obs_dtype);
  const int dt = obs_dtype == RL_F32 ? rl::DT_F32 : rl::DT_BF16;
  int32_t* st = static_cast<int32_t*>(state);
  const hipStream_t hs = (hipStream_t)stream;
  hipError_t e;
  if (es.kind == RL_ENV_LBF)
    e = rl::launch_lbf_step(es.lbf, st, t0, n_steps, actions, obs_out, dt, reward, done, legal_out, hs);
  else if (es.kind == RL_ENV_OVERCOOKED)
    e = rl::launch_oc_step(es.oc, st, t0, n_steps, actions, obs_out, dt, reward, done, legal_out, hs);
  else
    e = rl::launch_hn_step(es.hn, st, t0, n_steps, actions, obs_out, dt, reward, done, legal_out, hs);
  return launched(e, "rollout_step");
}

size_t rl_policy_packed_bytes(const rl_policy* policy) {
  rl::PolicyArgs a;
  if (check_policy(policy, &a) != RL_OK || a.dt != rl::DT_BF16) return 0;
  const int dims[4] = {a.D, a.H1, a.H2, a.NA};
  return rl::packed_layer_offset(dims, 2) + rl::packed_layer_bytes(a.NA, a.H2);
}

rl_status rl_policy_pack(const rl_policy* policy, void* packed, void* stream) {
  rl::PolicyArgs a;
  const rl_status s = check_policy(policy, &a);
  if (s != RL_OK) return s;
  if (a.dt != rl::DT_BF16) return fail(RL_EUNSUPPORTED, "packed weights are for bf16 policies only");
  if (!packed) return fail(RL_EINVAL, "packed is NULL");
  if ((uintptr_t)packed % 16) return fail(RL_EINVAL, "packed must be 16-byte aligned");
  return launched(rl::launch_policy_pack(a, packed, (hipStream_t)stream), "rl_policy_pack");
}

rl_status policy_forward(const rl_policy* policy, const void* obs, const uint8_t* legal, int64_t rows,
                         float* logits, void* stream) {
  rl::PolicyArgs a;
  rl_status s = check_policy(policy, &a);
  if (s != RL_OK) return s;
  if (!obs || !logits) return fail(RL_EINVAL, "obs or logits is NULL");
  if (rows < 1 || rows > ((int64_t)1 << 31)) return fail(RL_EINVAL, "rows %lld outside 1..2^31", (long long)rows);
  if (rl::policy_lds_bytes(a) > rl::MAX_LDS_BYTES)
    return fail(RL_EUNSUPPORTED, "policy tiles need more than 160 KiB of LDS");
  return launched(rl::launch_policy_forward(a, obs, legal, rows, logits, (hipStream_t)stream), "policy_forward");
}

rl_status rollout_run(const rl_env_config* cfg, const rl_policy* policy, void* state, uint64_t t0, int32_t n_steps,
                      const rl_traj* out, void* stream) {
  EnvSpec es;
  rl_status s = check_cfg(cfg, &es);
  if (s != RL_OK) return s;
  rl::PolicyArgs a;
  s = check_policy(policy, &a);
  if (s != RL_OK) return s;
  if (!state) return fail(RL_EINVAL, "state is NULL");
  if (!out) return fail(RL_EINVAL, "out is NULL");
  if (n_steps < 1) return fail(RL_EINVAL, "n_steps %d must be >= 1", n_steps);
  if (t0 > UINT64_MAX - (uint64_t)n_steps) return fail(RL_EINVAL, "t0 + n_steps overflows");
  if (a.D != es.D) return fail(RL_ESHAPE, "policy input size %d != observation size %d", a.D, es.D);
  if (a.NA != es.NA) return fail(RL_ESHAPE, "policy has %d actions, the env %d", a.NA, es.NA);
  const size_t lds = es.kind == RL_ENV_LBF          ? rl::make_run_layout(es.A, es.D, a.H1, a.H2, a.dt).total
                     : es.kind == RL_ENV_OVERCOOKED ? rl::oc_run_lds_bytes(a)
                                                    : rl::hn_run_lds_bytes(a);
  if (lds > rl::MAX_LDS_BYTES)
    return fail(RL_EUNSUPPORTED, "rollout tile needs %zu bytes of LDS (max %zu)", lds, rl::MAX_LDS_BYTES);
  const rl::TrajArgs o{out->obs, out->actions, out->logits, out->reward, out->done, out->obs_last};
  int32_t* st = static_cast<int32_t*>(state);
  const hipStream_t hs = (hipStream_t)stream;
  return launched(es.kind == RL_ENV_LBF          ? rl::launch_lbf_run(es.lbf, a, st, t0, n_steps, o, hs)
                  : es.kind == RL_ENV_OVERCOOKED ? rl::launch_oc_run(es.oc, a, st, t0, n_steps, o, hs)
                                                 : rl::launch_hn_run(es.hn, a, st, t0, n_steps, o, hs),
                  "rollout_run");
}

rl_status rollout_run_teams(const rl_env_config* cfg, const rl_policy* policy, const int32_t* teammates, void* state,
                            uint64_t t0, int32_t n_steps, const rl_traj* out, void* stream) {
  EnvSpec es;
  rl_status s = check_cfg(cfg, &es);
  if (s != RL_OK) return s;
  if (es.kind != RL_ENV_LBF) return fail(RL_EUNSUPPORTED, "rollout_run_teams is implemented for LBF only");
  rl::PolicyArgs a;
  s = check_policy(policy, &a);
  if (s != RL_OK) return s;
  if (!teammates) return fail(RL_EINVAL, "teammates is NULL");
  if (!state) return fail(RL_EINVAL, "state is NULL");
  if (!out) return fail(RL_EINVAL, "out is NULL");
  if (n_steps < 1) return fail(RL_EINVAL, "n_steps %d must be >= 1", n_steps);
  if (t0 > UINT64_MAX - (uint64_t)n_steps) return fail(RL_EINVAL, "t0 + n_steps overflows");
  if (a.D != es.D) return fail(RL_ESHAPE, "policy input size %d != observation size %d", a.D, es.D);
  if (a.NA != es.NA) return fail(RL_ESHAPE, "policy has %d actions, the env %d", a.NA, es.NA);
  const size_t lds = rl::make_run_layout(es.A, es.D, a.H1, a.H2, a.dt).total;
  if (lds > rl::MAX_LDS_BYTES)
    return fail(RL_EUNSUPPORTED, "rollout tile needs %zu bytes of LDS (max %zu)", lds, rl::MAX_LDS_BYTES);
  rl::TrajArgs o{out->obs, out->actions, out->logits, out->reward, out->done, out->obs_last};
  o.teammates = teammates;
  return launched(rl::launch_lbf_run(es.lbf, a, static_cast<int32_t*>(state), t0, n_steps, o, (hipStream_t)stream),
                  "rollout_run_teams");
}

rl_status rollout_run_ac(const rl_env_config* cfg, const rl_policy* policy, void* state, uint64_t t0,
                         int32_t n_steps, const rl_traj* out, const rl_ac_traj* ac, void* stream) {
  EnvSpec es;
  rl_status s = check_cfg(cfg, &es);
  if (s != RL_OK) return s;
  if (es.kind != RL_ENV_LBF) return fail(RL_EUNSUPPORTED, "rollout_run_ac is implemented for LBF only");
  rl::PolicyArgs a;
  s = check_policy(policy, &a);
  if (s != RL_OK) return s;
  if (!state) return fail(RL_EINVAL, "state is NULL");
  if (!out || !ac) return fail(RL_EINVAL, "out or ac is NULL");
  if (n_steps < 1) return fail(RL_EINVAL, "n_steps %d must be >= 1", n_steps);
  if (t0 > UINT64_MAX - (uint64_t)n_steps) return fail(RL_EINVAL, "t0 + n_steps overflows");
  if (a.D != es.D) return fail(RL_ESHAPE, "policy input size %d != observation size %d", a.D, es.D);
  if (a.NA != es.NA + 1)
    return fail(RL_ESHAPE, "policy has %d outputs, the env's %d actions plus the value need %d", a.NA, es.NA,
                es.NA + 1);
  a.VH = 1;
  const size_t lds = rl::make_run_layout(es.A, es.D, a.H1, a.H2, a.dt).total;
  if (lds > rl::MAX_LDS_BYTES)
    return fail(RL_EUNSUPPORTED, "rollout tile needs %zu bytes of LDS (max %zu)", lds, rl::MAX_LDS_BYTES);
  rl::TrajArgs o{out->obs, out->actions, out->logits, out->reward, out->done, out->obs_last};
  o.value = ac->value;
  o.logp = ac->logp;
  o.value_last = ac->value_last;
  return launched(rl::launch_lbf_run(es.lbf, a, static_cast<int32_t*>(state), t0, n_steps, o, (hipStream_t)stream),
                  "rollout_run_ac");
}

rl_status rl_s5_discretize(int32_t d_state, int32_t d_model, const float* lambda, const float* log_dt,
                           const float* b, float* lambda_bar, float* b_bar, void* stream) {
  if (!lambda || !log_dt || !b || !lambda_bar || !b_bar) return fail(RL_EINVAL, "a required pointer is NULL");
  if (d_state < 1 || d_model < 1 || (int64_t)d_state * d_model > ((int64_t)1 << 30))
    return fail(RL_EINVAL, "d_state %d, d_model %d out of range", d_state, d_model);
  return launched(rl::launch_s5_discretize(d_state, d_model, lambda, log_dt, b, lambda_bar, b_bar,
                                           (hipStream_t)stream),
                  "rl_s5_discretize");
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

static rl_status check_s5(const rl_env_config* cfg, const rl_s5_policy* pol, EnvSpec* es, rl::S5Net* net) {
  rl_status s = check_cfg(cfg, es);
  if (s != RL_OK) return s;
  if (es->kind != RL_ENV_LBF) return fail(RL_EUNSUPPORTED, "rollout_run_s5 is implemented for LBF only");
  if (!pol) return fail(RL_EINVAL, "policy is NULL");
  if (pol->dtype != RL_BF16) return fail(RL_EUNSUPPORTED, "the S5 policy runs in bfloat16 only");
  const int H = pol->d_model, P = pol->d_state, F = pol->head_width, NA = pol->n_actions;
  if (H < 64 || H > 256 || H % 64) return fail(RL_EUNSUPPORTED, "d_model %d must be a multiple of 64 in 64..256", H);
  if (P < 16 || P > 128 || P % 16) return fail(RL_EUNSUPPORTED, "d_state %d must be a multiple of 16 in 16..128", P);
  if (F < 128 || F > 4096 || F % 128)
    return fail(RL_EUNSUPPORTED, "head_width %d must be a multiple of 128 in 128..4096", F);
  if (pol->obs_dim != es->D) return fail(RL_ESHAPE, "policy obs_dim %d != observation size %d", pol->obs_dim, es->D);
  if (es->D > 1024) return fail(RL_EUNSUPPORTED, "observation size %d above 1024", es->D);
  if (NA != es->NA) return fail(RL_ESHAPE, "policy has %d actions, the env %d", NA, es->NA);
  const void* ptrs[] = {pol->w_enc, pol->b_enc, pol->lambda_bar, pol->b_bar, pol->c, pol->d};
  for (const void* q : ptrs)
    if (!q || !aligned16(q)) return fail(RL_EINVAL, "an S5 parameter pointer is NULL or not 16-byte aligned");
  for (int l = 0; l < 4; ++l)
    if (!pol->actor_w[l] || !pol->actor_b[l] || !pol->critic_w[l] || !pol->critic_b[l] ||
        !aligned16(pol->actor_w[l]) || !aligned16(pol->actor_b[l]) || !aligned16(pol->critic_w[l]) ||
        !aligned16(pol->critic_b[l]))
      return fail(RL_EINVAL, "head layer %d pointer is NULL or not 16-byte aligned", l);
  if (rl::s5_front_lds_bytes(es->D, H, P) > rl::MAX_LDS_BYTES)
    return fail(RL_EUNSUPPORTED, "S5 tile needs more than %zu bytes of LDS", rl::MAX_LDS_BYTES);
  net->D = es->D;
  net->H = H;
  net->P = P;
  net->F = F;
  net->NA = NA;
  net->w_enc = pol->w_enc;
  net->b_enc = pol->b_enc;
  net->lbar = pol->lambda_bar;
  net->bbar = pol->b_bar;
  net->c = pol->c;
  net->d = pol->d;
  for (int l = 0; l < 4; ++l) {
    net->actor_w[l] = pol->actor_w[l];
    net->actor_b[l] = pol->actor_b[l];
    net->critic_w[l] = pol->critic_w[l];
    net->critic_b[l] = pol->critic_b[l];
  }
  return RL_OK;
}

size_t rl_s5_workspace_bytes(const rl_env_config* cfg, const rl_s5_policy* policy) {
  EnvSpec es;
  rl::S5Net net;
  if (check_s5(cfg, policy, &es, &net) != RL_OK) return 0;
  return rl::s5_workspace(es.lbf, net).bytes;
}

rl_status rollout_run_s5(const rl_env_config* cfg, const rl_s5_policy* policy, void* state, float* carry,
                         uint64_t t0, int32_t n_steps, const rl_traj* out, const rl_ac_traj* ac, void* workspace,
                         size_t workspace_bytes, void* stream) {
  EnvSpec es;
  rl::S5Net net;
  rl_status s = check_s5(cfg, policy, &es, &net);
  if (s != RL_OK) return s;
  if (!state || !carry) return fail(RL_EINVAL, "state or carry is NULL");
  if (!out || !ac) return fail(RL_EINVAL, "out or ac is NULL");
  if (n_steps < 1) return fail(RL_EINVAL, "n_steps %d must be >= 1", n_steps);
  if (t0 > UINT64_MAX - (uint64_t)n_steps) return fail(RL_EINVAL, "t0 + n_steps overflows");
  if ((int64_t)es.E * es.A > ((int64_t)1 << 24)) return fail(RL_EINVAL, "n_envs * n_agents above 2^24");
  const size_t need = rl::s5_workspace(es.lbf, net).bytes;
  if (!workspace || !aligned16(workspace) || workspace_bytes < need)
    return fail(RL_EINVAL, "workspace needs %zu bytes, 16-byte aligned (got %zu)", need, workspace_bytes);
  if ((out->obs && !aligned16(out->obs)) || (out->obs_last && !aligned16(out->obs_last)))
    return fail(RL_EINVAL, "obs and obs_last must be 16-byte aligned");
  rl::TrajArgs o{out->obs, out->actions, out->logits, out->reward, out->done, out->obs_last};
  o.value = ac->value;
  o.logp = ac->logp;
  o.value_last = ac->value_last;
  return launched(rl::launch_s5_rollout(es.lbf, net, static_cast<int32_t*>(state), carry, t0, n_steps, o, workspace,
                                        (hipStream_t)stream),
                  "rollout_run_s5");
}

rl_status rollout_run_s5_noalloc(const rl_env_config* cfg, const rl_s5_policy* policy, void* state, float* carry,
                                 uint64_t t0, int32_t n_steps, const rl_traj* out, const rl_ac_traj* ac,
                                 void* stream) {
  EnvSpec es;
  rl::S5Net net;
  rl_status s = check_s5(cfg, policy, &es, &net);
  if (s != RL_OK) return s;
  if (!state || !carry) return fail(RL_EINVAL, "state or carry is NULL");
  if (!out || !ac) return fail(RL_EINVAL, "out or ac is NULL");
  if (n_steps < 1) return fail(RL_EINVAL, "n_steps %d must be >= 1", n_steps);
  if (t0 > UINT64_MAX - (uint64_t)n_steps) return fail(RL_EINVAL, "t0 + n_steps overflows");
  if ((int64_t)es.E * es.A > ((int64_t)1 << 24)) return fail(RL_EINVAL, "n_envs * n_agents above 2^24");
  const size_t need = rl::s5_workspace(es.lbf, net).bytes;
  if (need > rl::S5_SCRATCH_BYTES)
    return fail(RL_EINVAL, "this rollout needs %zu bytes of workspace; the built-in scratch holds %zu "
                "(use rollout_run_s5 with a caller-owned workspace)", need, rl::S5_SCRATCH_BYTES);
  if ((out->obs && !aligned16(out->obs)) || (out->obs_last && !aligned16(out->obs_last)))
    return fail(RL_EINVAL, "obs and obs_last must be 16-byte aligned");
  void* scratch = nullptr;
  const hipError_t e = rl::s5_scratch_ptr(&scratch);
  if (e != hipSuccess) return fail(RL_EDEVICE, "resolving the S5 scratch array failed: %s", hipGetErrorString(e));
  rl::TrajArgs o{out->obs, out->actions, out->logits, out->reward, out->done, out->obs_last};
  o.value = ac->value;
  o.logp = ac->logp;
  o.value_last = ac->value_last;
  return launched(rl::launch_s5_rollout(es.lbf, net, static_cast<int32_t*>(state), carry, t0, n_steps, o, scratch,
                                        (hipStream_t)stream),
                  "rollout_run_s5_noalloc");
}

rl_status rl_gae(const float* reward, const uint8_t* done, const float* value, const float* value_last,
                 int32_t n_steps, int32_t n_envs, int32_t n_agents, float gamma, float lambda, float* adv,
                 float* ret, void* stream) {
  if (!reward || !done || !value || !value_last || !adv) return fail(RL_EINVAL, "a required pointer is NULL");
  if (n_steps < 1 || n_envs < 1 || n_agents < 1) return fail(RL_EINVAL, "sizes must be >= 1");
  if ((int64_t)n_envs * n_agents > ((int64_t)1 << 31)) return fail(RL_EINVAL, "n_envs * n_agents exceeds 2^31");
  if (!(gamma >= 0.f && gamma <= 1.f) || !(lambda >= 0.f && lambda <= 1.f))
    return fail(RL_EINVAL, "gamma and lambda must lie in [0, 1]");
  return launched(rl::launch_gae(reward, done, value, value_last, n_steps, n_envs, n_agents, gamma, lambda, adv,
                                 ret, (hipStream_t)stream),
                  "rl_gae");
}

rl_status rollout_run_pop(const rl_env_config* cfg, const rl_policy* pop, int32_t n_policies,
                          const int32_t* policy_index, void* state, uint64_t t0, int32_t n_steps, const rl_traj* out,
                          void* stream) {
  EnvSpec es;
  rl_status s = check_cfg(cfg, &es);
  if (s != RL_OK) return s;
  if (es.kind != RL_ENV_LBF) return fail(RL_EUNSUPPORTED, "rollout_run_pop is implemented for LBF only");
  rl::PolicyArgs a;
  s = check_policy(pop, &a);
  if (s != RL_OK) return s;
  if (n_policies < 1 || n_policies > 4096) return fail(RL_EINVAL, "n_policies %d outside 1..4096", n_policies);
  if (!policy_index) return fail(RL_EINVAL, "policy_index is NULL");
  if (!state) return fail(RL_EINVAL, "state is NULL");
  if (!out) return fail(RL_EINVAL, "out is NULL");
  if (n_steps < 1) return fail(RL_EINVAL, "n_steps %d must be >= 1", n_steps);
  if (t0 > UINT64_MAX - (uint64_t)n_steps) return fail(RL_EINVAL, "t0 + n_steps overflows");
  if (a.D != es.D) return fail(RL_ESHAPE, "policy input size %d != observation size %d", a.D, es.D);
  if (a.NA != es.NA) return fail(RL_ESHAPE, "policy has %d actions, the env %d", a.NA, es.NA);
  const size_t lds = rl::lbf_pop_lds_bytes(es.lbf, a);
  if (lds + rl::LBF_POP_STATIC_LDS > rl::MAX_LDS_BYTES)
    return fail(RL_EUNSUPPORTED, "rollout tile needs %zu bytes of LDS (max %zu)", lds,
                rl::MAX_LDS_BYTES - rl::LBF_POP_STATIC_LDS);
  const rl::TrajArgs o{out->obs, out->actions, out->logits, out->reward, out->done, out->obs_last};
  return launched(rl::launch_lbf_run_pop(es.lbf, a, n_policies, policy_index, static_cast<int32_t*>(state), t0,
                                         n_steps, o, (hipStream_t)stream),
                  "rollout_run_pop");
}

rl_status rollout_sample(const rl_env_config* cfg, uint64_t t, const float* logits, const uint8_t* legal,
                         int32_t* actions, void* stream) {
  EnvSpec es;
  rl_status s = check_cfg(cfg, &es);
  if (s != RL_OK) return s;
  if (!logits || !actions) return fail(RL_EINVAL, "logits or actions is NULL");
  return launched(rl::launch_sample(cfg->seed, cfg->env_base, es.E, es.A, es.NA, t, logits, legal, actions,
                                    (hipStream_t)stream),
                  "rollout_sample");
}

rl_status rl_gumbel_noise(const uint32_t* u, int64_t n, float* g, void* stream) {
  if (!u || !g) return fail(RL_EINVAL, "u or g is NULL");
  if (n < 1 || n > ((int64_t)1 << 32)) return fail(RL_EINVAL, "n %lld outside 1..2^32", (long long)n);
  return launched(rl::launch_gumbel(u, n, g, (hipStream_t)stream), "rl_gumbel_noise");
}

}  // extern "C"
