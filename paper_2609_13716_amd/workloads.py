"""Seeded synthetic workloads and input generators.

This module holds the sizes of the benchmark workloads and draws the inputs
that both the GPU path and the CPU oracle consume: policy weights (normal,
variance 1 / fan_in, float32) and injected actions (uniform integers).  It
contains none of the rollout's arithmetic.

Workloads (Level-Based Foraging; env dynamics and observation as documented
in include/rollout.h):
    lbf8_small   8x8, 2 agents, 3 foods, levels 1..2 / 1..3, 16 envs x 128 steps,
                 MLP 192-64-64-6 float32 (a correctness-size workload)
    lbf8_4096    8x8, 2 agents, 3 foods, levels 1..2 / 1..3, 4096 envs x 128 steps,
                 MLP 192-128-128-6 in float32 and in bf16
    lbf12_16k    12x12, 3 agents, 6 foods, levels 1..3 / 1..6, 16384 envs x 256 steps,
                 MLP 432-256-256-6 bf16
All LBF episodes are truncated after 50 steps.

Overcooked-style kitchen (two agents; seeded random kitchens of 5x4 to 9x5,
rules and observation as documented in include/rollout.h):
    oc_4096      4096 envs x 400 steps, cook time 20, soup reward 20, episodes of
                 400 steps, MLP 1170-256-256-6 bf16

Two-player Hanabi (5 colours x 5 ranks, hands of 5, 8 info tokens, 3 lives):
    hn_4096      4096 envs x 80 steps, MLP 658-512-512-20 bf16 on the mover's
                 observation, illegal actions masked

Actor-critic rollout (what a PPO-style learner consumes after a rollout):
    lbf8_4096_ac lbf8_4096's envs, an MLP 192-128-128-7 bf16 whose last output
                 is the value head; the rollout writes values and log pi(a), then
                 generalised advantage estimation (gamma 0.99, lambda 0.95) runs
                 over the stored trajectory

Population rollout (ad hoc teamwork evaluation: one ego policy paired with a
set of teammate policies, all of one shape):
    lbf8_4096_pop  lbf8_4096's envs, a population of 9 MLPs 192-128-128-6 bf16:
                 agent 0 of every env is the ego (policy 0), agent 1 of env e
                 is teammate 1 + e // 512 (8 blocks of 512 envs, one teammate each)
"""

import numpy as np

WORKLOADS = {
    "lbf8_small": dict(env=dict(grid_h=8, grid_w=8, n_agents=2, n_food=3, max_agent_level=2, max_food_level=3,
                                max_steps=50),
                       n_envs=16, n_steps=128, hidden=(64, 64), dtypes=("f32",)),
    "lbf8_4096": dict(env=dict(grid_h=8, grid_w=8, n_agents=2, n_food=3, max_agent_level=2, max_food_level=3,
                               max_steps=50),
                      n_envs=4096, n_steps=128, hidden=(128, 128), dtypes=("f32", "bf16")),
    "lbf12_16k": dict(env=dict(grid_h=12, grid_w=12, n_agents=3, n_food=6, max_agent_level=3, max_food_level=6,
                               max_steps=50),
                      n_envs=16384, n_steps=256, hidden=(256, 256), dtypes=("bf16",)),
    # the constant-levels variant on a 7x7 grid: agents at level 1, foods at
    # level 2, so every food takes both agents loading together
    "lbf7_const_4096": dict(env=dict(grid_h=7, grid_w=7, n_agents=2, n_food=3, max_agent_level=1, max_food_level=2,
                                     max_steps=50, const_levels=True),
                            n_envs=4096, n_steps=128, hidden=(128, 128), dtypes=("bf16",)),
    # the paper's ego agent: S5 actor-critic (model 128, state 128, heads of
    # three 1024-unit layers) on LBF 8x8
    "lbf8_4096_s5": dict(env=dict(grid_h=8, grid_w=8, n_agents=2, n_food=3, max_agent_level=2, max_food_level=3,
                                  max_steps=50),
                         n_envs=4096, n_steps=128, s5=dict(d_model=128, d_state=128, head_width=1024),
                         dtypes=("bf16",)),
    # ego policy (agent 0) with heuristic teammates (agent 1: Greedy / Sequential kind e mod 11)
    "lbf7_teams_4096": dict(env=dict(grid_h=7, grid_w=7, n_agents=2, n_food=3, max_agent_level=1, max_food_level=2,
                                     max_steps=50, const_levels=True),
                            n_envs=4096, n_steps=128, hidden=(128, 128), dtypes=("bf16",), teammates=True),
    "oc_4096": dict(kind="overcooked", env=dict(cook_time=20, soup_reward=20, max_steps=400),
                    n_envs=4096, n_steps=400, hidden=(256, 256), dtypes=("bf16",)),
    "hn_4096": dict(kind="hanabi", env=dict(max_steps=1000), n_envs=4096, n_steps=80, hidden=(512, 512),
                    dtypes=("bf16",)),
    "hn_mini_4096": dict(kind="hanabi", env=dict(max_steps=1000, colours=3, ranks=3), n_envs=4096, n_steps=80,
                         hidden=(256, 256), dtypes=("bf16",)),
    "lbf8_4096_ac": dict(env=dict(grid_h=8, grid_w=8, n_agents=2, n_food=3, max_agent_level=2, max_food_level=3,
                                  max_steps=50),
                         n_envs=4096, n_steps=128, hidden=(128, 128), dtypes=("bf16",), value_head=True,
                         gamma=0.99, lam=0.95),
    "lbf8_4096_pop": dict(env=dict(grid_h=8, grid_w=8, n_agents=2, n_food=3, max_agent_level=2, max_food_level=3,
                                   max_steps=50),
                          n_envs=4096, n_steps=128, hidden=(128, 128), dtypes=("bf16",), population=9),
}

LBF_ACTIONS = 6
OC_ACTIONS = 6
OC_OBS_DIM = 26 * 45
HN_ACTIONS = 20
HN_OBS_DIM = 658


def lbf_obs_dim(env):
    return 3 * env["grid_h"] * env["grid_w"]


def kind(name):
    return WORKLOADS[name].get("kind", "lbf")


def policy_dims(name):
    """(D, H1, H2, outputs): the outputs include the value when the workload has a value head."""
    w = WORKLOADS[name]
    if w.get("value_head"):
        return (lbf_obs_dim(w["env"]), *w["hidden"], LBF_ACTIONS + 1)
    if kind(name) == "overcooked":
        return (OC_OBS_DIM, *w["hidden"], OC_ACTIONS)
    if kind(name) == "hanabi":
        if w["env"].get("colours") == 3:  # the mini game: 278 features, 16 actions
            return (278, *w["hidden"], 16)
        return (HN_OBS_DIM, *w["hidden"], HN_ACTIONS)
    return (lbf_obs_dim(w["env"]), *w["hidden"], LBF_ACTIONS)


def policy_weights(dims, seed, bias_scale=0.0):
    """float32 weights W_l ~ N(0, 1/fan_in) in the [fan_out, fan_in] layout, and biases.

    Biases are zero unless ``bias_scale`` > 0 (then N(0, bias_scale^2)).
    """
    rng = np.random.default_rng(seed)
    ws, bs = [], []
    for i in range(len(dims) - 1):
        ws.append((rng.standard_normal((dims[i + 1], dims[i])) / np.sqrt(dims[i])).astype(np.float32))
        bs.append((rng.standard_normal(dims[i + 1]) * bias_scale).astype(np.float32))
    return ws, bs


def s5_params(D, H, P, F, n_actions, seed):
    """Synthetic continuous-time parameters of an S5 actor-critic (float32 arrays).

    Encoder [H, D]; S5 with Re(lambda) = -0.5 and Im(lambda_p) = pi * p (the
    shape of the diagonalised HiPPO-N start of S5), log step uniform in
    [log 1e-3, log 1e-1], B and C complex normal (variance 1/H and 1/P split
    over real and imaginary parts), D standard normal; actor and critic heads
    H -> F -> F -> F -> (n_actions | 1) with N(0, 1/fan_in) weights."""
    rng = np.random.default_rng(seed)
    we, be = policy_weights((D, H), seed + 1, bias_scale=0.1)
    aw, ab = policy_weights((H, F, F, F, n_actions), seed + 2, bias_scale=0.1)
    cw, cb = policy_weights((H, F, F, F, 1), seed + 3, bias_scale=0.1)
    f32 = np.float32
    return dict(
        w_enc=we[0], b_enc=be[0],
        lam_re=np.full(P, -0.5, f32), lam_im=(np.pi * np.arange(P)).astype(f32),
        log_dt=rng.uniform(np.log(1e-3), np.log(1e-1), P).astype(f32),
        b_re=(rng.standard_normal((P, H)) / np.sqrt(2 * H)).astype(f32),
        b_im=(rng.standard_normal((P, H)) / np.sqrt(2 * H)).astype(f32),
        c_re=(rng.standard_normal((H, P)) / np.sqrt(2 * P)).astype(f32),
        c_im=(rng.standard_normal((H, P)) / np.sqrt(2 * P)).astype(f32),
        d=rng.standard_normal(H).astype(f32),
        actor_w=aw, actor_b=ab, critic_w=cw, critic_b=cb)


def injected_actions(n_steps, n_envs, n_agents, n_actions, seed, p_invalid=0.0):
    """Uniform actions [T, E, A] int32; a fraction ``p_invalid`` is replaced by out-of-range values."""
    rng = np.random.default_rng(seed)
    a = rng.integers(0, n_actions, size=(n_steps, n_envs, n_agents), dtype=np.int64)
    if p_invalid > 0:
        bad = rng.random(a.shape) < p_invalid
        a[bad] = rng.choice(np.array([-1, n_actions, n_actions + 7, 1 << 20]), size=int(bad.sum()))
    return a.astype(np.int32)


def population_index(name):
    """[E, A] int32 policy of every agent of a population workload: agent 0 the ego (policy 0), the other
    agents of env e the teammate 1 + e // (E / (P - 1))."""
    w = WORKLOADS[name]
    E, A, P = w["n_envs"], w["env"]["n_agents"], w["population"]
    block = max(1, E // (P - 1))
    idx = np.zeros((E, A), dtype=np.int32)
    for a in range(1, A):
        idx[:, a] = 1 + np.minimum(np.arange(E) // block, P - 2)
    return idx


def population_weights(name, seed):
    """Per-policy (weights, biases) of a population workload, policy p drawn with seed + p."""
    dims = policy_dims(name)
    ws, bs = [], []
    for p in range(WORKLOADS[name]["population"]):
        w, b = policy_weights(dims, seed + p)
        ws.append(w)
        bs.append(b)
    return ws, bs

