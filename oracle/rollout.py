"""The rollout loop: observe, act, step, auto-reset (test infrastructure).

One rollout step for each env is the Dec-POMDP step of the paper's problem
setting (Section 3): every agent i observes o_i, samples a_i from its policy
pi_i(. | o_i), the joint action moves the state through P and yields the
shared reward r; an env whose episode ended starts a fresh one drawn from rho
(auto-reset, with the reset drawn at step t + 1).  Envs are independent, and
step t of env e consumes only draws keyed by (e, t), so any subset of env ids
can be rolled out on its own and matches the same envs in a full batch.

Output layout (``n`` = number of env ids, A agents, D obs features):
    obs      [T, n, A, D] float64  observation the step's action was taken on
    logits   [T, n, A, nA] float64 the oracle's policy logits for that obs
    actions  [T, n, A]    int64
    reward   [T, n]       float32
    done     [T, n]       uint8   bit 0 terminated, bit 1 truncated
    obs_last [n, A, D]    float64 observation after the last step
    states   list of the n env states after the last step
"""

import numpy as np

from . import actor_critic, lbf_heuristics, mlp, s5, sampling


def initial_states(env, cfg, seed, env_ids):
    """States at t = 0 (the first episode of every env is drawn at step 0)."""
    return [env.reset(cfg, seed, e, 0) for e in env_ids]


def observe_all(env, cfg, states):
    """[n, A, D] float64 observations and [n, A, nA] bool legal masks."""
    A = cfg.n_agents
    obs = np.stack([np.stack([env.observe(cfg, s, a) for a in range(A)]) for s in states])
    mask = np.array([[env.legal_mask(cfg, s, a) for a in range(A)] for s in states], dtype=bool)
    return obs, mask


def policy_logits(obs, weights, biases, dtype, policy_index=None):
    """Logits [n, A, nA] float64 of observations [n, A, D].

    Without ``policy_index`` every agent uses the one network (weights,
    biases).  With it, ``weights[p]`` and ``biases[p]`` are the layers of
    policy p of a population and agent a of env index i acts with policy
    ``policy_index[i][a]``: the ego agent and its teammates of the ad hoc
    teamwork objective (Section 3, the J_AHT equation) each run their own
    network.  An index outside the population selects policy 0 (reading).
    """
    n, A, D = obs.shape
    flat = obs.reshape(n * A, D)
    if policy_index is None:
        return mlp.forward(flat, weights, biases, dtype).reshape(n, A, -1)
    ids = np.asarray(policy_index, dtype=np.int64).reshape(n * A)
    ids = np.where((ids >= 0) & (ids < len(weights)), ids, 0)
    out = None
    for p in np.unique(ids):
        sel = ids == p
        lg = mlp.forward(flat[sel], weights[p], biases[p], dtype)
        if out is None:
            out = np.zeros((n * A, lg.shape[1]), dtype=np.float64)
        out[sel] = lg
    return out.reshape(n, A, -1)


def rollout(env, cfg, seed, env_ids, t0, n_steps, weights, biases, dtype,
            states=None, logits_source=None, action_hook=None, policy_index=None, value_head=False,
            recurrent=None, carry=None, teammates=None, start_cells=None):
    """Roll ``env_ids`` forward ``n_steps`` steps from absolute step ``t0``.

    ``states`` are the env states at t0 (default: the initial states, t0 = 0).
    ``logits_source(k, logits64)`` may return float32 logits [n, A, nA] to
    sample from at step t0 + k instead of the oracle's own.
    ``action_hook(k, i, agent, action, logits32, mask)`` may replace the
    sampled action of env index i, agent ``agent``.
    ``policy_index`` [n, A]: per-agent policies of a population (see
    ``policy_logits``); ``weights`` and ``biases`` are then per policy.
    ``value_head``: the network has nA + 1 outputs, the last being the
    critic's value V(o); the result then also holds ``value`` [T, n, A],
    ``value_last`` [n, A] (V of obs_last), ``logits_last`` [n, A, nA] (the
    logits of obs_last, for scaling value_last's tolerance like the values of
    the steps) and ``logp`` [T, n, A], the float64
    log-probability of each sampled action under the float32 logits it was
    sampled from (``logits`` keeps the nA action logits).
    ``recurrent``: an ``s5.Params`` actor-critic that replaces (weights,
    biases) and implies ``value_head``; ``carry`` [n * A, P] complex is its
    state at t0 (rows env-major, default zeros).  An agent's state is zeroed
    at every step whose observation starts an episode (step counter 0); the
    result also holds ``carry``, the state after the last step (value_last is
    computed without advancing it).
    ``teammates`` [n, A] (LBF): k in 0..len(KINDS)-1 = heuristic k of
    ``lbf_heuristics`` (its logits replace the network's); any other value =
    the network.  The start cells of the episodes (which the Sequential
    nearest/farthest-agent teammates plan from) are tracked along the rollout:
    the agents' cells in the first state of each episode.  ``start_cells``
    [n][A] gives them for the episodes running at t0; by default they are the
    cells of the given states when t0 = 0 (initial states), else the cells of
    the reset of step t0 - step_count (where those episodes began).
    """
    env_ids = list(env_ids)
    if states is None:
        if t0 != 0:
            raise ValueError("states are required when t0 != 0")
        states = initial_states(env, cfg, seed, env_ids)
    states = [s.copy() for s in states]
    n, A = len(env_ids), cfg.n_agents
    nA = env.N_ACTIONS
    out = {k: [] for k in ("obs", "logits", "actions", "reward", "done", "mask", "value", "logp")}
    if recurrent is not None:
        value_head = True
        carry = s5.initial_state(n * A, recurrent) if carry is None else np.array(carry, dtype=np.complex128)

    def net(obs, states, commit):
        nonlocal carry
        if recurrent is None:
            return policy_logits(obs, weights, biases, dtype, policy_index)
        start = np.repeat([s.step_count == 0 for s in states], A)
        lg, v, x = s5.step(recurrent, obs.reshape(n * A, -1), carry, start, dtype)
        if commit:
            carry = x
        return np.concatenate([lg, v[:, None]], axis=1).reshape(n, A, -1)

    if teammates is not None:
        if start_cells is not None:
            starts = [list(c) for c in start_cells]
        elif t0 == 0:
            starts = [list(s.agent_cell) for s in states]
        else:
            starts = [list(env.reset(cfg, seed, e, t0 - s.step_count).agent_cell) for e, s in zip(env_ids, states)]
    for k in range(n_steps):
        t = t0 + k
        obs, mask = observe_all(env, cfg, states)
        logits64 = net(obs, states, True)
        if teammates is not None:
            for i in range(n):
                for a in range(A):
                    if 0 <= teammates[i][a] < len(lbf_heuristics.KINDS):
                        logits64[i, a, :nA] = lbf_heuristics.logits(cfg, states[i], a, int(teammates[i][a]),
                                                                    starts[i][a])
        if value_head:
            out["value"].append(logits64[..., nA])
            logits64 = logits64[..., :nA]
        logits32 = logits64.astype(np.float32)
        if logits_source is not None:
            logits32 = np.asarray(logits_source(k, logits64), dtype=np.float32)
        actions = np.zeros((n, A), dtype=np.int64)
        for i, e in enumerate(env_ids):
            for a in range(A):
                act = sampling.sample_action(seed, e, t, a, list(logits32[i, a]), list(mask[i, a]))
                if action_hook is not None:
                    act = action_hook(k, i, a, act, logits32[i, a], mask[i, a])
                actions[i, a] = act
        if value_head:
            out["logp"].append(np.array([[actor_critic.log_prob(logits32[i, a], actions[i, a], mask[i, a])
                                          for a in range(A)] for i in range(n)]))
        rewards = np.zeros(n, dtype=np.float32)
        dones = np.zeros(n, dtype=np.uint8)
        for i, e in enumerate(env_ids):
            states[i], rewards[i], dones[i] = env.step(cfg, seed, e, t, states[i], list(actions[i]))
            if teammates is not None and dones[i]:  # a new episode starts from the reset's cells
                starts[i] = list(states[i].agent_cell)
        out["obs"].append(obs)
        out["mask"].append(mask)
        out["logits"].append(logits64)
        out["actions"].append(actions)
        out["reward"].append(rewards)
        out["done"].append(dones)
    res = {k: np.stack(v) if v else None for k, v in out.items()}
    res["obs_last"], res["mask_last"] = observe_all(env, cfg, states)
    if value_head:
        last = net(res["obs_last"], states, False)
        res["value_last"] = last[..., nA]
        res["logits_last"] = last[..., :nA]
    res["states"] = states
    if recurrent is not None:
        res["carry"] = carry
    return res


def env_only(env, cfg, seed, env_ids, t0, actions, states=None):
    """Step ``env_ids`` with injected actions [T, n, A] from absolute step ``t0``.

    Returns per-step post-transition observations obs_{t+1} [T, n, A, D]
    (after any auto-reset), masks, rewards, dones and the final states.
    """
    env_ids = list(env_ids)
    if states is None:
        if t0 != 0:
            raise ValueError("states are required when t0 != 0")
        states = initial_states(env, cfg, seed, env_ids)
    states = [s.copy() for s in states]
    actions = np.asarray(actions)
    T, n = actions.shape[0], len(env_ids)
    obs_out, mask_out = [], []
    rewards = np.zeros((T, n), dtype=np.float32)
    dones = np.zeros((T, n), dtype=np.uint8)
    for k in range(T):
        for i, e in enumerate(env_ids):
            states[i], rewards[k, i], dones[k, i] = env.step(
                cfg, seed, e, t0 + k, states[i], list(actions[k, i]))
        o, m = observe_all(env, cfg, states)
        obs_out.append(o)
        mask_out.append(m)
    return {"obs": np.stack(obs_out), "mask": np.stack(mask_out), "reward": rewards,
            "done": dones, "states": states}
