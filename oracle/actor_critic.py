"""Actor-critic outputs of a rollout: log pi(a | o) of the sampled actions and
generalised advantage estimates (test infrastructure).

The learners the paper benchmarks are built on PPO (appendix, Algorithms
Overview); what every one of them consumes right after a rollout is, per agent
and step, the log-probability of the action taken, the critic's value of the
observation, and advantages / returns computed from the stored trajectory.
The paper gives neither the advantage estimator nor its constants; the
reading here is generalised advantage estimation with caller-given gamma (the
Dec-POMDP discount of Section 3) and lambda, the team reward shared by all
agents, and every episode end (terminated or truncated) cutting the
recurrence: the observation after it belongs to the next episode (auto-reset),
so nothing is bootstrapped across it.
"""

import math

import numpy as np


def log_prob(logits, action, mask=None):
    """log pi(action) of a softmax over the legal entries of ``logits``, in float64.

    Illegal actions (mask False) have probability 0; ``action`` must be legal.
    """
    x = np.asarray(logits, dtype=np.float64)
    legal = np.ones(x.shape, dtype=bool) if mask is None else np.asarray(mask, dtype=bool)
    m = max(x[i] for i in range(len(x)) if legal[i])
    s = sum(math.exp(x[i] - m) for i in range(len(x)) if legal[i])
    return float(x[action] - (m + math.log(s)))


def gae(reward, done, value, value_last, gamma, lam):
    """Advantages and returns [T, n, A] (float64) by a backward scan over the steps.

    reward [T, n] (shared team reward of the transition at t), done [T, n]
    (nonzero: the episode ended at that transition), value [T, n, A] = V(o_t),
    value_last [n, A] = V(o_T) after the last step.
        delta_t = r_t + gamma * (1 - d_t) * V_{t+1} - V_t
        A_t     = delta_t + gamma * lam * (1 - d_t) * A_{t+1},   A_T = 0
        R_t     = A_t + V_t
    """
    reward = np.asarray(reward, dtype=np.float64)
    done = np.asarray(done)
    value = np.asarray(value, dtype=np.float64)
    T = reward.shape[0]
    adv = np.zeros(value.shape, dtype=np.float64)
    nxt_adv = np.zeros(value.shape[1:], dtype=np.float64)
    nxt_v = np.asarray(value_last, dtype=np.float64)
    for t in range(T - 1, -1, -1):
        keep = (done[t] == 0).astype(np.float64)[:, None]
        delta = reward[t][:, None] + gamma * keep * nxt_v - value[t]
        nxt_adv = delta + gamma * lam * keep * nxt_adv
        adv[t] = nxt_adv
        nxt_v = value[t]
    return adv, adv + value
