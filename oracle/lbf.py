"""Level-Based Foraging (LBF) environment, plain CPU reference (test infrastructure).

The paper runs LBF (Section 4, environment table: the Jumanji version, variants
7x7 with constant levels and 12x12) as a cooperative Dec-POMDP (Section 3):
agents with levels walk a grid and jointly load food whose level does not
exceed the summed level of the agents loading it; the team shares one reward.
Games last at most 50 steps (the human-data appendix).  The rules the paper
does not restate are fixed by the following readings.

Grid and actions
    H x W cells, rows top-down, cols left-right; cell id = row * W + col.
    Actions 0 noop, 1 north (row - 1), 2 south (row + 1), 3 west (col - 1),
    4 east (col + 1), 5 load.  An action outside 0..5 is treated as noop.

Reset (initial-state distribution rho), drawn from the reset stream
(seed; env, t, *, TAG_RESET) in this order:
    1. agent levels  l_i = 1 + uniform_int(d, Lmax)                 (A draws)
    2. food levels   f_j = 1 + uniform_int(d, min(Fmax, sum_i l_i))  (F draws)
       -- this is exactly "f_j uniform on 1..Fmax conditioned on
       max_j f_j <= sum_i l_i", since that condition factorises over j.
    3. food cells: the uniform_int(d, n)-th of the n interior cells (rows
       1..H-2, cols 1..W-2) not yet holding food, in row-major order (F draws)
    4. agent cells: the uniform_int(d, n)-th of the n cells holding neither
       food nor an earlier agent, in row-major order               (A draws)
    5. den = sum_j f_j, step count 0.

Step (transition P and shared reward r), evaluated in this order:
    1. Moves.  A move is legal iff its target cell is on the grid, holds no
       uneaten food and holds no agent in the pre-step state.  Legal movers
       that share a target all stay.  Everyone else stays.
    2. Loads.  Food j (uneaten) is eaten iff the agents that chose load and
       are 4-adjacent to it exist and their levels sum to >= f_j.  A loader
       counts towards every food adjacent to it.  Food eaten this step still
       blocked moves this step (moves are resolved first, against the pre-step
       food).
    3. Reward r = float32(sum of eaten levels) / float32(den), one IEEE
       float32 division, shared by the team.
    4. step count += 1.  done bit 0 (terminated) = every food eaten; done bit 1
       (truncated) = step count reached max_steps.

Observation of agent i: 3 planes of H x W, plane-major:
    plane 0 holds l_k at agent k's cell (every agent, i included),
    plane 1 holds f_j at each uneaten food's cell,
    plane 2 holds 1 at agent i's own cell.
"""

from dataclasses import dataclass

import numpy as np

from . import philox

NOOP, NORTH, SOUTH, WEST, EAST, LOAD = range(6)
N_ACTIONS = 6
_DELTA = {NORTH: (-1, 0), SOUTH: (1, 0), WEST: (0, -1), EAST: (0, 1)}


@dataclass(frozen=True)
class Config:
    grid_h: int
    grid_w: int
    n_agents: int
    n_food: int
    max_agent_level: int
    max_food_level: int
    max_steps: int = 50
    # the constant-levels variant of the paper's LBF task table: every agent at
    # max_agent_level, every food at max_food_level.  Reading: the reset still
    # takes its level draws (and ignores them), so cells match the game with
    # drawn levels under the same seed.
    const_levels: bool = False

    @property
    def obs_dim(self):
        return 3 * self.grid_h * self.grid_w


@dataclass
class State:
    agent_cell: list   # [A] cell ids
    agent_level: list  # [A]
    food_cell: list    # [F] cell ids
    food_level: list   # [F]
    food_eaten: list   # [F] bools
    step_count: int
    den: int

    def copy(self):
        return State(list(self.agent_cell), list(self.agent_level), list(self.food_cell),
                     list(self.food_level), list(self.food_eaten), self.step_count, self.den)


def reset(cfg, seed, env_id, t):
    """Draw a fresh episode for ``env_id`` from the reset stream at step ``t``."""
    A, F, H, W = cfg.n_agents, cfg.n_food, cfg.grid_h, cfg.grid_w
    draws = iter(philox.u32_draws(seed, env_id, t, philox.TAG_RESET, 2 * A + 2 * F))
    agent_level = [1 + philox.uniform_int(next(draws), cfg.max_agent_level) for _ in range(A)]
    fmax = min(cfg.max_food_level, sum(agent_level))
    food_level = [1 + philox.uniform_int(next(draws), fmax) for _ in range(F)]
    if cfg.const_levels:
        agent_level = [cfg.max_agent_level] * A
        food_level = [cfg.max_food_level] * F
    food_cell = []
    for _ in range(F):
        free = [r * W + c for r in range(1, H - 1) for c in range(1, W - 1)
                if r * W + c not in food_cell]
        food_cell.append(free[philox.uniform_int(next(draws), len(free))])
    agent_cell = []
    for _ in range(A):
        free = [x for x in range(H * W) if x not in food_cell and x not in agent_cell]
        agent_cell.append(free[philox.uniform_int(next(draws), len(free))])
    return State(agent_cell, agent_level, food_cell, food_level, [False] * F, 0, sum(food_level))


def _adjacent(cfg, a, b):
    ra, ca = divmod(a, cfg.grid_w)
    rb, cb = divmod(b, cfg.grid_w)
    return abs(ra - rb) + abs(ca - cb) == 1


def transition(cfg, state, actions):
    """Apply one joint action.  Returns (next_state, reward float32, done bits).

    ``next_state`` is the post-transition state before any auto-reset.
    """
    H, W = cfg.grid_h, cfg.grid_w
    A = cfg.n_agents
    acts = [a if 0 <= a < N_ACTIONS else NOOP for a in (int(x) for x in actions)]
    food_here = {c for c, e in zip(state.food_cell, state.food_eaten) if not e}
    occupied = set(state.agent_cell)

    targets = []
    for i in range(A):
        tgt = None
        if acts[i] in _DELTA:
            r, c = divmod(state.agent_cell[i], W)
            dr, dc = _DELTA[acts[i]]
            r2, c2 = r + dr, c + dc
            if 0 <= r2 < H and 0 <= c2 < W:
                cell = r2 * W + c2
                if cell not in food_here and cell not in occupied:
                    tgt = cell
        targets.append(tgt)
    new_cell = list(state.agent_cell)
    for i in range(A):
        if targets[i] is not None and sum(1 for t in targets if t == targets[i]) == 1:
            new_cell[i] = targets[i]

    eaten_now = 0
    new_eaten = list(state.food_eaten)
    for j in range(cfg.n_food):
        if state.food_eaten[j]:
            continue
        loaders = [i for i in range(A)
                   if acts[i] == LOAD and _adjacent(cfg, state.agent_cell[i], state.food_cell[j])]
        if loaders and sum(state.agent_level[i] for i in loaders) >= state.food_level[j]:
            new_eaten[j] = True
            eaten_now += state.food_level[j]

    reward = np.float32(eaten_now) / np.float32(state.den)
    step_count = state.step_count + 1
    done = 0
    if all(new_eaten):
        done |= 1
    if step_count >= cfg.max_steps:
        done |= 2
    nxt = State(new_cell, list(state.agent_level), list(state.food_cell), list(state.food_level),
                new_eaten, step_count, state.den)
    return nxt, np.float32(reward), done


def step(cfg, seed, env_id, t, state, actions):
    """Transition at step ``t`` followed by the auto-reset.

    Returns (state_{t+1}, reward, done): when done, state_{t+1} is the fresh
    episode drawn from the reset stream at step t + 1 and the step count
    restarts at 0.
    """
    nxt, reward, done = transition(cfg, state, actions)
    if done:
        nxt = reset(cfg, seed, env_id, t + 1)
    return nxt, reward, done


def observe(cfg, state, agent):
    """Observation of ``agent`` as a float64 vector of length 3*H*W."""
    HW = cfg.grid_h * cfg.grid_w
    o = np.zeros(3 * HW, dtype=np.float64)
    for k in range(cfg.n_agents):
        o[state.agent_cell[k]] = state.agent_level[k]
    for j in range(cfg.n_food):
        if not state.food_eaten[j]:
            o[HW + state.food_cell[j]] = state.food_level[j]
    o[2 * HW + state.agent_cell[agent]] = 1.0
    return o


def legal_mask(cfg, state, agent):
    """Every LBF action is always legal."""
    return [True] * N_ACTIONS
