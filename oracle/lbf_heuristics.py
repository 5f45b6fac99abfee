"""Heuristic LBF teammates (test infrastructure).

The paper's LBF evaluation teammates (Appendix, the table of heuristic
teammates) include Sequential agents, which plan a food order before the
episode from a fixed ordering of the food cells, and Greedy agents, which pick
the next uneaten food online by a criterion.  The paper names the variants but
not their mechanics; this module is the reading the rollout kernels implement:

* target: Greedy variants take the uneaten food minimising their key, ties to
  the lowest food index: closest_self (Manhattan distance from the agent),
  closest_teammate (from agent (i + 1) mod A), closest_avg (sum of both
  distances), lowest_level / highest_level (food level, then distance from
  the agent).  Sequential variants take the first uneaten food in a fixed
  order of the food cells: lexicographic (row, then column), its reverse,
  column_major (column, then row), its reverse.  These orders depend only on
  the food cells, which do not move, so the plan made at the episode start is
  the same order read at every step.  nearest_agent / farthest_agent order
  the foods by Manhattan distance from the agent's cell at the start of the
  episode, nearest (farthest) first: the plan the agent makes before the
  episode from where it stands.  The env state does not hold that start
  cell; a rollout passes it (``start_cell``): the agent's cell in the first
  state of its episode, as observed.
* action: LOAD when the agent is next to its target (4-neighbourhood);
  otherwise one step along the axis with the larger remaining distance (the
  row axis on ties): NORTH/SOUTH by the sign of the row difference,
  WEST/EAST by the column difference.  When that cell holds an uneaten food
  or another agent and the other axis also closes in, the step goes along
  the other axis instead; otherwise the blocked move is taken (the env
  leaves the agent in place).  The heuristics draw no random numbers.
* in a rollout, an agent driven by a heuristic gets the logits 0 for its
  action and -inf for the others, so the Gumbel-max sampler returns that
  action whatever its noise.
"""

import numpy as np

from . import lbf

KINDS = ("greedy_closest_self", "greedy_closest_teammate", "greedy_closest_avg", "greedy_lowest_level",
         "greedy_highest_level", "seq_lexicographic", "seq_reverse_lexicographic", "seq_column_major",
         "seq_reverse_column_major", "seq_nearest_agent", "seq_farthest_agent")
NEEDS_START = ("seq_nearest_agent", "seq_farthest_agent")  # kinds that read the agent's episode start cell


def _rc(cfg, cell):
    return divmod(cell, cfg.grid_w)


def _dist(cfg, a, b):
    (ra, ca), (rb, cb) = _rc(cfg, a), _rc(cfg, b)
    return abs(ra - rb) + abs(ca - cb)


def target(cfg, state, agent, kind, start_cell=None):
    """Index of the food the heuristic ``kind`` (an index into KINDS) heads for.

    ``start_cell``: the agent's cell at the start of the episode (needed by the kinds in NEEDS_START)."""
    name = KINDS[kind]
    if name in NEEDS_START and start_cell is None:
        raise ValueError(f"{name} plans from the agent's start cell; pass start_cell")
    me = state.agent_cell[agent]
    mate = state.agent_cell[(agent + 1) % cfg.n_agents]
    live = [j for j in range(cfg.n_food) if not state.food_eaten[j]]
    fc = state.food_cell
    keys = {
        "greedy_closest_self": lambda j: (_dist(cfg, me, fc[j]),),
        "greedy_closest_teammate": lambda j: (_dist(cfg, mate, fc[j]),),
        "greedy_closest_avg": lambda j: (_dist(cfg, me, fc[j]) + _dist(cfg, mate, fc[j]),),
        "greedy_lowest_level": lambda j: (state.food_level[j], _dist(cfg, me, fc[j])),
        "greedy_highest_level": lambda j: (-state.food_level[j], _dist(cfg, me, fc[j])),
        "seq_lexicographic": lambda j: _rc(cfg, fc[j]),
        "seq_reverse_lexicographic": lambda j: tuple(-x for x in _rc(cfg, fc[j])),
        "seq_column_major": lambda j: _rc(cfg, fc[j])[::-1],
        "seq_reverse_column_major": lambda j: tuple(-x for x in _rc(cfg, fc[j])[::-1]),
        "seq_nearest_agent": lambda j: (_dist(cfg, start_cell, fc[j]),),
        "seq_farthest_agent": lambda j: (-_dist(cfg, start_cell, fc[j]),),
    }[name]
    return min(live, key=lambda j: (keys(j), j))


def action(cfg, state, agent, kind, start_cell=None):
    """The heuristic's action for ``agent`` in ``state``."""
    j = target(cfg, state, agent, kind, start_cell)
    (r, c), (tr, tc) = _rc(cfg, state.agent_cell[agent]), _rc(cfg, state.food_cell[j])
    dr, dc = tr - r, tc - c
    if abs(dr) + abs(dc) == 1:
        return lbf.LOAD
    vert = lbf.NORTH if dr < 0 else lbf.SOUTH
    horiz = lbf.WEST if dc < 0 else lbf.EAST
    first, other = (vert, horiz) if abs(dr) >= abs(dc) else (horiz, vert)
    other_closes = dc != 0 if first == vert else dr != 0
    blocked = {c for c, e in zip(state.food_cell, state.food_eaten) if not e}
    blocked |= {x for i, x in enumerate(state.agent_cell) if i != agent}
    step = {lbf.NORTH: -cfg.grid_w, lbf.SOUTH: cfg.grid_w, lbf.WEST: -1, lbf.EAST: 1}
    if state.agent_cell[agent] + step[first] in blocked and other_closes:
        return other
    return first


def logits(cfg, state, agent, kind, start_cell=None):
    """float64 logits [nA] of the heuristic: 0 for its action, -inf for the others."""
    out = np.full(lbf.N_ACTIONS, -np.inf)
    out[action(cfg, state, agent, kind, start_cell)] = 0.0
    return out
