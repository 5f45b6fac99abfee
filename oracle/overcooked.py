"""Overcooked-style two-agent kitchen, plain CPU reference (test infrastructure).

The paper runs Overcooked (Section 4, environment table: the JaxMARL version
with five named layouts) as a cooperative Dec-POMDP (Section 3).  The named
layouts are not available here; seeded synthetic kitchens stand in for them.
The rules the paper does not restate follow these readings.

Canvas and cells
    Kitchens are W x H with W in 5..9 and H in 4..5, placed at the top-left of
    a fixed 5-row x 9-column canvas (cell id = row * 9 + col).  Cell types:
    FLOOR, COUNTER (the border, interior counters, and every canvas cell
    outside the kitchen), ONION (dispenser), PLATE (dispenser), POT, SERVE.

Layout (drawn once per env, TAG_LAYOUT stream, the attempt number in the
step slot of the counter; draws consumed in this order per attempt):
    1. W = 5 + u(5), H = 4 + u(2)                  (u(n) = uniform_int(draw, n))
    2. n_ic = u(floor((H-2)(W-2)/4) + 1) interior counters, each on the
       u(n)-th still-free interior cell (row-major)
    3. n_onion = 1 + u(2), n_pot = 1 + u(2); then n_onion onion dispensers,
       n_pot pots, one plate dispenser and one serving cell, each on the u(n)-th
       remaining candidate: a non-corner border cell with a FLOOR 4-neighbour
       (row-major)
    4. valid iff the floor is 4-connected, has >= 2 cells and no station ran
       out of candidates; otherwise the next attempt.  After 64 invalid
       attempts, attempt 64 is used with n_ic forced to 0 (always valid).

Reset (initial-state distribution rho), TAG_RESET stream at step t:
    the layout is kept; agent 0 on the u(n_floor)-th floor cell, agent 1 on the
    u(n_floor - 1)-th of the others; both face north; hands, pots and counters
    empty; step count 0.

Actions: 0 noop, 1 north, 2 south, 3 west, 4 east, 5 interact (out of range:
noop).  Facing: 0 N, 1 S, 2 W, 3 E.  Held items: 0 none, 1 onion, 2 plate,
3 soup.

Step (transition P and shared reward r), in this order:
    1. A move action sets the agent's facing to that direction even when
       blocked.  A move is legal iff the target is FLOOR and held no agent
       before the step; legal movers sharing a target both stay.
    2. Interacts, agent 0 then agent 1, on the cell each faces (after the
       moves), each seeing the state left by the previous one:
         ONION / PLATE dispenser + empty hand -> take an onion / a plate;
         POT + onion + pot idle with < 3 onions -> add it; the third onion
           starts cooking with timer = cook_time;
         POT + plate + pot ready -> the hand holds a soup, the pot empties;
         SERVE + soup -> reward += soup_reward, the hand empties;
         COUNTER + item + empty counter -> place it;
         COUNTER + empty hand + item on it -> pick it up;
         anything else -> nothing.
    3. Every pot that was cooking before this step decrements its timer; a pot
       with 3 onions and timer 0 is ready (plateable from step k + cook_time + 1
       when the third onion went in at step k).
    4. step count += 1; done = 2 (truncated) when it reaches max_steps; there
       is no terminal state.

Observation of agent i: 26 planes over the 45 canvas cells, plane-major:
    0 own cell, 1 other's cell, 2-5 own facing (at own cell), 6-9 other's
    facing (at other's cell), 10 COUNTER, 11 ONION, 12 PLATE, 13 POT, 14 SERVE,
    15-17 onion / plate / soup lying on a counter, 18-20 own held onion /
    plate / soup (at own cell), 21-23 the other's (at its cell), 24 onions in
    the pot (at the pot cell), 25 cooking timer remaining (at the pot cell).
"""

from dataclasses import dataclass, field

import numpy as np

from . import philox

CH, CW = 5, 9
NCELL = CH * CW
FLOOR, COUNTER, ONION, PLATE, POT, SERVE = range(6)
NOOP, NORTH, SOUTH, WEST, EAST, INTERACT = range(6)
N_ACTIONS = 6
N_PLANES = 26
HELD_NONE, HELD_ONION, HELD_PLATE, HELD_SOUP = range(4)
_DIR = {0: (-1, 0), 1: (1, 0), 2: (0, -1), 3: (0, 1)}  # facing -> (drow, dcol)
MAX_ATTEMPTS = 64


@dataclass(frozen=True)
class Config:
    cook_time: int = 20
    soup_reward: int = 20
    max_steps: int = 400
    n_agents: int = 2

    @property
    def obs_dim(self):
        return N_PLANES * NCELL


@dataclass
class State:
    W: int
    H: int
    cells: list           # [45] cell types
    items: list           # [45] item on each counter cell (0 none, 1 onion, 2 plate, 3 soup)
    agent_cell: list      # [2]
    facing: list          # [2]
    held: list            # [2]
    pot_onions: dict = field(default_factory=dict)  # pot cell -> onions 0..3
    pot_timer: dict = field(default_factory=dict)   # pot cell -> timer 0..cook_time
    step_count: int = 0

    def copy(self):
        return State(self.W, self.H, list(self.cells), list(self.items), list(self.agent_cell), list(self.facing),
                     list(self.held), dict(self.pot_onions), dict(self.pot_timer), self.step_count)

    def pots(self):
        return [c for c in range(NCELL) if self.cells[c] == POT]


class _Draws:
    """Sequential 32-bit draws of one (env, t, tag) stream."""

    def __init__(self, seed, env_id, t, tag):
        self.seed, self.env, self.t, self.tag = seed, env_id, t, tag
        self.buf = []
        self.sub = 0

    def u(self, n):
        if not self.buf:
            for w in philox.block(self.seed, self.env, self.t, self.sub, self.tag):
                self.buf += [(w >> 32) & philox.MASK32, w & philox.MASK32]
            self.sub += 1
        return philox.uniform_int(self.buf.pop(0), n)


def _neighbours(c):
    r, q = divmod(c, CW)
    for dr, dq in _DIR.values():
        r2, q2 = r + dr, q + dq
        if 0 <= r2 < CH and 0 <= q2 < CW:
            yield r2 * CW + q2


def floor_connected(cells):
    """True iff the FLOOR cells form one 4-connected component (breadth-first search)."""
    floor = [c for c in range(NCELL) if cells[c] == FLOOR]
    if not floor:
        return False
    seen = {floor[0]}
    frontier = [floor[0]]
    while frontier:
        nxt = []
        for c in frontier:
            for n in _neighbours(c):
                if cells[n] == FLOOR and n not in seen:
                    seen.add(n)
                    nxt.append(n)
        frontier = nxt
    return len(seen) == len(floor)


def _attempt(seed, env_id, attempt, force_no_counters):
    d = _Draws(seed, env_id, attempt, philox.TAG_LAYOUT)
    W = 5 + d.u(5)
    H = 4 + d.u(2)
    cells = [COUNTER] * NCELL
    for r in range(1, H - 1):
        for q in range(1, W - 1):
            cells[r * CW + q] = FLOOR
    n_ic = d.u((H - 2) * (W - 2) // 4 + 1)
    if force_no_counters:
        n_ic = 0
    for _ in range(n_ic):
        free = [r * CW + q for r in range(1, H - 1) for q in range(1, W - 1) if cells[r * CW + q] == FLOOR]
        cells[free[d.u(len(free))]] = COUNTER
    n_onion = 1 + d.u(2)
    n_pot = 1 + d.u(2)
    corners = {0, W - 1, (H - 1) * CW, (H - 1) * CW + W - 1}
    border = [r * CW + q for r in range(H) for q in range(W)
              if (r in (0, H - 1) or q in (0, W - 1)) and r * CW + q not in corners]
    ok = True
    for kind in [ONION] * n_onion + [POT] * n_pot + [PLATE, SERVE]:
        cand = [c for c in border if cells[c] == COUNTER and any(cells[n] == FLOOR for n in _neighbours(c))]
        if not cand:
            ok = False
            break
        cells[cand[d.u(len(cand))]] = kind
    n_floor = sum(1 for c in cells if c == FLOOR)
    ok = ok and n_floor >= 2 and floor_connected(cells)
    return ok, W, H, cells


def layout(seed, env_id):
    """(W, H, cells) of env_id's kitchen."""
    for a in range(MAX_ATTEMPTS):
        ok, W, H, cells = _attempt(seed, env_id, a, False)
        if ok:
            return W, H, cells
    ok, W, H, cells = _attempt(seed, env_id, MAX_ATTEMPTS, True)
    assert ok
    return W, H, cells


def reset_agents(cfg, seed, env_id, t, W, H, cells):
    """A fresh episode on a kept layout, from the reset stream at step t."""
    d = _Draws(seed, env_id, t, philox.TAG_RESET)
    floor = [c for c in range(NCELL) if cells[c] == FLOOR]
    a0 = floor[d.u(len(floor))]
    rest = [c for c in floor if c != a0]
    a1 = rest[d.u(len(rest))]
    pots = [c for c in range(NCELL) if cells[c] == POT]
    return State(W, H, list(cells), [0] * NCELL, [a0, a1], [0, 0], [HELD_NONE, HELD_NONE],
                 {c: 0 for c in pots}, {c: 0 for c in pots}, 0)


def reset(cfg, seed, env_id, t, layout_of=None):
    """Initial state of env_id at step t (its layout drawn from the layout stream)."""
    W, H, cells = layout(seed, env_id) if layout_of is None else layout_of
    return reset_agents(cfg, seed, env_id, t, W, H, cells)


def _faced(cell, facing):
    r, q = divmod(cell, CW)
    dr, dq = _DIR[facing]
    r2, q2 = r + dr, q + dq
    if 0 <= r2 < CH and 0 <= q2 < CW:
        return r2 * CW + q2
    return None


def transition(cfg, state, actions):
    """One joint action; returns (next_state, reward float32, done bits) without reset."""
    s = state.copy()
    acts = [a if 0 <= a < N_ACTIONS else NOOP for a in (int(x) for x in actions)]
    # 1. facing and moves against the pre-step state
    targets = []
    for i in range(2):
        tgt = None
        if NORTH <= acts[i] <= EAST:
            s.facing[i] = acts[i] - 1
            n = _faced(state.agent_cell[i], s.facing[i])
            if n is not None and state.cells[n] == FLOOR and n not in state.agent_cell:
                tgt = n
        targets.append(tgt)
    for i in range(2):
        if targets[i] is not None and targets[i] != targets[1 - i]:
            s.agent_cell[i] = targets[i]
    # 2. interacts in agent order
    cooking_before = {c for c in state.pots() if state.pot_onions[c] == 3 and state.pot_timer[c] > 0}
    reward = 0
    for i in range(2):
        if acts[i] != INTERACT:
            continue
        c = _faced(s.agent_cell[i], s.facing[i])
        if c is None:
            continue
        kind, h = s.cells[c], s.held[i]
        if kind == ONION and h == HELD_NONE:
            s.held[i] = HELD_ONION
        elif kind == PLATE and h == HELD_NONE:
            s.held[i] = HELD_PLATE
        elif kind == POT:
            n, tm = s.pot_onions[c], s.pot_timer[c]
            if h == HELD_ONION and n < 3:
                s.held[i] = HELD_NONE
                s.pot_onions[c] = n + 1
                if n + 1 == 3:
                    s.pot_timer[c] = cfg.cook_time
            elif h == HELD_PLATE and n == 3 and tm == 0:
                s.held[i] = HELD_SOUP
                s.pot_onions[c] = 0
        elif kind == SERVE and h == HELD_SOUP:
            s.held[i] = HELD_NONE
            reward += cfg.soup_reward
        elif kind == COUNTER:
            if h != HELD_NONE and s.items[c] == 0:
                s.items[c] = h
                s.held[i] = HELD_NONE
            elif h == HELD_NONE and s.items[c] != 0:
                s.held[i] = s.items[c]
                s.items[c] = 0
    # 3. cooking
    for c in cooking_before:
        s.pot_timer[c] -= 1
    s.step_count += 1
    done = 2 if s.step_count >= cfg.max_steps else 0
    return s, np.float32(reward), done


def step(cfg, seed, env_id, t, state, actions):
    """Transition at step t, then the auto-reset (layout kept) when done."""
    nxt, reward, done = transition(cfg, state, actions)
    if done:
        nxt = reset_agents(cfg, seed, env_id, t + 1, nxt.W, nxt.H, nxt.cells)
    return nxt, reward, done


def observe(cfg, state, agent):
    """Observation of `agent` as a float64 vector of 26 * 45 features."""
    o = np.zeros((N_PLANES, NCELL), dtype=np.float64)
    me, other = agent, 1 - agent
    for who, base_pos, base_face, base_held in ((me, 0, 2, 18), (other, 1, 6, 21)):
        c = state.agent_cell[who]
        o[base_pos, c] = 1
        o[base_face + state.facing[who], c] = 1
        if state.held[who] != HELD_NONE:
            o[base_held + state.held[who] - 1, c] = 1
    for c in range(NCELL):
        k = state.cells[c]
        if k != FLOOR:
            o[10 + k - 1, c] = 1
        if state.items[c]:
            o[15 + state.items[c] - 1, c] = 1
    for c in state.pots():
        o[24, c] = state.pot_onions[c]
        o[25, c] = state.pot_timer[c]
    return o.reshape(-1)


def legal_mask(cfg, state, agent):
    """Every action is always legal."""
    return [True] * N_ACTIONS
