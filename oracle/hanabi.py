"""Two-player Hanabi, plain CPU reference (test infrastructure).

The paper runs Hanabi (Section 4, environment table: the JaxMARL version with
the full 5 colours x 5 ranks game) as a cooperative Dec-POMDP (Section 3).
The benchmark workload fixes 2 players, a 50-card deck, hands of 5, 8 info
tokens, 3 lives, 20 actions (play / discard per hand slot, colour / rank
hints) with illegal actions masked out before sampling, and a 658-feature
observation.  What the paper leaves open is fixed by these readings.

Cards and deck
    card id = colour * R + (rank - 1); rank 1 has 3 copies, ranks 2..R-1 two,
    rank R one (50 cards for 5 x 5).  The unshuffled deck lists colours in
    order and, within a colour, ranks in order with their copies.
Reset (initial-state distribution rho), TAG_RESET stream at step t:
    Fisher-Yates: for i = N-1 down to 1, j = u(i + 1) (N - 1 draws, u(n) =
    uniform_int(draw, n)), swap deck[i] and deck[j].  Player 0 is dealt
    deck[0..H-1] into slots 0..H-1, player 1 deck[H..2H-1]; the next card
    drawn is deck[2H].  Player 0 moves first; all info tokens and lives are
    available; fireworks and discards are empty; knowledge is blank.
Actions (2 players, hand size H): 0..H-1 discard slot, H..2H-1 play slot,
    2H..2H+C-1 hint colour c to the partner, 2H+C..2H+C+R-1 hint rank r.
Legal actions of the player to move: play a held slot; discard a held slot
    when info tokens < max; hint a colour / rank when tokens > 0 and the
    partner holds at least one matching card.  The other player has no legal
    action (its row of the mask is all zero and its action is ignored).  An
    illegal or out-of-range action of the mover acts as its lowest-index
    legal action.
Step (transition P and shared reward r):
    play   the card extends its colour's firework iff its rank is one above
           the firework's height: reward +1, and a completed firework (rank
           R) returns one info token if below the maximum; otherwise the
           card goes to the discards and a life is lost.
    discard the card goes to the discards, +1 info token.
    After a play or discard, the hand closes up (later slots move left one)
    and, if the deck is not empty, the drawn card enters the last slot with
    blank knowledge.
    hint   costs one token; every partner card of that colour (rank) learns
           it exactly (its possible set becomes that one value and the hint
           is recorded); every other partner card drops that value from its
           possible set.
    The move passes to the other player.
End of a game (done bit 0, terminated):
    all lives lost: the reward of that step is minus the fireworks total
    (the game scores 0); every firework complete; or the second step after
    the step that drew the last card of the deck.  done bit 1 (truncated)
    when the episode reaches max_steps.  A done env is reset with the draws
    of step t + 1.
Observation of agent i (the observer), features in this order (658 for 5x5):
    partner hand      H slots x C*R one-hot of the card          125
    missing cards     [observer hand short, partner hand short]      2
    deck thermometer  bit k = more than k cards left, N - 2H bits   40
    fireworks         per colour, one-hot of its height (none at 0)  25
    info tokens       thermometer                                    8
    lives             thermometer                                    3
    discards          per card id, thermometer of its copies        50
    last action       actor (relative to the observer) 2, kind 4
                      (play, discard, hint colour, hint rank), hint
                      target (relative) 2, hinted colour C, hinted rank
                      R, revealed slots H, acted slot H, the played /
                      discarded card C*R, play succeeded 1, info token
                      gained 1 -- all zero before the first move       55
    knowledge         observer then partner, H slots x (C*R plausible
                      cards, hinted colour one-hot C, hinted rank
                      one-hot R); empty slots are zero                 350
    plausible(c, r) = colour c and rank r both still possible for the card.
"""

from dataclasses import dataclass

import numpy as np

from . import philox

LAST_PLAY, LAST_DISCARD, LAST_HINT_COLOUR, LAST_HINT_RANK = range(4)


@dataclass(frozen=True)
class Config:
    colours: int = 5
    ranks: int = 5
    hand_size: int = 5
    info_tokens: int = 8
    life_tokens: int = 3
    max_steps: int = 1000
    n_agents: int = 2

    @property
    def copies(self):
        """Copies of each rank (index rank - 1)."""
        return [3] + [2] * (self.ranks - 2) + [1] if self.ranks > 1 else [3]

    @property
    def n_cards(self):
        return self.colours * sum(self.copies)

    @property
    def n_actions(self):
        return 2 * self.hand_size + self.colours + self.ranks

    @property
    def obs_dim(self):
        C, R, H = self.colours, self.ranks, self.hand_size
        last = 2 + 4 + 2 + C + R + H + H + C * R + 1 + 1
        return (H * C * R + 2 + (self.n_cards - 2 * H) + C * R + self.info_tokens + self.life_tokens
                + self.n_cards + last + 2 * H * (C * R + C + R))


N_ACTIONS = Config().n_actions  # 20 for the standard game


@dataclass
class Knowledge:
    colours: int          # bitmask of still-possible colours
    ranks: int            # bitmask of still-possible ranks (bit r - 1)
    hint_colour: int = -1
    hint_rank: int = -1   # 1..R once hinted

    def copy(self):
        return Knowledge(self.colours, self.ranks, self.hint_colour, self.hint_rank)


@dataclass
class LastAction:
    actor: int
    kind: int
    target: int = -1      # hinted player
    colour: int = -1      # hinted colour
    rank: int = -1        # hinted rank
    revealed: int = 0     # bitmask of target slots matching the hint
    slot: int = -1        # played / discarded slot
    card: int = -1        # played / discarded card
    success: bool = False
    token: bool = False


@dataclass
class State:
    deck: list            # the shuffled deck; deck[next_card:] is still to be drawn
    next_card: int
    hands: list           # [2] lists of card ids, slot order
    know: list            # [2] lists of Knowledge, parallel to hands
    fireworks: list       # [C] heights 0..R
    discards: list        # [C*R] copies discarded
    info: int
    lives: int
    cur: int              # player to move
    turns_left: int       # -1 while the deck has cards, else moves left in the game
    last: object = None   # LastAction or None
    step_count: int = 0

    def copy(self):
        return State(list(self.deck), self.next_card, [list(h) for h in self.hands],
                     [[k.copy() for k in ks] for ks in self.know], list(self.fireworks), list(self.discards),
                     self.info, self.lives, self.cur, self.turns_left,
                     None if self.last is None else LastAction(**vars(self.last)), self.step_count)


def colour_of(cfg, card):
    return card // cfg.ranks


def rank_of(cfg, card):
    return card % cfg.ranks + 1


def ordered_deck(cfg):
    deck = []
    for c in range(cfg.colours):
        for r in range(1, cfg.ranks + 1):
            deck += [c * cfg.ranks + r - 1] * cfg.copies[r - 1]
    return deck


def fisher_yates(items, draws):
    """Shuffle a copy of ``items`` with one uniform_int draw per position from the top down."""
    a = list(items)
    k = 0
    for i in range(len(a) - 1, 0, -1):
        j = philox.uniform_int(draws[k], i + 1)
        k += 1
        a[i], a[j] = a[j], a[i]
    return a


def _blank(cfg):
    return Knowledge((1 << cfg.colours) - 1, (1 << cfg.ranks) - 1)


def reset(cfg, seed, env_id, t):
    deck0 = ordered_deck(cfg)
    draws = philox.u32_draws(seed, env_id, t, philox.TAG_RESET, len(deck0) - 1)
    deck = fisher_yates(deck0, draws)
    H = cfg.hand_size
    hands = [deck[0:H], deck[H:2 * H]]
    know = [[_blank(cfg) for _ in range(H)] for _ in range(2)]
    return State(deck, 2 * H, hands, know, [0] * cfg.colours, [0] * (cfg.colours * cfg.ranks), cfg.info_tokens,
                 cfg.life_tokens, 0, -1, None, 0)


def legal_mask(cfg, state, agent):
    C, R, H = cfg.colours, cfg.ranks, cfg.hand_size
    m = [False] * cfg.n_actions
    if agent != state.cur:
        return m
    hand = state.hands[agent]
    partner = state.hands[1 - agent]
    for i in range(len(hand)):
        m[H + i] = True
        m[i] = state.info < cfg.info_tokens
    if state.info > 0:
        for c in range(C):
            m[2 * H + c] = any(colour_of(cfg, x) == c for x in partner)
        for r in range(1, R + 1):
            m[2 * H + C + r - 1] = any(rank_of(cfg, x) == r for x in partner)
    return m


def transition(cfg, state, actions):
    """The mover's action (illegal -> its lowest legal one); returns (next_state, reward float32, done bits)."""
    C, R, H = cfg.colours, cfg.ranks, cfg.hand_size
    s = state.copy()
    p, q = state.cur, 1 - state.cur
    mask = legal_mask(cfg, state, p)
    a = int(actions[p])
    if not (0 <= a < cfg.n_actions and mask[a]):
        a = mask.index(True)
    reward = 0
    terminated = False
    drew_last = False
    if a < 2 * H:
        slot = a % H
        card = s.hands[p][slot]
        last = LastAction(p, LAST_DISCARD if a < H else LAST_PLAY, slot=slot, card=card)
        if a < H:
            s.discards[card] += 1
            s.info += 1
            last.token = True
        else:
            c, r = colour_of(cfg, card), rank_of(cfg, card)
            if s.fireworks[c] + 1 == r:
                s.fireworks[c] = r
                reward += 1
                last.success = True
                if r == R and s.info < cfg.info_tokens:
                    s.info += 1
                    last.token = True
            else:
                s.discards[card] += 1
                s.lives -= 1
        del s.hands[p][slot]
        del s.know[p][slot]
        if s.next_card < len(s.deck):
            s.hands[p].append(s.deck[s.next_card])
            s.know[p].append(_blank(cfg))
            s.next_card += 1
            drew_last = s.next_card == len(s.deck)
    else:
        h = a - 2 * H
        is_colour = h < C
        val = h if is_colour else h - C + 1
        last = LastAction(p, LAST_HINT_COLOUR if is_colour else LAST_HINT_RANK, target=q,
                          colour=val if is_colour else -1, rank=-1 if is_colour else val)
        s.info -= 1
        for i, card in enumerate(s.hands[q]):
            k = s.know[q][i]
            if is_colour:
                if colour_of(cfg, card) == val:
                    k.colours, k.hint_colour = 1 << val, val
                    last.revealed |= 1 << i
                else:
                    k.colours &= ~(1 << val)
            else:
                if rank_of(cfg, card) == val:
                    k.ranks, k.hint_rank = 1 << (val - 1), val
                    last.revealed |= 1 << i
                else:
                    k.ranks &= ~(1 << (val - 1))
    s.last = last
    if s.turns_left > 0:
        s.turns_left -= 1
    if drew_last:
        s.turns_left = 2  # one more move for each player
    if s.lives == 0:
        terminated = True
        reward = -sum(state.fireworks)
    elif all(f == R for f in s.fireworks) or s.turns_left == 0:
        terminated = True
    s.cur = q
    s.step_count += 1
    done = (1 if terminated else 0) | (2 if s.step_count >= cfg.max_steps else 0)
    return s, np.float32(reward), done


def step(cfg, seed, env_id, t, state, actions):
    """Transition at step t, then the auto-reset when done."""
    nxt, reward, done = transition(cfg, state, actions)
    if done:
        nxt = reset(cfg, seed, env_id, t + 1)
    return nxt, reward, done


def observe(cfg, state, agent):
    """Observation of ``agent`` as a float64 vector of cfg.obs_dim features (0/1)."""
    C, R, H = cfg.colours, cfg.ranks, cfg.hand_size
    CR = C * R
    me, other = agent, 1 - agent
    parts = []
    ph = np.zeros((H, CR))
    for i, card in enumerate(state.hands[other]):
        ph[i, card] = 1
    parts.append(ph.reshape(-1))
    parts.append(np.array([len(state.hands[me]) < H, len(state.hands[other]) < H], dtype=np.float64))
    left = len(state.deck) - state.next_card
    parts.append(np.array([left > k for k in range(cfg.n_cards - 2 * H)], dtype=np.float64))
    fw = np.zeros((C, R))
    for c in range(C):
        if state.fireworks[c] > 0:
            fw[c, state.fireworks[c] - 1] = 1
    parts.append(fw.reshape(-1))
    parts.append(np.array([state.info > k for k in range(cfg.info_tokens)], dtype=np.float64))
    parts.append(np.array([state.lives > k for k in range(cfg.life_tokens)], dtype=np.float64))
    disc = []
    for card in range(CR):
        n = cfg.copies[rank_of(cfg, card) - 1]
        disc += [state.discards[card] > k for k in range(n)]
    parts.append(np.array(disc, dtype=np.float64))
    la = np.zeros(2 + 4 + 2 + C + R + H + H + CR + 2)
    if state.last is not None:
        L = state.last
        o = 0
        la[o + (L.actor - me) % 2] = 1
        o += 2
        la[o + L.kind] = 1
        o += 4
        if L.kind in (LAST_HINT_COLOUR, LAST_HINT_RANK):
            la[o + (L.target - me) % 2] = 1
        o += 2
        if L.kind == LAST_HINT_COLOUR:
            la[o + L.colour] = 1
        o += C
        if L.kind == LAST_HINT_RANK:
            la[o + L.rank - 1] = 1
        o += R
        for i in range(H):
            if (L.revealed >> i) & 1:
                la[o + i] = 1
        o += H
        if L.kind in (LAST_PLAY, LAST_DISCARD):
            la[o + L.slot] = 1
            la[o + H + L.card] = 1
        o += H + CR
        la[o] = float(L.success)
        la[o + 1] = float(L.token)
    parts.append(la)
    kn = np.zeros((2, H, CR + C + R))
    for j, who in enumerate((me, other)):
        for i, k in enumerate(state.know[who]):
            for c in range(C):
                for r in range(R):
                    if (k.colours >> c) & 1 and (k.ranks >> r) & 1:
                        kn[j, i, c * R + r] = 1
            if k.hint_colour >= 0:
                kn[j, i, CR + k.hint_colour] = 1
            if k.hint_rank >= 1:
                kn[j, i, CR + C + k.hint_rank - 1] = 1
    parts.append(kn.reshape(-1))
    o = np.concatenate(parts)
    assert o.size == cfg.obs_dim
    return o
