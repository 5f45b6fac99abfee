"""Python binding of the C-ABI rollout library (argument marshalling only).

Every function here has the name of the C entry point it calls and does no
arithmetic of its own: it checks tensor shapes/dtypes/devices, builds the
host structs, passes raw device pointers and the current HIP stream, and
raises ``RolloutError`` on a non-zero status.  PyTorch supplies device memory
and streams.  The library must have been built
(``python -m paper_2609_13716_amd.build``); importing this module fails
loudly otherwise -- there is no fallback path.
"""

import ctypes
import os
from dataclasses import dataclass, field

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# RL_LIB_PATH selects another build of the same library (the phase-stamped
# one of build.py --stamps); by default the product library next to this file.
LIB_PATH = os.environ.get("RL_LIB_PATH") or os.path.join(_HERE, "librollout.so")

RL_OK, RL_EINVAL, RL_EUNSUPPORTED, RL_ESHAPE, RL_EDEVICE = 0, -1, -2, -3, -4
RL_ENV_LBF, RL_ENV_OVERCOOKED, RL_ENV_HANABI = 0, 1, 2
RL_F32, RL_BF16 = 0, 1

_TORCH_DT = {RL_F32: torch.float32, RL_BF16: torch.bfloat16}
_DT_CODE = {"f32": RL_F32, "bf16": RL_BF16, torch.float32: RL_F32, torch.bfloat16: RL_BF16}


class RolloutError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"status {status}: {message}")
        self.status = status


class _EnvConfig(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32), ("n_envs", ctypes.c_int32), ("n_agents", ctypes.c_int32),
        ("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32), ("n_food", ctypes.c_int32),
        ("max_agent_level", ctypes.c_int32), ("max_food_level", ctypes.c_int32),
        ("max_steps", ctypes.c_int32), ("oc_cook_time", ctypes.c_int32),
        ("oc_soup_reward", ctypes.c_int32), ("hn_colors", ctypes.c_int32),
        ("hn_ranks", ctypes.c_int32), ("hn_hand_size", ctypes.c_int32),
        ("hn_info_tokens", ctypes.c_int32), ("hn_life_tokens", ctypes.c_int32),
        ("lbf_const_levels", ctypes.c_int32), ("env_base", ctypes.c_int64), ("seed", ctypes.c_uint64),
    ]


class _Policy(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("dims", ctypes.c_int32 * 4),
                ("W", ctypes.c_void_p * 3), ("b", ctypes.c_void_p * 3), ("packed", ctypes.c_void_p)]


class _Traj(ctypes.Structure):
    _fields_ = [("obs", ctypes.c_void_p), ("actions", ctypes.c_void_p), ("logits", ctypes.c_void_p),
                ("reward", ctypes.c_void_p), ("done", ctypes.c_void_p), ("obs_last", ctypes.c_void_p)]


class _AcTraj(ctypes.Structure):
    _fields_ = [("value", ctypes.c_void_p), ("logp", ctypes.c_void_p), ("value_last", ctypes.c_void_p)]


class _S5Policy(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("obs_dim", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("d_state", ctypes.c_int32), ("head_width", ctypes.c_int32), ("n_actions", ctypes.c_int32),
                ("w_enc", ctypes.c_void_p), ("b_enc", ctypes.c_void_p), ("lambda_bar", ctypes.c_void_p),
                ("b_bar", ctypes.c_void_p), ("c", ctypes.c_void_p), ("d", ctypes.c_void_p),
                ("actor_w", ctypes.c_void_p * 4), ("actor_b", ctypes.c_void_p * 4),
                ("critic_w", ctypes.c_void_p * 4), ("critic_b", ctypes.c_void_p * 4)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2609_13716_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, cfgp, st = ctypes.c_void_p, ctypes.POINTER(_EnvConfig), ctypes.c_int32
    lib.rl_state_bytes.argtypes, lib.rl_state_bytes.restype = [cfgp], ctypes.c_size_t
    lib.rl_obs_dim.argtypes, lib.rl_obs_dim.restype = [cfgp], ctypes.c_int32
    lib.rl_num_actions.argtypes, lib.rl_num_actions.restype = [cfgp], ctypes.c_int32
    lib.rollout_last_error.argtypes, lib.rollout_last_error.restype = [], ctypes.c_char_p
    lib.rollout_init.argtypes, lib.rollout_init.restype = [cfgp, P, P, ctypes.c_int32, P, P], st
    lib.rollout_step.argtypes = [cfgp, P, ctypes.c_uint64, ctypes.c_int32, P, P, ctypes.c_int32, P, P, P, P]
    lib.rollout_step.restype = st
    lib.policy_forward.argtypes = [ctypes.POINTER(_Policy), P, P, ctypes.c_int64, P, P]
    lib.policy_forward.restype = st
    lib.rollout_run.argtypes = [cfgp, ctypes.POINTER(_Policy), P, ctypes.c_uint64, ctypes.c_int32,
                                ctypes.POINTER(_Traj), P]
    lib.rollout_run.restype = st
    lib.rollout_run_ac.argtypes = [cfgp, ctypes.POINTER(_Policy), P, ctypes.c_uint64, ctypes.c_int32,
                                   ctypes.POINTER(_Traj), ctypes.POINTER(_AcTraj), P]
    lib.rollout_run_ac.restype = st
    lib.rl_gae.argtypes = [P, P, P, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_float, ctypes.c_float,
                           P, P, P]
    lib.rl_gae.restype = st
    lib.rollout_run_pop.argtypes = [cfgp, ctypes.POINTER(_Policy), ctypes.c_int32, P, P, ctypes.c_uint64,
                                    ctypes.c_int32, ctypes.POINTER(_Traj), P]
    lib.rollout_run_pop.restype = st
    lib.rollout_sample.argtypes = [cfgp, ctypes.c_uint64, P, P, P, P]
    lib.rollout_sample.restype = st
    lib.rl_gumbel_noise.argtypes, lib.rl_gumbel_noise.restype = [P, ctypes.c_int64, P, P], st
    lib.rollout_run_teams.argtypes = [cfgp, ctypes.POINTER(_Policy), P, P, ctypes.c_uint64, ctypes.c_int32,
                                      ctypes.POINTER(_Traj), P]
    lib.rollout_run_teams.restype = st
    s5p = ctypes.POINTER(_S5Policy)
    lib.rl_s5_discretize.argtypes = [ctypes.c_int32, ctypes.c_int32, P, P, P, P, P, P]
    lib.rl_s5_discretize.restype = st
    lib.rl_s5_workspace_bytes.argtypes, lib.rl_s5_workspace_bytes.restype = [cfgp, s5p], ctypes.c_size_t
    lib.rollout_run_s5.argtypes = [cfgp, s5p, P, P, ctypes.c_uint64, ctypes.c_int32, ctypes.POINTER(_Traj),
                                   ctypes.POINTER(_AcTraj), P, ctypes.c_size_t, P]
    lib.rollout_run_s5.restype = st
    lib.rollout_run_s5_noalloc.argtypes = [cfgp, s5p, P, P, ctypes.c_uint64, ctypes.c_int32, ctypes.POINTER(_Traj),
                                           ctypes.POINTER(_AcTraj), P]
    lib.rollout_run_s5_noalloc.restype = st
    lib.rl_policy_packed_bytes.argtypes = [ctypes.POINTER(_Policy)]
    lib.rl_policy_packed_bytes.restype = ctypes.c_size_t
    lib.rl_policy_pack.argtypes, lib.rl_policy_pack.restype = [ctypes.POINTER(_Policy), P, P], st
    return lib


lib = _load()

# Every symbol the C header declares (checked by the test suite).
EXPORTED = ("rl_state_bytes", "rl_obs_dim", "rl_num_actions", "rollout_last_error", "rollout_init",
            "rollout_step", "policy_forward", "rollout_run", "rollout_sample", "rl_gumbel_noise", "rollout_run_pop",
            "rollout_run_ac", "rl_gae", "rl_s5_discretize", "rl_s5_workspace_bytes", "rollout_run_s5",
            "rollout_run_teams", "rl_policy_packed_bytes", "rl_policy_pack", "rollout_run_s5_noalloc")
HEURISTICS = ("greedy_closest_self", "greedy_closest_teammate", "greedy_closest_avg", "greedy_lowest_level",
              "greedy_highest_level", "seq_lexicographic", "seq_reverse_lexicographic", "seq_column_major",
              "seq_reverse_column_major", "seq_nearest_agent", "seq_farthest_agent")  # kind k of rollout_run_teams


def _check(status):
    if status != RL_OK:
        raise RolloutError(status, lib.rollout_last_error().decode())


@dataclass
class EnvConfig:
    """Mirror of ``rl_env_config`` (defaults: LBF 8x8, 2 agents, 3 foods).

    Only the fields of ``kind`` are passed to the library (the LBF grid
    fields are sent as 0 for other kinds); ``extra`` holds the Overcooked /
    Hanabi fields by their C names."""
    n_envs: int
    kind: int = RL_ENV_LBF
    n_agents: int = 2
    grid_h: int = 8
    grid_w: int = 8
    n_food: int = 3
    max_agent_level: int = 2
    max_food_level: int = 3
    max_steps: int = 50
    const_levels: bool = False  # LBF constant-levels variant: agents at max_agent_level, foods at max_food_level
    env_base: int = 0
    seed: int = 0
    extra: dict = field(default_factory=dict)  # Overcooked / Hanabi fields

    def c(self):
        s = _EnvConfig()
        names = ("kind", "n_envs", "n_agents", "max_steps", "env_base", "seed")
        if self.kind == RL_ENV_LBF:
            names += ("grid_h", "grid_w", "n_food", "max_agent_level", "max_food_level")
            s.lbf_const_levels = int(self.const_levels)
        for k in names:
            setattr(s, k, getattr(self, k))
        for k, v in self.extra.items():
            setattr(s, k, v)
        return s


def overcooked_config(n_envs, cook_time=20, soup_reward=20, max_steps=400, env_base=0, seed=0):
    """An ``EnvConfig`` for the two-agent Overcooked-style kitchen."""
    return EnvConfig(n_envs, kind=RL_ENV_OVERCOOKED, n_agents=2, max_steps=max_steps, env_base=env_base, seed=seed,
                     extra={"oc_cook_time": cook_time, "oc_soup_reward": soup_reward})


def hanabi_config(n_envs, max_steps=1000, env_base=0, seed=0, colours=5, ranks=5):
    """An ``EnvConfig`` for two-player Hanabi: the standard 5 colours x 5 ranks game, or with colours=ranks=3
    the mini game (hands of 5, 8 info tokens, 3 lives either way)."""
    return EnvConfig(n_envs, kind=RL_ENV_HANABI, n_agents=2, max_steps=max_steps, env_base=env_base, seed=seed,
                     extra={"hn_colors": colours, "hn_ranks": ranks, "hn_hand_size": 5, "hn_info_tokens": 8,
                            "hn_life_tokens": 3})


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _need(t, name, dtype=None, shape=None):
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _need_state(cfg, state):
    """The env state buffer: a contiguous int32 device tensor of exactly rl_state_bytes(cfg) bytes."""
    if state is None:
        raise ValueError("state is required")
    n = rl_state_bytes(cfg)
    if n == 0:
        _check(lib.rl_obs_dim(ctypes.byref(cfg.c())))
    if state.numel() * state.element_size() != n:
        raise ValueError(f"state holds {state.numel() * state.element_size()} bytes; "
                         f"this config needs rl_state_bytes = {n}")
    _need(state, "state", torch.int32)


def rl_state_bytes(cfg):
    return lib.rl_state_bytes(ctypes.byref(cfg.c()))


def rl_obs_dim(cfg):
    return lib.rl_obs_dim(ctypes.byref(cfg.c()))


def rl_num_actions(cfg):
    return lib.rl_num_actions(ctypes.byref(cfg.c()))


class Policy:
    """Device weights of the 3-layer MLP in the nn.Linear layout, and the C struct pointing at them.

    ``pack`` (bf16 only; default on): also keep the fragment-major copy that
    ``rl_policy_pack`` writes, which the streamed-weight rollout kernels read.
    """

    def __init__(self, weights, biases, dtype="f32", device="cuda", pack=True):
        self.dtype = _DT_CODE[dtype]
        tdt = _TORCH_DT[self.dtype]
        self.W = [torch.as_tensor(w).to(device=device, dtype=tdt).contiguous() for w in weights]
        self.b = [torch.as_tensor(b).to(device=device, dtype=tdt).contiguous() for b in biases]
        self.dims = [self.W[0].shape[1]] + [w.shape[0] for w in self.W]
        self.packed = None
        if pack and self.dtype == _DT_CODE["bf16"]:
            pc = self.c()
            n = lib.rl_policy_packed_bytes(ctypes.byref(pc))
            if n == 0:
                raise RolloutError(RL_EINVAL, lib.rollout_last_error().decode())
            self.packed = torch.empty(n, dtype=torch.uint8, device=device)
            _check(lib.rl_policy_pack(ctypes.byref(pc), self.packed.data_ptr(), _stream(None)))

    @property
    def torch_dtype(self):
        return _TORCH_DT[self.dtype]

    def c(self):
        p = _Policy()
        p.dtype = self.dtype
        p.n_layers = len(self.W)
        for i, d in enumerate(self.dims):
            p.dims[i] = d
        for i in range(3):
            p.W[i] = self.W[i].data_ptr()
            p.b[i] = self.b[i].data_ptr()
        p.packed = self.packed.data_ptr() if getattr(self, "packed", None) is not None else None
        return p


class Population:
    """Device weights of n policies of one shape, stacked per layer ([n, fan_out, fan_in] and [n, fan_out]).

    ``weights[p]`` / ``biases[p]`` are policy p's layers in the nn.Linear layout.
    ``pack`` (bf16 only; default on): also keep the policies' fragment-major copies, policy p
    at p * rl_policy_packed_bytes, which the population rollout reads.
    """

    def __init__(self, weights, biases, dtype="f32", device="cuda", pack=True):
        if len(weights) < 1 or len(weights) != len(biases):
            raise ValueError("a population needs one (weights, biases) pair per policy")
        self.dtype = _DT_CODE[dtype]
        tdt = _TORCH_DT[self.dtype]
        self.n = len(weights)
        self.W = [torch.stack([torch.as_tensor(w[l]) for w in weights]).to(device=device, dtype=tdt).contiguous()
                  for l in range(3)]
        self.b = [torch.stack([torch.as_tensor(b[l]) for b in biases]).to(device=device, dtype=tdt).contiguous()
                  for l in range(3)]
        self.dims = [self.W[0].shape[2]] + [w.shape[1] for w in self.W]
        self.packed = None
        if pack and self.dtype == _DT_CODE["bf16"]:
            pc = self.c()
            per = lib.rl_policy_packed_bytes(ctypes.byref(pc))
            if per == 0:
                raise RolloutError(RL_EINVAL, lib.rollout_last_error().decode())
            self.packed = torch.empty(self.n * per, dtype=torch.uint8, device=device)
            for q in range(self.n):
                for i in range(3):
                    pc.W[i] = self.W[i][q].data_ptr()
                    pc.b[i] = self.b[i][q].data_ptr()
                _check(lib.rl_policy_pack(ctypes.byref(pc), self.packed.data_ptr() + q * per, _stream(None)))

    @property
    def torch_dtype(self):
        return _TORCH_DT[self.dtype]

    def c(self):
        p = _Policy()
        p.dtype = self.dtype
        p.n_layers = 3
        for i, d in enumerate(self.dims):
            p.dims[i] = d
        for i in range(3):
            p.W[i] = self.W[i].data_ptr()
            p.b[i] = self.b[i].data_ptr()
        p.packed = self.packed.data_ptr() if getattr(self, "packed", None) is not None else None
        return p


def new_state(cfg, device="cuda"):
    """A device buffer of rl_state_bytes(cfg) bytes (as int32)."""
    n = rl_state_bytes(cfg)
    if n == 0:
        _check(lib.rl_obs_dim(ctypes.byref(cfg.c())))
    return torch.empty(n // 4, dtype=torch.int32, device=device)


def rollout_init(cfg, state, obs=None, legal=None, stream=None):
    E, A = cfg.n_envs, cfg.n_agents
    D, nA = rl_obs_dim(cfg), rl_num_actions(cfg)
    _need_state(cfg, state)
    if obs is not None:
        _need(obs, "obs", shape=(E, A, D))
    _need(legal, "legal", torch.uint8, (E, A, nA))
    code = _DT_CODE.get(obs.dtype, -1) if obs is not None else RL_F32
    _check(lib.rollout_init(ctypes.byref(cfg.c()), _ptr(state), _ptr(obs), code, _ptr(legal), _stream(stream)))


def rollout_step(cfg, state, t0, actions, obs_out=None, reward=None, done=None, legal_out=None, stream=None):
    E, A = cfg.n_envs, cfg.n_agents
    D, nA = rl_obs_dim(cfg), rl_num_actions(cfg)
    _need_state(cfg, state)
    _need(actions, "actions", torch.int32)
    if actions.dim() != 3 or tuple(actions.shape[1:]) != (E, A):
        raise ValueError(f"actions must be [T, {E}, {A}], got {tuple(actions.shape)}")
    T = actions.shape[0]
    if obs_out is not None:
        _need(obs_out, "obs_out", shape=(T, E, A, D))
    _need(reward, "reward", torch.float32, (T, E))
    _need(done, "done", torch.uint8, (T, E))
    _need(legal_out, "legal_out", torch.uint8, (T, E, A, nA))
    code = _DT_CODE.get(obs_out.dtype, -1) if obs_out is not None else RL_F32
    _check(lib.rollout_step(ctypes.byref(cfg.c()), _ptr(state), t0, T, _ptr(actions), _ptr(obs_out), code,
                            _ptr(reward), _ptr(done), _ptr(legal_out), _stream(stream)))


def policy_forward(policy, obs, legal=None, logits=None, stream=None):
    rows = obs.shape[0]
    nA = policy.dims[3]
    _need(obs, "obs", policy.torch_dtype, (rows, policy.dims[0]))
    _need(legal, "legal", torch.uint8, (rows, nA))
    if logits is None:
        logits = torch.empty(rows, nA, dtype=torch.float32, device=obs.device)
    _need(logits, "logits", torch.float32, (rows, nA))
    pc = policy.c()
    _check(lib.policy_forward(ctypes.byref(pc), _ptr(obs), _ptr(legal), rows, _ptr(logits), _stream(stream)))
    return logits


def rollout_run(cfg, policy, state, t0, n_steps, obs=None, actions=None, logits=None, reward=None, done=None,
                obs_last=None, stream=None):
    E, A = cfg.n_envs, cfg.n_agents
    D, nA = rl_obs_dim(cfg), rl_num_actions(cfg)
    T = n_steps
    _need_state(cfg, state)
    _need(obs, "obs", policy.torch_dtype, (T, E, A, D))
    _need(actions, "actions", torch.int32, (T, E, A))
    _need(logits, "logits", torch.float32, (T, E, A, nA))
    _need(reward, "reward", torch.float32, (T, E))
    _need(done, "done", torch.uint8, (T, E))
    _need(obs_last, "obs_last", policy.torch_dtype, (E, A, D))
    tr = _Traj(obs=_ptr(obs), actions=_ptr(actions), logits=_ptr(logits), reward=_ptr(reward), done=_ptr(done),
               obs_last=_ptr(obs_last))
    pc = policy.c()
    _check(lib.rollout_run(ctypes.byref(cfg.c()), ctypes.byref(pc), _ptr(state), t0, T, ctypes.byref(tr),
                           _stream(stream)))


def rollout_run_ac(cfg, policy, state, t0, n_steps, value=None, logp=None, value_last=None, obs=None, actions=None,
                   logits=None, reward=None, done=None, obs_last=None, stream=None):
    """rollout_run for an actor-critic network (last layer: nA logits, then the value); also writes
    value [T, E, A], logp [T, E, A] and value_last [E, A]."""
    E, A = cfg.n_envs, cfg.n_agents
    D, nA = rl_obs_dim(cfg), rl_num_actions(cfg)
    T = n_steps
    _need_state(cfg, state)
    _need(obs, "obs", policy.torch_dtype, (T, E, A, D))
    _need(actions, "actions", torch.int32, (T, E, A))
    _need(logits, "logits", torch.float32, (T, E, A, nA))
    _need(reward, "reward", torch.float32, (T, E))
    _need(done, "done", torch.uint8, (T, E))
    _need(obs_last, "obs_last", policy.torch_dtype, (E, A, D))
    _need(value, "value", torch.float32, (T, E, A))
    _need(logp, "logp", torch.float32, (T, E, A))
    _need(value_last, "value_last", torch.float32, (E, A))
    tr = _Traj(obs=_ptr(obs), actions=_ptr(actions), logits=_ptr(logits), reward=_ptr(reward), done=_ptr(done),
               obs_last=_ptr(obs_last))
    ac = _AcTraj(value=_ptr(value), logp=_ptr(logp), value_last=_ptr(value_last))
    pc = policy.c()
    _check(lib.rollout_run_ac(ctypes.byref(cfg.c()), ctypes.byref(pc), _ptr(state), t0, T, ctypes.byref(tr),
                              ctypes.byref(ac), _stream(stream)))


def rollout_run_teams(cfg, policy, teammates, state, t0, n_steps, obs=None, actions=None, logits=None, reward=None,
                      done=None, obs_last=None, stream=None):
    """rollout_run where agent a of env e acts with heuristic teammates[e, a] (0..8, see HEURISTICS) or,
    for any other value, with the policy."""
    E, A = cfg.n_envs, cfg.n_agents
    D, nA = rl_obs_dim(cfg), rl_num_actions(cfg)
    T = n_steps
    _need(teammates, "teammates", torch.int32, (E, A))
    _need_state(cfg, state)
    _need(obs, "obs", policy.torch_dtype, (T, E, A, D))
    _need(actions, "actions", torch.int32, (T, E, A))
    _need(logits, "logits", torch.float32, (T, E, A, nA))
    _need(reward, "reward", torch.float32, (T, E))
    _need(done, "done", torch.uint8, (T, E))
    _need(obs_last, "obs_last", policy.torch_dtype, (E, A, D))
    tr = _Traj(obs=_ptr(obs), actions=_ptr(actions), logits=_ptr(logits), reward=_ptr(reward), done=_ptr(done),
               obs_last=_ptr(obs_last))
    pc = policy.c()
    _check(lib.rollout_run_teams(ctypes.byref(cfg.c()), ctypes.byref(pc), _ptr(teammates), _ptr(state), t0, T,
                                 ctypes.byref(tr), _stream(stream)))


class S5Policy:
    """Device parameters of the recurrent S5 actor-critic (bfloat16 dense layers, float32 S5).

    ``params``: continuous-time parameters as numpy arrays (keys w_enc, b_enc,
    lam_re, lam_im, log_dt, b_re, b_im, c_re, c_im, d, actor_w, actor_b,
    critic_w, critic_b); lambda_bar and b_bar are made on the device by
    rl_s5_discretize."""

    def __init__(self, params, device="cuda", stream=None):
        bf = lambda a: torch.as_tensor(np.asarray(a, np.float32)).to(device=device, dtype=torch.bfloat16).contiguous()
        f32 = lambda a: torch.as_tensor(np.ascontiguousarray(a, np.float32)).to(device).contiguous()
        self.w_enc, self.b_enc = bf(params["w_enc"]), bf(params["b_enc"])
        self.D, self.H = self.w_enc.shape[1], self.w_enc.shape[0]
        self.P = len(params["lam_re"])
        self.actor_w = [bf(w) for w in params["actor_w"]]
        self.actor_b = [bf(b) for b in params["actor_b"]]
        self.critic_w = [bf(w) for w in params["critic_w"]]
        self.critic_b = [bf(b) for b in params["critic_b"]]
        self.F, self.nA = self.actor_w[0].shape[0], self.actor_w[3].shape[0]
        self.lam = f32(np.stack([params["lam_re"], params["lam_im"]]))
        self.log_dt = f32(params["log_dt"])
        self.b = f32(np.stack([params["b_re"], params["b_im"]]))
        self.c_mat = f32(np.stack([params["c_re"], params["c_im"]]))
        self.d = f32(params["d"])
        self.lambda_bar = torch.empty(2, self.P, device=device)
        self.b_bar = torch.empty(2, self.P, self.H, device=device)
        s5_discretize(self.lam, self.log_dt, self.b, self.lambda_bar, self.b_bar, stream)

    def c(self):
        p = _S5Policy(dtype=RL_BF16, obs_dim=self.D, d_model=self.H, d_state=self.P, head_width=self.F,
                      n_actions=self.nA, w_enc=self.w_enc.data_ptr(), b_enc=self.b_enc.data_ptr(),
                      lambda_bar=self.lambda_bar.data_ptr(), b_bar=self.b_bar.data_ptr(), c=self.c_mat.data_ptr(),
                      d=self.d.data_ptr())
        for l in range(4):
            p.actor_w[l], p.actor_b[l] = self.actor_w[l].data_ptr(), self.actor_b[l].data_ptr()
            p.critic_w[l], p.critic_b[l] = self.critic_w[l].data_ptr(), self.critic_b[l].data_ptr()
        return p


def s5_discretize(lam, log_dt, b, lambda_bar, b_bar, stream=None):
    """Zero-order hold on the device: lam [2, P], log_dt [P], b [2, P, H] -> lambda_bar [2, P], b_bar [2, P, H]."""
    P, H = b.shape[1], b.shape[2]
    _need(lam, "lam", torch.float32, (2, P))
    _need(log_dt, "log_dt", torch.float32, (P,))
    _need(b, "b", torch.float32, (2, P, H))
    _need(lambda_bar, "lambda_bar", torch.float32, (2, P))
    _need(b_bar, "b_bar", torch.float32, (2, P, H))
    _check(lib.rl_s5_discretize(P, H, _ptr(lam), _ptr(log_dt), _ptr(b), _ptr(lambda_bar), _ptr(b_bar),
                                _stream(stream)))


def s5_workspace_bytes(cfg, policy):
    return lib.rl_s5_workspace_bytes(ctypes.byref(cfg.c()), ctypes.byref(policy.c()))


def rollout_run_s5(cfg, policy, state, carry, t0, n_steps, value=None, logp=None, value_last=None, obs=None,
                   actions=None, logits=None, reward=None, done=None, obs_last=None, workspace=None, stream=None):
    """rollout_run_ac with the recurrent S5 actor-critic; ``carry`` [E * A, 2, P] float32 is the S5 state.
    ``workspace``: a uint8 device tensor of at least s5_workspace_bytes(cfg, policy) bytes (allocated when None)."""
    E, A = cfg.n_envs, cfg.n_agents
    D, nA = rl_obs_dim(cfg), rl_num_actions(cfg)
    T = n_steps
    _need_state(cfg, state)
    _need(carry, "carry", torch.float32, (E * A, 2, policy.P))
    _need(obs, "obs", torch.bfloat16, (T, E, A, D))
    _need(actions, "actions", torch.int32, (T, E, A))
    _need(logits, "logits", torch.float32, (T, E, A, nA))
    _need(reward, "reward", torch.float32, (T, E))
    _need(done, "done", torch.uint8, (T, E))
    _need(obs_last, "obs_last", torch.bfloat16, (E, A, D))
    _need(value, "value", torch.float32, (T, E, A))
    _need(logp, "logp", torch.float32, (T, E, A))
    _need(value_last, "value_last", torch.float32, (E, A))
    pc = policy.c()
    nbytes = lib.rl_s5_workspace_bytes(ctypes.byref(cfg.c()), ctypes.byref(pc))
    if workspace is None:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=carry.device)
    tr = _Traj(obs=_ptr(obs), actions=_ptr(actions), logits=_ptr(logits), reward=_ptr(reward), done=_ptr(done),
               obs_last=_ptr(obs_last))
    ac = _AcTraj(value=_ptr(value), logp=_ptr(logp), value_last=_ptr(value_last))
    _check(lib.rollout_run_s5(ctypes.byref(cfg.c()), ctypes.byref(pc), _ptr(state), _ptr(carry), t0, T,
                              ctypes.byref(tr), ctypes.byref(ac), _ptr(workspace), workspace.numel(),
                              _stream(stream)))
    return workspace


def rollout_run_s5_noalloc(cfg, policy, state, carry, t0, n_steps, value=None, logp=None, value_last=None, obs=None,
                           actions=None, logits=None, reward=None, done=None, obs_last=None, stream=None):
    """rollout_run_s5 on the library's built-in device scratch (no workspace, nothing allocated)."""
    E, A = cfg.n_envs, cfg.n_agents
    D, nA = rl_obs_dim(cfg), rl_num_actions(cfg)
    T = n_steps
    _need_state(cfg, state)
    _need(carry, "carry", torch.float32, (E * A, 2, policy.P))
    _need(obs, "obs", torch.bfloat16, (T, E, A, D))
    _need(actions, "actions", torch.int32, (T, E, A))
    _need(logits, "logits", torch.float32, (T, E, A, nA))
    _need(reward, "reward", torch.float32, (T, E))
    _need(done, "done", torch.uint8, (T, E))
    _need(obs_last, "obs_last", torch.bfloat16, (E, A, D))
    _need(value, "value", torch.float32, (T, E, A))
    _need(logp, "logp", torch.float32, (T, E, A))
    _need(value_last, "value_last", torch.float32, (E, A))
    tr = _Traj(obs=_ptr(obs), actions=_ptr(actions), logits=_ptr(logits), reward=_ptr(reward), done=_ptr(done),
               obs_last=_ptr(obs_last))
    ac = _AcTraj(value=_ptr(value), logp=_ptr(logp), value_last=_ptr(value_last))
    _check(lib.rollout_run_s5_noalloc(ctypes.byref(cfg.c()), ctypes.byref(policy.c()), _ptr(state), _ptr(carry), t0,
                                      T, ctypes.byref(tr), ctypes.byref(ac), _stream(stream)))


def gae(reward, done, value, value_last, gamma, lam, adv=None, ret=None, stream=None):
    """Advantages (and returns) [T, E, A] of a stored trajectory; see rl_gae in include/rollout.h."""
    T, E, A = value.shape
    _need(reward, "reward", torch.float32, (T, E))
    _need(done, "done", torch.uint8, (T, E))
    _need(value, "value", torch.float32, (T, E, A))
    _need(value_last, "value_last", torch.float32, (E, A))
    if adv is None:
        adv = torch.empty(T, E, A, device=value.device)
    _need(adv, "adv", torch.float32, (T, E, A))
    _need(ret, "ret", torch.float32, (T, E, A))
    _check(lib.rl_gae(_ptr(reward), _ptr(done), _ptr(value), _ptr(value_last), T, E, A, gamma, lam, _ptr(adv),
                      _ptr(ret), _stream(stream)))
    return adv, ret


def rollout_run_pop(cfg, pop, policy_index, state, t0, n_steps, obs=None, actions=None, logits=None, reward=None,
                    done=None, obs_last=None, stream=None):
    """rollout_run with agent a of env e acting with policy policy_index[e, a] of the population ``pop``."""
    E, A = cfg.n_envs, cfg.n_agents
    D, nA = rl_obs_dim(cfg), rl_num_actions(cfg)
    T = n_steps
    _need(policy_index, "policy_index", torch.int32, (E, A))
    _need_state(cfg, state)
    _need(obs, "obs", pop.torch_dtype, (T, E, A, D))
    _need(actions, "actions", torch.int32, (T, E, A))
    _need(logits, "logits", torch.float32, (T, E, A, nA))
    _need(reward, "reward", torch.float32, (T, E))
    _need(done, "done", torch.uint8, (T, E))
    _need(obs_last, "obs_last", pop.torch_dtype, (E, A, D))
    tr = _Traj(obs=_ptr(obs), actions=_ptr(actions), logits=_ptr(logits), reward=_ptr(reward), done=_ptr(done),
               obs_last=_ptr(obs_last))
    pc = pop.c()
    _check(lib.rollout_run_pop(ctypes.byref(cfg.c()), ctypes.byref(pc), pop.n, _ptr(policy_index), _ptr(state), t0,
                               T, ctypes.byref(tr), _stream(stream)))


def rollout_sample(cfg, t, logits, legal=None, actions=None, stream=None):
    E, A, nA = cfg.n_envs, cfg.n_agents, rl_num_actions(cfg)
    _need(logits, "logits", torch.float32, (E, A, nA))
    _need(legal, "legal", torch.uint8, (E, A, nA))
    if actions is None:
        actions = torch.empty(E, A, dtype=torch.int32, device=logits.device)
    _need(actions, "actions", torch.int32, (E, A))
    _check(lib.rollout_sample(ctypes.byref(cfg.c()), t, _ptr(logits), _ptr(legal), _ptr(actions), _stream(stream)))
    return actions


def rl_gumbel_noise(u, g=None, stream=None):
    _need(u, "u", torch.int32)
    if g is None:
        g = torch.empty(u.shape, dtype=torch.float32, device=u.device)
    _need(g, "g", torch.float32, tuple(u.shape))
    _check(lib.rl_gumbel_noise(_ptr(u), u.numel(), _ptr(g), _stream(stream)))
    return g


# ---- LBF state layout (see the LBF section of include/rollout.h) ----

LBF_FIELDS = ("agent_cell", "agent_level", "food_cell", "food_level", "eaten", "steps", "den")


def lbf_state_planes(cfg, state):
    """Split a state buffer (host or device int32 tensor) into named [.., E] planes."""
    E, A, F = cfg.n_envs, cfg.n_agents, cfg.n_food
    p = state.reshape(2 * A + 2 * F + 3, E)
    return {"agent_cell": p[:A], "agent_level": p[A:2 * A], "food_cell": p[2 * A:2 * A + F],
            "food_level": p[2 * A + F:2 * A + 2 * F], "eaten": p[2 * A + 2 * F], "steps": p[2 * A + 2 * F + 1],
            "den": p[2 * A + 2 * F + 2]}


def lbf_pack_state(cfg, planes, device="cuda"):
    """Inverse of lbf_state_planes: a state buffer from named planes ([A, E], [F, E] or [E])."""
    E, A, F = cfg.n_envs, cfg.n_agents, cfg.n_food
    buf = torch.empty(2 * A + 2 * F + 3, E, dtype=torch.int32)
    v = lbf_state_planes(cfg, buf)
    for k in LBF_FIELDS:
        v[k].copy_(torch.as_tensor(planes[k], dtype=torch.int32).reshape(v[k].shape))
    return buf.reshape(-1).to(device)


# ---- Overcooked state layout (see the Overcooked section of include/rollout.h) ----

OC_MASKS = ("floor", "counter", "onion", "plate", "pot", "serve", "item_onion", "item_plate", "item_soup")
OC_N_PLANES = 32


def oc_state_planes(cfg, state):
    """Split an Overcooked state buffer into named planes: 45-bit cell masks as
    int64 [E] (from their lo/hi words), and int32 [E] / [2, E] fields."""
    E = cfg.n_envs
    p = state.reshape(OC_N_PLANES, E)
    out = {}
    for i, k in enumerate(OC_MASKS):
        lo = p[2 * i].to(torch.int64) & 0xFFFFFFFF
        hi = p[2 * i + 1].to(torch.int64) & 0xFFFFFFFF
        out[k] = lo | (hi << 32)
    out["W"] = p[18] & 0xFF
    out["H"] = (p[18] >> 8) & 0xFF
    out["agent_cell"], out["facing"], out["held"] = p[19:21], p[21:23], p[23:25]
    out["pot_cell"], out["pot_onions"], out["pot_timer"] = p[25:27], p[27:29], p[29:31]
    out["steps"] = p[31]
    return out


def oc_pack_state(cfg, planes, device="cuda"):
    """Inverse of oc_state_planes: a state buffer from named planes."""
    E = cfg.n_envs
    buf = torch.empty(OC_N_PLANES, E, dtype=torch.int32)
    for i, k in enumerate(OC_MASKS):
        m = torch.as_tensor(planes[k], dtype=torch.int64).reshape(E)
        buf[2 * i] = (((m & 0xFFFFFFFF) ^ 0x80000000) - 0x80000000).to(torch.int32)  # low word as signed int32
        buf[2 * i + 1] = (m >> 32).to(torch.int32)
    buf[18] = (torch.as_tensor(planes["W"]) | (torch.as_tensor(planes["H"]) << 8)).to(torch.int32).reshape(E)
    for lo, k in ((19, "agent_cell"), (21, "facing"), (23, "held"), (25, "pot_cell"), (27, "pot_onions"),
                  (29, "pot_timer")):
        buf[lo:lo + 2] = torch.as_tensor(planes[k], dtype=torch.int32).reshape(2, E)
    buf[31] = torch.as_tensor(planes["steps"], dtype=torch.int32).reshape(E)
    return buf.reshape(-1).to(device)


# ---- Hanabi state layout (see the Hanabi section of include/rollout.h) ----

HN_N_PLANES = 35
HN_FIELDS = {"hand": (13, 2), "n": (15, 2), "kc": (17, 2), "kr": (19, 2), "hc": (21, 2), "hr": (23, 2),
             "fw": (25, 1), "disc0": (26, 1), "disc1": (27, 1), "info": (28, 1), "lives": (29, 1), "cur": (30, 1),
             "turns_left": (31, 1), "next": (32, 1), "steps": (33, 1), "last": (34, 1)}


def hn_state_planes(cfg, state):
    """Split a Hanabi state buffer into named int32 planes: "deck" [13, E] and the packed fields."""
    p = state.reshape(HN_N_PLANES, cfg.n_envs)
    out = {"deck": p[0:13]}
    for k, (lo, n) in HN_FIELDS.items():
        out[k] = p[lo:lo + n] if n > 1 else p[lo]
    return out


def hn_pack_state(cfg, planes, device="cuda"):
    """Inverse of hn_state_planes."""
    E = cfg.n_envs
    buf = torch.empty(HN_N_PLANES, E, dtype=torch.int32)
    buf[0:13] = torch.as_tensor(planes["deck"], dtype=torch.int64).reshape(13, E).to(torch.int32)
    for k, (lo, n) in HN_FIELDS.items():
        v = torch.as_tensor(planes[k], dtype=torch.int64).reshape(n, E)
        buf[lo:lo + n] = (((v & 0xFFFFFFFF) ^ 0x80000000) - 0x80000000).to(torch.int32)
    return buf.reshape(-1).to(device)
