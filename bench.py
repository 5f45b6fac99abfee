"""Throughput of the batched multi-agent rollout on one MI355X.

One step = one ``rollout_run`` over the whole batch: 4096 Level-Based
Foraging envs (8x8 grid, 2 agents, 3 foods) x 128 steps, every agent's MLP
(192-128-128-6) forward, Gumbel-max sampling, env step and auto-reset, with
the trajectory (observations, actions, rewards, dones, final observation)
written to HBM.  The headline is bf16; the same workload in float32, the
env-only stepping kernel and the standalone policy forward are reported
alongside.  Inputs (weights, initial states) are seeded synthetic data that
is resident in HBM before the timed region starts.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
Prints one JSON line.
"""

import argparse
import glob
import hashlib
import re
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "agent-env steps/sec incl. policy forward (1 MI355X) at 4096 envs; % HBM/MFMA peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
WORKLOAD = "lbf8_4096"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-leg", nargs=5, default=None, metavar=("WORKLOAD", "ENV0", "N_ENVS", "DTYPE", "CORE"),
                    help="(internal) run one timed oracle leg in this process and print its result")
    ap.add_argument("--cpu-only", action="store_true", help="only the CPU baseline (no GPU work)")
    ap.add_argument("--only", choices=["run_bf16", "run_f32", "env_bf16", "env_f32", "policy_bf16", "policy_f32",
                                       "copy"], default=None,
                    help="time one kernel only (for profiler runs); 'copy' runs a plain 512 MiB device copy, "
                         "the reference for scaling HBM byte counters")
    ap.add_argument("--workload-only", default=None,
                    help="time one secondary workload only (lbf12_16k, oc_4096, hn_4096; for profiler runs)")
    ap.add_argument("--no-workloads", action="store_true", help="skip the secondary workloads")
    ap.add_argument("--counter-plan", action="store_true",
                    help="print the rocprofv3 counter passes (one command per line) and exit")
    ap.add_argument("--phases", action="store_true",
                    help="per-phase cycles of the fused and env-only kernels' step loops from the phase-stamped "
                         "library (python -m paper_2609_13716_amd.build --stamps); writes "
                         "profiles/phase_stamps.md")
    ap.add_argument("--phases-child", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--summarize-counters", metavar="DIR", default=None,
                    help="read the counter CSVs of the passes under DIR and write profiles/traffic.json and "
                         "profiles/counters_all_workloads.md (no GPU needed)")
    return ap.parse_args()


def csrc_hash():
    """Hash of every kernel source (comments removed) and of the workload definitions: hardware counters
    taken on the benchmark's kernels stay valid while their code is unchanged."""
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2609_13716_amd", "csrc", "*")))
    files.append(os.path.join(ROOT, "paper_2609_13716_amd", "workloads.py"))
    for f in files:
        h.update(os.path.basename(f).encode())
        text = open(f, encoding="utf-8").read()
        if not f.endswith(".py"):  # C++/HIP: drop // and /* */ comments, then blank lines
            text = re.sub(r"/\*.*?\*/|//[^\n]*", "", text, flags=re.S)
            text = "\n".join(line.rstrip() for line in text.splitlines() if line.strip())
        h.update(text.encode())
    return h.hexdigest()[:16]


def timed(fn, steps, warmup):
    """Run fn warmup times, then `steps` times; returns (mean kernel ms from events, wall ms per step)."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    t0 = time.perf_counter()
    for a, b in evs:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    kern = sum(a.elapsed_time(b) for a, b in evs) / steps
    return kern, wall


def roofline(bound, achieved, peak, unit, traffic=None):
    return {"bound": bound, "achieved": round(achieved, 3), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": traffic}


def load_traffic(key):
    """HBM bytes per launch of one benchmark leg's kernels ("leg:role") from the committed rocprofv3 counter
    summary, if that summary was taken on these kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except ValueError:
        return None
    if rec.get("csrc_hash") != csrc_hash():
        return None
    k = rec.get("legs", {}).get(key)
    return None if k is None else k.get("hbm_bytes_per_launch")


def run_bytes(E, T, A, D, es, state_bytes, per_agent_extra=0):
    """Algorithmic HBM bytes of one rollout_run launch: the trajectory (observations, actions, reward,
    done, plus per_agent_extra bytes per agent-step) and the state read and written once."""
    return E * T * (A * D * es + A * 4 + 4 + 1 + A * per_agent_extra) + 2 * state_bytes


def env_bytes(E, T, A, D, es, state_bytes):
    """Algorithmic HBM bytes of one env-only rollout_step launch: actions read, observations, reward and
    done written, the state read and written once."""
    return E * T * (A * 4 + A * D * es + 4 + 1) + 2 * state_bytes


def env_config(R, workloads, name, n_envs=None, seed=0):
    w = workloads.WORKLOADS[name]
    E = w["n_envs"] if n_envs is None else n_envs
    kind = workloads.kind(name)
    if kind == "overcooked":
        return R.overcooked_config(E, seed=seed, **w["env"])
    if kind == "hanabi":
        return R.hanabi_config(E, seed=seed, **w["env"])
    return R.EnvConfig(n_envs=E, seed=seed, **w["env"])


def measure_workload(R, workloads, name, dt, steps, warmup):
    """rollout_run and rollout_step of one workload at full size: times, throughput and rooflines."""
    import torch
    w = workloads.WORKLOADS[name]
    cfg = env_config(R, workloads, name)
    E, T, A = cfg.n_envs, w["n_steps"], cfg.n_agents
    D, nA = R.rl_obs_dim(cfg), R.rl_num_actions(cfg)
    dims = workloads.policy_dims(name)
    ws, bs = workloads.policy_weights(dims, seed=1000)
    pol = R.Policy(ws, bs, dt)
    es = 2 if dt == "bf16" else 4
    acting = 1 if workloads.kind(name) == "hanabi" else A  # Hanabi: only the mover's row affects an action
    flop_per_row = 2 * sum(dims[i] * dims[i + 1] for i in range(3))
    state_bytes = R.rl_state_bytes(cfg)
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    obs = torch.empty(T, E, A, D, dtype=pol.torch_dtype, device="cuda")
    acts = torch.empty(T, E, A, dtype=torch.int32, device="cuda")
    rew = torch.empty(T, E, device="cuda")
    done = torch.empty(T, E, dtype=torch.uint8, device="cuda")
    t_next = [0]

    tm = None
    if w.get("teammates"):  # agent 0 the policy, agent 1 heuristic kind e mod 11 (every Greedy and Sequential kind)
        tm = torch.full((E, A), -1, dtype=torch.int32)
        tm[:, 1] = torch.arange(E, dtype=torch.int32) % len(R.HEURISTICS)
        tm = tm.cuda()

    def run():
        if tm is None:
            R.rollout_run(cfg, pol, state, t_next[0], T, obs=obs, actions=acts, reward=rew, done=done)
        else:
            R.rollout_run_teams(cfg, pol, tm, state, t_next[0], T, obs=obs, actions=acts, reward=rew, done=done)
        t_next[0] += T

    kern_ms, wall_ms = timed(run, steps, warmup)
    nbytes = run_bytes(E, T, A, D, es, state_bytes)
    flops = E * T * acting * flop_per_row
    traffic = load_traffic(f"{name}:run")
    out = {"workload": name, "dtype": dt, "n_envs": E, "steps_per_rollout": T, "policy": "-".join(map(str, dims)),
           "value": round(E * T * acting / (wall_ms * 1e-3), 1), "unit": "agent-env steps/s",
           "env_steps_per_s": round(E * T / (wall_ms * 1e-3), 1), "ms_per_step": round(wall_ms, 4),
           "kernel_ms": round(kern_ms, 4),
           "roofline_hbm": roofline("hbm", nbytes / (kern_ms * 1e-3) / 1e9, HBM_PEAK_GBS, "GB/s", traffic),
           "roofline_mfma": roofline("mfma", flops / (kern_ms * 1e-3) / 1e12, MFMA_PEAK_TFLOPS[dt], "TFLOP/s",
                                     traffic)}
    # env-only stepping with injected uniform actions (illegal ones fall back to the lowest legal action)
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    inj = torch.randint(0, nA, (T, E, A), dtype=torch.int32, device="cuda", generator=g)
    R.rollout_init(cfg, state)
    t_next[0] = 0

    def env():
        R.rollout_step(cfg, state, t_next[0], inj, obs, rew, done)
        t_next[0] += T

    kern_ms, wall_ms = timed(env, steps, warmup)
    nbytes = env_bytes(E, T, A, D, es, state_bytes)
    out["env_only"] = {"env_steps_per_s": round(E * T / (wall_ms * 1e-3), 1), "kernel_ms": round(kern_ms, 4),
                       "roofline": roofline("hbm", nbytes / (kern_ms * 1e-3) / 1e9, HBM_PEAK_GBS, "GB/s",
                                            load_traffic(f"{name}:env"))}
    del obs
    # standalone policy forward over a batch of this workload's observations
    rows = min(E * A * T, 1 << 18)
    g.manual_seed(8)
    x = torch.randint(0, 3, (rows, D), device="cuda", generator=g).to(pol.torch_dtype)
    lg = torch.empty(rows, nA, device="cuda")
    kern_ms, _ = timed(lambda: R.policy_forward(pol, x, logits=lg), steps, warmup)
    out["policy_forward"] = {"rows": rows, "kernel_ms": round(kern_ms, 4),
                             "roofline": roofline("mfma", rows * flop_per_row / (kern_ms * 1e-3) / 1e12,
                                                  MFMA_PEAK_TFLOPS[dt], "TFLOP/s", load_traffic(f"{name}:policy"))}
    del x, lg
    torch.cuda.empty_cache()
    return out


def measure_population(R, workloads, name, dt, steps, warmup):
    """rollout_run_pop of a population workload at full size: time, throughput and rooflines."""
    import torch
    w = workloads.WORKLOADS[name]
    cfg = env_config(R, workloads, name)
    E, T, A = cfg.n_envs, w["n_steps"], cfg.n_agents
    D = R.rl_obs_dim(cfg)
    dims = workloads.policy_dims(name)
    ws, bs = workloads.population_weights(name, seed=1000)
    pop = R.Population(ws, bs, dt)
    idx = torch.as_tensor(workloads.population_index(name)).cuda()
    es = 2 if dt == "bf16" else 4
    flop_per_row = 2 * sum(dims[i] * dims[i + 1] for i in range(3))
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    obs = torch.empty(T, E, A, D, dtype=pop.torch_dtype, device="cuda")
    acts = torch.empty(T, E, A, dtype=torch.int32, device="cuda")
    rew = torch.empty(T, E, device="cuda")
    done = torch.empty(T, E, dtype=torch.uint8, device="cuda")
    t_next = [0]

    def run():
        R.rollout_run_pop(cfg, pop, idx, state, t_next[0], T, obs=obs, actions=acts, reward=rew, done=done)
        t_next[0] += T

    kern_ms, wall_ms = timed(run, steps, warmup)
    nbytes = run_bytes(E, T, A, D, es, R.rl_state_bytes(cfg))
    flops = E * T * A * flop_per_row
    traffic = load_traffic(f"{name}:run")
    n_teammates = w["population"] - 1
    return {"workload": name, "dtype": dt, "n_envs": E, "steps_per_rollout": T, "policy": "-".join(map(str, dims)),
            "population": w["population"], "assignment": f"agent 0: ego; agent 1: one of {n_teammates} teammates "
                                                          f"per block of {E // n_teammates} envs",
            "value": round(E * T * A / (wall_ms * 1e-3), 1), "unit": "agent-env steps/s",
            "ms_per_step": round(wall_ms, 4), "kernel_ms": round(kern_ms, 4),
            "roofline_hbm": roofline("hbm", nbytes / (kern_ms * 1e-3) / 1e9, HBM_PEAK_GBS, "GB/s", traffic),
            "roofline_mfma": roofline("mfma", flops / (kern_ms * 1e-3) / 1e12, MFMA_PEAK_TFLOPS[dt], "TFLOP/s",
                                      traffic)}


def measure_actor_critic(R, workloads, name, dt, steps, warmup):
    """rollout_run_ac then rl_gae of an actor-critic workload at full size: times, throughput and rooflines."""
    import torch
    w = workloads.WORKLOADS[name]
    cfg = env_config(R, workloads, name)
    E, T, A = cfg.n_envs, w["n_steps"], cfg.n_agents
    D, nA = R.rl_obs_dim(cfg), R.rl_num_actions(cfg)
    dims = workloads.policy_dims(name)
    ws, bs = workloads.policy_weights(dims, seed=1000)
    pol = R.Policy(ws, bs, dt)
    es = 2 if dt == "bf16" else 4
    flop_per_row = 2 * sum(dims[i] * dims[i + 1] for i in range(3))
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    f = dict(device="cuda")
    obs = torch.empty(T, E, A, D, dtype=pol.torch_dtype, **f)
    acts = torch.empty(T, E, A, dtype=torch.int32, **f)
    rew, done = torch.empty(T, E, **f), torch.empty(T, E, dtype=torch.uint8, **f)
    value, logp, vlast = torch.empty(T, E, A, **f), torch.empty(T, E, A, **f), torch.empty(E, A, **f)
    adv, ret = torch.empty(T, E, A, **f), torch.empty(T, E, A, **f)
    t_next = [0]

    def run():
        R.rollout_run_ac(cfg, pol, state, t_next[0], T, value=value, logp=logp, value_last=vlast, obs=obs,
                         actions=acts, reward=rew, done=done)
        t_next[0] += T

    kern_ms, wall_ms = timed(run, steps, warmup)
    nbytes = run_bytes(E, T, A, D, es, R.rl_state_bytes(cfg), per_agent_extra=8) + E * A * 4
    flops = E * T * A * flop_per_row
    traffic = load_traffic(f"{name}:run")
    gae_ms, _ = timed(lambda: R.gae(rew, done, value, vlast, w["gamma"], w["lam"], adv=adv, ret=ret), steps, warmup)
    gae_bytes = gae_alg_bytes(E, T, A)
    return {"workload": name, "dtype": dt, "n_envs": E, "steps_per_rollout": T, "policy": "-".join(map(str, dims)),
            "value": round(E * T * A / (wall_ms * 1e-3), 1), "unit": "agent-env steps/s",
            "ms_per_step": round(wall_ms, 4), "kernel_ms": round(kern_ms, 4),
            "roofline_hbm": roofline("hbm", nbytes / (kern_ms * 1e-3) / 1e9, HBM_PEAK_GBS, "GB/s", traffic),
            "roofline_mfma": roofline("mfma", flops / (kern_ms * 1e-3) / 1e12, MFMA_PEAK_TFLOPS[dt], "TFLOP/s",
                                      traffic),
            "gae": {"kernel_ms": round(gae_ms, 4),
                    "roofline": roofline("hbm", gae_bytes / (gae_ms * 1e-3) / 1e9, HBM_PEAK_GBS, "GB/s",
                                         load_traffic(f"{name}:gae"))}}


def gae_alg_bytes(E, T, A):
    """Algorithmic HBM bytes of one GAE launch: reward and done read, values read, advantages and returns
    written, the bootstrap values read."""
    return T * E * (4 + 1) + T * E * A * (4 + 8) + E * A * 4


def measure_s5(R, workloads, name, dt, steps, warmup):
    """rollout_run_s5 (recurrent S5 actor-critic) at full size: time, throughput, dense-layer MFMA rate."""
    import torch
    w = workloads.WORKLOADS[name]
    cfg = env_config(R, workloads, name)
    E, T, A = cfg.n_envs, w["n_steps"], cfg.n_agents
    D, nA = R.rl_obs_dim(cfg), R.rl_num_actions(cfg)
    H, P, F = w["s5"]["d_model"], w["s5"]["d_state"], w["s5"]["head_width"]
    pol = R.S5Policy(workloads.s5_params(D, H, P, F, nA, seed=1000))
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    f = dict(device="cuda")
    carry = torch.zeros(E * A, 2, P, **f)
    obs = torch.empty(T, E, A, D, dtype=torch.bfloat16, **f)
    acts = torch.empty(T, E, A, dtype=torch.int32, **f)
    rew, done = torch.empty(T, E, **f), torch.empty(T, E, dtype=torch.uint8, **f)
    value, logp, vlast = torch.empty(T, E, A, **f), torch.empty(T, E, A, **f), torch.empty(E, A, **f)
    wsp = torch.empty(R.s5_workspace_bytes(cfg, pol), dtype=torch.uint8, **f)
    t_next = [0]

    def run():
        R.rollout_run_s5(cfg, pol, state, carry, t_next[0], T, value=value, logp=logp, value_last=vlast, obs=obs,
                         actions=acts, reward=rew, done=done, workspace=wsp)
        t_next[0] += T

    kern_ms, wall_ms = timed(run, steps, warmup)
    head_macs = 2 * (H * F + 2 * F * F) + F * (nA + 1)
    macs_per_row = D * H + 4 * P * H + head_macs  # encoder, B_bar u and Re(C x) as real products, heads
    rows = E * A * (T + 1)  # T steps plus the value of the final observation
    return {"workload": name, "dtype": dt, "n_envs": E, "steps_per_rollout": T,
            "policy": f"S5 D{D}-H{H}-P{P}, heads 3x{F}", "value": round(E * T * A / (wall_ms * 1e-3), 1),
            "unit": "agent-env steps/s", "ms_per_step": round(wall_ms, 4), "kernel_ms": round(kern_ms, 4),
            "roofline_mfma": roofline("mfma", 2 * macs_per_row * rows / (kern_ms * 1e-3) / 1e12,
                                      MFMA_PEAK_TFLOPS[dt], "TFLOP/s", load_traffic(f"{name}:run")),
            "note": "MFMA rate over the whole rollout (every kernel of every step); per-kernel times in the "
                    "rocprofv3 summary of this workload"}


# ---------------------------------------------------------------- hardware counters
# Each counter pass is its own rocprofv3 process over one benchmark leg (bench.py with the leg's arguments,
# two timed launches after one warm-up, so every kernel of the leg is dispatched COUNTER_CALLS times); one
# pass asks for no more counters of a hardware block than one run can collect.
COUNTER_PASSES = {
    "fetch": ("FETCH_SIZE",),
    "write": ("WRITE_SIZE",),
    "mfma": ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CU_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_BF16",
             "SQ_INSTS_VALU_MFMA_MOPS_F32", "GRBM_GUI_ACTIVE"),
    "l1": ("TCP_TCC_READ_REQ_sum", "TCP_TCC_WRITE_REQ_sum", "TCP_TOTAL_CACHE_ACCESSES_sum", "GRBM_GUI_ACTIVE"),
}
COUNTER_CALLS = 3
_SECONDARY = ("lbf12_16k", "oc_4096", "hn_4096", "hn_mini_4096", "lbf7_const_4096", "lbf7_teams_4096",
              "lbf8_4096_ac", "lbf8_4096_pop", "lbf8_4096_s5")
COUNTER_LEGS = (
    ("lbf8_4096_run_bf16", "--only run_bf16", ("fetch", "write", "mfma", "l1")),
    ("lbf8_4096_env_bf16", "--only env_bf16", ("fetch", "write")),
    ("lbf8_4096_policy_bf16", "--only policy_bf16", ("fetch", "write", "mfma")),
    ("lbf8_4096_run_f32", "--only run_f32", ("fetch", "write", "mfma")),
    ("lbf8_4096_env_f32", "--only env_f32", ("fetch", "write")),
    ("lbf8_4096_policy_f32", "--only policy_f32", ("fetch", "write", "mfma")),
) + tuple((n, f"--workload-only {n}", ("fetch", "write", "mfma") + (("l1",) if n in ("hn_4096", "oc_4096") else ()))
          for n in _SECONDARY) + (("copy", "--only copy", ("fetch", "write")),)


def counter_commands(out_dir="gpurun_out/pmc"):
    """(pass, leg, command) of every counter pass, each to be run alone from the repository root."""
    cmds = []
    for leg, args, passes in COUNTER_LEGS:
        for ps in passes:
            steps = "" if leg == "copy" else " --steps 2 --warmup 1 --no-cpu-baseline"
            cmds.append((ps, leg, f"rocprofv3 --pmc {' '.join(COUNTER_PASSES[ps])} -d {out_dir}/{ps}/{leg} -o run "
                                  f"--output-format csv -- python3 bench.py {args}{steps}"))
    return cmds


def kernel_role(name):
    """Which benchmarked call a kernel belongs to: 'run', 'env', 'policy', 'gae', 'copy' or None (init
    kernels and the input generators)."""
    if "policy_fwd" in name or "policy_forward" in name:
        return "policy"
    if "_env_kernel" in name or "_env3_kernel" in name:
        return "env"
    if "gae" in name:
        return "gae"
    if any(k in name for k in ("lbf_rollout_kernel", "_run_kernel", "_run_pop_kernel", "_pop2_kernel", "s5_")):
        return "run"
    if "copyBuffer" in name:
        return "copy"
    return None


def _read_counter_csv(d):
    """{dispatch id: (kernel name, {counter: value})} from the counter CSV under directory d."""
    import csv
    paths = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    out = {}
    for path in paths:
        for r in csv.DictReader(open(path)):
            rec = out.setdefault((path, r["Dispatch_Id"]), (r["Kernel_Name"], {}))
            rec[1][r["Counter_Name"]] = rec[1].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return out


def _algorithmic(R, workloads, leg, role):
    """(algorithmic bytes, algorithmic flop) of one launch of a leg's call, by the formulas of the timed legs
    (None where the leg has no such figure)."""
    name = "lbf8_4096" if leg.startswith("lbf8_4096_") and leg.split("_")[2] in ("run", "env", "policy") else leg
    dt = leg.rsplit("_", 1)[1] if name != leg else "bf16"
    if name not in workloads.WORKLOADS:
        return None, None
    w = workloads.WORKLOADS[name]
    cfg = env_config(R, workloads, name)
    E, T, A = cfg.n_envs, w["n_steps"], cfg.n_agents
    D, nA = R.rl_obs_dim(cfg), R.rl_num_actions(cfg)
    es = 2 if dt == "bf16" else 4
    sb = R.rl_state_bytes(cfg)
    if "s5" in w:
        return None, None
    dims = workloads.policy_dims(name)
    fpr = 2 * sum(dims[i] * dims[i + 1] for i in range(3))
    acting = 1 if workloads.kind(name) == "hanabi" else A
    if role == "run":
        b = run_bytes(E, T, A, D, es, sb, per_agent_extra=8 if w.get("value_head") else 0)
        b += E * A * D * es if name != leg else (E * A * 4 if w.get("value_head") else 0)
        return b, E * T * acting * fpr
    if role == "env":
        return env_bytes(E, T, A, D, es, sb), None
    if role == "policy":
        rows = E * A * T if name != leg else min(E * A * T, 1 << 18)
        return rows * (D * es + nA * 4), rows * fpr
    if role == "gae":
        return gae_alg_bytes(E, T, A), None
    return None, None


def summarize_counters(src):
    """Write profiles/traffic.json (HBM bytes per launch of every leg's calls, FETCH_SIZE and WRITE_SIZE
    scaled by what each reads on a plain 512 MiB device copy) and profiles/counters_all_workloads.md."""
    import statistics

    from paper_2609_13716_amd import rollout as R
    from paper_2609_13716_amd import workloads
    n_copy = 512 << 20
    scale = {}
    for ps, ctr in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
        d = _read_counter_csv(os.path.join(src, ps, "copy"))
        vals = [c[ctr] for k, c in d.values() if kernel_role(k) == "copy" and c[ctr] > 1024]  # the 512 MiB copies
        scale[ctr] = n_copy / (statistics.mean(vals) * 1024)
    legs, rows = {}, []
    for leg, _, passes in COUNTER_LEGS:
        if leg == "copy":
            continue
        one_call = "s5" in workloads.WORKLOADS.get(leg, {})  # the S5 leg times one call (its env steps included)
        per_role = {}
        for ps in passes:
            for k, c in _read_counter_csv(os.path.join(src, ps, leg)).values():
                role = kernel_role(k)
                if role is None or role == "copy":  # (device copies outside the copy leg are set-up)
                    continue
                if one_call:
                    role = "run"
                rr = per_role.setdefault(role, {"kernels": set(), "sum": {}})
                rr["kernels"].add(k.split("(")[0].replace("void ", "").replace("rl::", ""))
                for ctr, v in c.items():
                    rr["sum"][ctr] = rr["sum"].get(ctr, 0.0) + v
        for role, rr in sorted(per_role.items()):
            sm = {k: v / COUNTER_CALLS for k, v in rr["sum"].items()}
            rec = {"kernels": sorted(rr["kernels"])}
            if "FETCH_SIZE" in sm and "WRITE_SIZE" in sm:
                rb = sm["FETCH_SIZE"] * 1024 * scale["FETCH_SIZE"]
                wb = sm["WRITE_SIZE"] * 1024 * scale["WRITE_SIZE"]
                rec.update(read_bytes=round(rb), write_bytes=round(wb), hbm_bytes_per_launch=round(rb + wb))
            alg_b, alg_f = _algorithmic(R, workloads, leg, role)
            if alg_b:
                rec["algorithmic_bytes_per_launch"] = alg_b
            if "SQ_VALU_MFMA_BUSY_CYCLES" in sm and sm.get("GRBM_GUI_ACTIVE"):
                simd_cycles = 256 * 4 * sm["GRBM_GUI_ACTIVE"] / 8  # GRBM_GUI_ACTIVE is summed over the 8 XCDs
                rec["mfma_busy_frac"] = round(sm["SQ_VALU_MFMA_BUSY_CYCLES"] / simd_cycles, 4)
                mops = sm.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) + sm.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0)
                rec["mfma_flop_per_launch"] = round(512 * mops)
                if alg_f:
                    rec["algorithmic_flop_per_launch"] = alg_f
            if "TCP_TCC_READ_REQ_sum" in sm:
                rec["l2_to_l1_read_req_per_launch"] = round(sm["TCP_TCC_READ_REQ_sum"])
                rec["l1_to_l2_write_req_per_launch"] = round(sm.get("TCP_TCC_WRITE_REQ_sum", 0.0))
                rec["l1_tag_accesses_per_launch"] = round(sm.get("TCP_TOTAL_CACHE_ACCESSES_sum", 0.0))
            legs[f"{leg}:{role}"] = rec
            rows.append((leg, role, rec))
    cmds = counter_commands()
    out = {"csrc_hash": csrc_hash(),
           "note": "per launch of each benchmark leg's call: HBM bytes from rocprofv3 FETCH_SIZE / WRITE_SIZE "
                   "(KiB per dispatch, summed over the call's kernels) scaled by the factor that maps the same "
                   "counter on a plain 512 MiB device copy to 512 MiB; MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / "
                   "(1024 SIMDs x GRBM_GUI_ACTIVE / 8 XCDs); MFMA flop = 512 x SQ_INSTS_VALU_MFMA_MOPS",
           "scale": {k: round(v, 5) for k, v in scale.items()},
           "commands": [c for _, _, c in cmds], "legs": legs}
    json.dump(out, open(os.path.join(ROOT, "profiles", "traffic.json"), "w"), indent=1)
    md = ["# Hardware counters of every benchmarked kernel, one MI355X", "",
          "Each pass is its own process, run from the repository root after `cd /tmp && export TMPDIR=/tmp`; "
          "this summary is written by `python3 bench.py --summarize-counters gpurun_out/pmc` from their CSVs.", "",
          "```"] + [c for _, _, c in cmds] + ["```", "",
          f"Copy calibration (512 MiB device copy): FETCH_SIZE x {scale['FETCH_SIZE']:.4f}, "
          f"WRITE_SIZE x {scale['WRITE_SIZE']:.4f} (KiB to bytes).", "",
          "Per launch of the leg's call (its kernels summed; the policy leg of a workload is its standalone "
          "policy_forward over the first 2^18 rows).  MFMA busy: fraction of SIMD-cycles with the matrix "
          "unit busy; MFMA Gflop: 512 x SQ_INSTS_VALU_MFMA_MOPS (padding included) against the algorithmic "
          "flop.", "",
          "| leg | call | kernels | HBM MB (read + write) | algorithmic MB | ratio | MFMA busy | MFMA Gflop (alg.) "
          "| L2->L1 read req (M) |", "|---|---|---|---|---|---|---|---|---|"]
    for leg, role, r in rows:
        hb = r.get("hbm_bytes_per_launch")
        ab = r.get("algorithmic_bytes_per_launch")
        hbm = f"{hb / 1e6:,.1f} ({r['read_bytes'] / 1e6:,.1f} + {r['write_bytes'] / 1e6:,.1f})" if hb else "-"
        ratio = f"{hb / ab:.3f}" if hb and ab else "-"
        mf = f"{100 * r['mfma_busy_frac']:.1f}%" if r.get("mfma_flop_per_launch") else "-"
        fl = (f"{r['mfma_flop_per_launch'] / 1e9:,.1f} ({r['algorithmic_flop_per_launch'] / 1e9:,.1f})"
              if "algorithmic_flop_per_launch" in r else
              f"{r['mfma_flop_per_launch'] / 1e9:,.1f}" if r.get("mfma_flop_per_launch") else "-")
        l1 = f"{r['l2_to_l1_read_req_per_launch'] / 1e6:,.2f}" if "l2_to_l1_read_req_per_launch" in r else "-"
        ks = "<br>".join(f"`{k}`" for k in r["kernels"][:3]) + (" ..." if len(r["kernels"]) > 3 else "")
        abs_ = f"{ab / 1e6:,.1f}" if ab else "-"
        md.append(f"| {leg} | {role} | {ks} | {hbm} | {abs_} | {ratio} | {mf} | {fl} | {l1} |")
    open(os.path.join(ROOT, "profiles", "counters_all_workloads.md"), "w").write("\n".join(md) + "\n")
    return out


# ---------------------------------------------------------------- phase stamps
# (case, workload, call, stamp unit, iterations per launch beyond n_steps, role names, phase names)
PHASE_CASES = (
    ("headline fused rollout", "lbf8_4096", "run", "lbf", 0, ("env wave", "other waves"),
     {0: "barrier at the step's top", 1: "action Philox draws (one step in 16)", 2: "layer 1 + barrier",
      3: "layer 2 + barrier", 4: "layer 3 + Gumbel argmax", 5: "transition", 6: "resets",
      7: "paint o_t+1, reward/done stores", 8: "copy o_t to the trajectory", 9: "Gumbel noise of step t+1"}),
    ("12x12 fused rollout", "lbf12_16k", "run", "lbf", 0, ("env wave", "other waves"), None),
    ("Hanabi env-only", "hn_4096", "env", "hn", 2, ("env wave", "observation waves"),
     {0: "move (transition, reward/done)", 1: "re-deals (wave shuffles)", 2: "publish snapshot",
      4: "field passes (bit vectors)", 5: "legal masks", 6: "write out + clear rows", 7: "barrier wait"}),
    ("kitchen fused rollout", "oc_4096", "run", "oc", 0, ("env wave", "other waves"),
     {0: "barrier at the step's top", 1: "layer 1", 2: "layer 2", 3: "layer 3", 4: "Gumbel scores",
      5: "copy o_t to the trajectory (other waves)", 6: "barrier", 7: "argmax + barrier",
      8: "transition (env lanes)", 9: "barrier",
      10: "repaint o_t+1 (env lanes) / next step's noise (other waves; with no trajectory copy it is drawn during "
          "the transition)"}),
    ("Hanabi fused rollout", "hn_4096", "run", "hn", 0, ("all waves",),
     {0: "barrier at the step's top", 1: "observation bit vectors", 2: "paint layer-1 tile", 3: "layer 1",
      4: "layer 2", 5: "layer 3", 6: "legal mask + Gumbel scores", 7: "copy o_t to the trajectory",
      8: "argmax + transition", 9: "re-deals"}),
)


def phases_child():
    """(run with RL_LIB_PATH = the stamped library) one launch per case; prints the stamp tables as JSON."""
    import ctypes

    import torch

    from paper_2609_13716_amd import rollout as R
    from paper_2609_13716_amd import workloads
    out = []
    for case, name, call, unit, extra, _, _ in PHASE_CASES:
        w = workloads.WORKLOADS[name]
        cfg = env_config(R, workloads, name)
        E, T, A = cfg.n_envs, w["n_steps"], cfg.n_agents
        D, nA = R.rl_obs_dim(cfg), R.rl_num_actions(cfg)
        pol = R.Policy(*workloads.policy_weights(workloads.policy_dims(name), seed=1000), "bf16")
        state = R.new_state(cfg)
        R.rollout_init(cfg, state)
        obs = torch.empty(T, E, A, D, dtype=torch.bfloat16, device="cuda")
        rew, done = torch.empty(T, E, device="cuda"), torch.empty(T, E, dtype=torch.uint8, device="cuda")
        g = torch.Generator(device="cuda")
        g.manual_seed(7)
        inj = torch.randint(0, nA, (T, E, A), dtype=torch.int32, device="cuda", generator=g)
        reader = getattr(R.lib, f"rl_phase_stamps_{unit}")
        table = (ctypes.c_ulonglong * (8 * 12))()

        def launch(t0):
            if call == "run":
                R.rollout_run(cfg, pol, state, t0, T, obs=obs, reward=rew, done=done)
            else:
                R.rollout_step(cfg, state, t0, inj, obs, rew, done)
        launch(0)
        torch.cuda.synchronize()
        reader(table, 1)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        launch(T)
        b.record()
        torch.cuda.synchronize()
        reader(table, 1)
        out.append({"case": case, "iterations": T + extra, "ms": a.elapsed_time(b), "table": list(table)})
        del obs
        torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)


def phases():
    """Run phases_child on the stamped library and write profiles/phase_stamps.md."""
    import subprocess
    from paper_2609_13716_amd import build
    if not os.path.exists(build.LIB_STAMPS):
        raise SystemExit(f"{build.LIB_STAMPS} is not built; run `python -m paper_2609_13716_amd.build --stamps`")
    r = subprocess.run([sys.executable, os.path.abspath(__file__), "--phases-child"], capture_output=True,
                       text=True, env=dict(os.environ, RL_LIB_PATH=build.LIB_STAMPS), cwd=ROOT)
    if r.returncode != 0:
        raise SystemExit(f"stamped run failed ({r.returncode}):\n{r.stderr[-2000:]}")
    res = json.loads(r.stdout.strip().splitlines()[-1])
    md = ["# Phase stamps of the fused and env-only step loops, one MI355X", "",
          "Commands (repository root): `python -m paper_2609_13716_amd.build --stamps` (on the build host), then "
          "`python3 bench.py --phases` on the GPU.  The stamped library marks phase boundaries in the kernels' "
          "step loops with s_memtime; each wave sums the cycles between its marks, and the table below gives "
          "shader-clock cycles per step (per loop iteration) per wave of each role, averaged over the grid.  "
          "The stamps add waits of their own (each mark waits for the wave's outstanding LDS operations), so "
          "the launch takes longer than in the product build: read the split, not the total.", ""]
    for (case, name, call, unit, extra, roles, names), rr in zip(PHASE_CASES, res):
        names = names or PHASE_CASES[0][6]
        tab = rr["table"]
        md += [f"## {case} ({name}, {call}; stamped launch {rr['ms']:.3f} ms, {rr['iterations']} iterations)", "",
               "| phase | " + " | ".join(roles) + " |", "|---|" + "---|" * len(roles)]
        counts = [tab[ro * 12 + 11] for ro in range(len(roles))]
        # roles beyond the named ones (the other waves of a workgroup) are pooled into the last name
        pooled = []
        for ro in range(len(roles)):
            rows = range(ro, 8) if ro == len(roles) - 1 else [ro]
            n = sum(tab[x * 12 + 11] for x in rows)
            pooled.append([sum(tab[x * 12 + ph] for x in rows) / max(n, 1) / rr["iterations"] for ph in range(11)])
        for ph in range(11):
            if any(pr[ph] > 0.5 for pr in pooled):
                md.append(f"| {names.get(ph, ph)} | " + " | ".join(f"{pr[ph]:,.0f}" for pr in pooled) + " |")
        md.append("| total | " + " | ".join(f"{sum(pr):,.0f}" for pr in pooled) + " |")
        md.append("")
    open(os.path.join(ROOT, "profiles", "phase_stamps.md"), "w").write("\n".join(md))
    print("\n".join(md))


# The oracle's timed samples (the CPU baseline): the correctness workload in full, a prefix of each
# 4096+-env workload for its full step count (sized so that each leg takes a few seconds on one core), and
# the headline workload on every host core at once (CPU_SHARD envs per core).
CPU_LEGS = (("lbf8_small", 16, "f32"), ("lbf8_4096", 256, "bf16"), ("lbf12_16k", 64, "bf16"),
            ("oc_4096", 16, "bf16"), ("hn_4096", 64, "bf16"))
CPU_SHARD = 192


def cpu_leg(name, env0, n_envs, dtype, core):
    """One oracle rollout on one pinned core, in a process of its own that never touches the GPU (run as
    ``bench.py --cpu-leg``): envs env0 .. env0 + n_envs - 1 of workload ``name`` for its full step count,
    the workload's policy (weights seed 1000) sampling every action.  Prints agent-steps and seconds."""
    if core is not None:
        os.sched_setaffinity(0, {core})
    from threadpoolctl import threadpool_limits

    from oracle import hanabi, lbf, overcooked, rollout as orollout
    from paper_2609_13716_amd import workloads
    w = workloads.WORKLOADS[name]
    kind, e = workloads.kind(name), w["env"]
    if kind == "overcooked":
        env, oc, A = overcooked, overcooked.Config(e["cook_time"], e["soup_reward"], e["max_steps"], 2), 2
    elif kind == "hanabi":
        env, oc, A = hanabi, hanabi.Config(max_steps=e["max_steps"]), 2
    else:
        env, A = lbf, e["n_agents"]
        oc = lbf.Config(e["grid_h"], e["grid_w"], A, e["n_food"], e["max_agent_level"], e["max_food_level"],
                        e["max_steps"], e.get("const_levels", False))
    ws, bs = workloads.policy_weights(workloads.policy_dims(name), seed=1000)
    T = w["n_steps"]
    with threadpool_limits(1):
        t0 = time.perf_counter()
        orollout.rollout(env, oc, 0, range(env0, env0 + n_envs), 0, T, ws, bs, dtype)
        dt = time.perf_counter() - t0
    acting = 1 if kind == "hanabi" else A  # Hanabi: the mover's row only, as in the GPU figures
    print(json.dumps({"agent_steps": n_envs * T * acting, "env_steps": n_envs * T, "seconds": dt}), flush=True)


def _cpu_children(jobs):
    """Run oracle legs as child processes (each its own interpreter, pinned to one core, one BLAS thread);
    jobs = [(name, env0, n_envs, dtype, core)].  Returns their results and the wall time of the batch."""
    import subprocess
    env = dict(os.environ, OMP_NUM_THREADS="1", OPENBLAS_NUM_THREADS="1", MKL_NUM_THREADS="1")
    t0 = time.perf_counter()
    procs = [subprocess.Popen([sys.executable, os.path.abspath(__file__), "--cpu-leg", n, str(e0), str(ne), dt,
                               str(c)], stdout=subprocess.PIPE, env=env, cwd=ROOT)
             for n, e0, ne, dt, c in jobs]
    outs = []
    for pr in procs:
        out, _ = pr.communicate()
        if pr.returncode != 0:
            raise RuntimeError(f"oracle leg failed with status {pr.returncode}")
        outs.append(json.loads(out.decode().strip().splitlines()[-1]))
    return outs, time.perf_counter() - t0


def _host_info():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    rocm = "unknown"
    for path in ("/opt/rocm/.info/version", "/opt/rocm/.info/version-dev"):
        if os.path.exists(path):
            rocm = open(path).read().strip()
            break
    return model, rocm


def cpu_baseline():
    """The oracle timed on this host's cores: every leg of CPU_LEGS single-threaded on a core of its own, then the headline
    workload's CPU_SHARD-env shards on P cores at once (P = this process's CPU affinity count, one process per core,
    disjoint env ids).  The all-cores figure is the reported baseline value: the shards' agent-steps over the
    slowest shard's rollout time (process start-up excluded; the batch's wall time is given beside it)."""
    cores = sorted(os.sched_getaffinity(0))
    P = len(cores)
    legs = {}
    # the single-threaded legs run side by side, each alone on its own core
    outs, _ = _cpu_children([(name, 0, n, dt, cores[i % P]) for i, (name, n, dt) in enumerate(CPU_LEGS)])
    for (name, n, dt), r in zip(CPU_LEGS, outs):
        legs[name] = {"agent_steps_per_s": round(r["agent_steps"] / r["seconds"], 1),
                      "env_steps_per_s": round(r["env_steps"] / r["seconds"], 1),
                      "sample": f"envs 0..{n - 1} x the full step count, {dt} policy", "seconds": round(r["seconds"], 2)}
    n = CPU_SHARD
    outs, wall = _cpu_children([(WORKLOAD, n * i, n, "bf16", c) for i, c in enumerate(cores)])
    agent_steps = sum(o["agent_steps"] for o in outs)
    slowest = max(o["seconds"] for o in outs)
    model, rocm = _host_info()
    return {"value": round(agent_steps / slowest, 1), "unit": "agent-env steps/s", "cores": P, "kind": "oracle",
            "sample": f"{WORKLOAD}: {P} processes, one per core, each envs {n}i..{n}i+{n - 1} x 128 steps (bf16 "
                      f"policy); slowest shard {slowest:.1f} s, batch wall {wall:.1f} s",
            "single_thread": legs, "cpu_model": model, "rocm_version": rocm, "host_cpus": P}


def main():
    args = parse()
    if args.cpu_leg:
        n, e0, ne, dt, c = args.cpu_leg
        cpu_leg(n, int(e0), int(ne), dt, None if c == "none" else int(c))
        return
    if args.cpu_only:
        print(json.dumps({"cpu_baseline": cpu_baseline()}), flush=True)
        return
    if args.phases_child:
        phases_child()
        return
    if args.phases:
        phases()
        return
    if args.counter_plan:
        for ps, leg, cmd in counter_commands():
            print(f"{ps} {leg}\t{cmd}")
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the rollout shards over GPUs "
              "by env id with no exchange, and this benchmark times the single-GPU shard.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2609_13716_amd import rollout as R
    from paper_2609_13716_amd import workloads

    w = workloads.WORKLOADS[WORKLOAD]
    E, T = w["n_envs"], w["n_steps"]
    A = w["env"]["n_agents"]
    cfg = R.EnvConfig(n_envs=E, seed=0, **w["env"])
    D, nA = R.rl_obs_dim(cfg), R.rl_num_actions(cfg)
    dims = workloads.policy_dims(WORKLOAD)
    ws, bs = workloads.policy_weights(dims, seed=1000)
    flop_per_row = 2 * sum(dims[i] * dims[i + 1] for i in range(3))
    planes = 2 * A + 2 * w["env"]["n_food"] + 3
    results = {}

    def rollout_case(dt):
        pol = R.Policy(ws, bs, dt)
        es = 2 if dt == "bf16" else 4
        state = R.new_state(cfg)
        R.rollout_init(cfg, state)
        obs = torch.empty(T, E, A, D, dtype=pol.torch_dtype, device="cuda")
        acts = torch.empty(T, E, A, dtype=torch.int32, device="cuda")
        rew = torch.empty(T, E, device="cuda")
        done = torch.empty(T, E, dtype=torch.uint8, device="cuda")
        last = torch.empty(E, A, D, dtype=pol.torch_dtype, device="cuda")
        t_next = [0]

        def step():
            R.rollout_run(cfg, pol, state, t_next[0], T, obs=obs, actions=acts, reward=rew, done=done,
                          obs_last=last)
            t_next[0] += T

        kern_ms, wall_ms = timed(step, args.steps, args.warmup)
        # algorithmic bytes: trajectory outputs + final obs + state read and written once
        nbytes = run_bytes(E, T, A, D, es, E * planes * 4) + E * A * D * es
        flops = E * A * T * flop_per_row
        agent_steps = E * A * T
        return dict(kern_ms=kern_ms, wall_ms=wall_ms, bytes=nbytes, flops=flops,
                    value=agent_steps / (wall_ms * 1e-3), env_steps_s=E * T / (wall_ms * 1e-3),
                    gbs=nbytes / (kern_ms * 1e-3) / 1e9, tflops=flops / (kern_ms * 1e-3) / 1e12)

    def env_case(dt):
        tdt = torch.bfloat16 if dt == "bf16" else torch.float32
        es = 2 if dt == "bf16" else 4
        state = R.new_state(cfg)
        R.rollout_init(cfg, state)
        g = torch.Generator(device="cuda")
        g.manual_seed(7)
        acts = torch.randint(0, nA, (T, E, A), dtype=torch.int32, device="cuda", generator=g)
        obs = torch.empty(T, E, A, D, dtype=tdt, device="cuda")
        rew = torch.empty(T, E, device="cuda")
        done = torch.empty(T, E, dtype=torch.uint8, device="cuda")
        t_next = [0]

        def step():
            R.rollout_step(cfg, state, t_next[0], acts, obs, rew, done)
            t_next[0] += T

        kern_ms, wall_ms = timed(step, args.steps, args.warmup)
        nbytes = env_bytes(E, T, A, D, es, E * planes * 4)
        return dict(kern_ms=kern_ms, wall_ms=wall_ms, bytes=nbytes, gbs=nbytes / (kern_ms * 1e-3) / 1e9,
                    env_steps_s=E * T / (wall_ms * 1e-3))

    def policy_case(dt):
        pol = R.Policy(ws, bs, dt)
        rows = E * A * T
        g = torch.Generator(device="cuda")
        g.manual_seed(3)
        x = torch.randint(0, 3, (rows, D), device="cuda", generator=g).to(pol.torch_dtype)
        logits = torch.empty(rows, nA, device="cuda")

        def step():
            R.policy_forward(pol, x, logits=logits)

        kern_ms, wall_ms = timed(step, args.steps, args.warmup)
        flops = rows * flop_per_row
        return dict(kern_ms=kern_ms, rows=rows, flops=flops, tflops=flops / (kern_ms * 1e-3) / 1e12)

    if args.workload_only:
        wl = workloads.WORKLOADS[args.workload_only]
        measure = (measure_population if "population" in wl else measure_s5 if "s5" in wl else
                   measure_actor_critic if wl.get("value_head") else measure_workload)
        print(json.dumps(measure(R, workloads, args.workload_only, "bf16", args.steps, args.warmup)),
              flush=True)
        return

    if args.only == "copy":
        n = 512 << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"only": "copy", "bytes_read": n, "bytes_written": n}))
        return

    if args.only:
        kind, dt = args.only.split("_")
        {"run": rollout_case, "env": env_case, "policy": policy_case}[kind](dt)
        torch.cuda.synchronize()
        print(json.dumps({"only": args.only, "done": True}))
        return

    results["run_bf16"] = rollout_case("bf16")
    results["run_f32"] = rollout_case("f32")
    results["env_bf16"] = env_case("bf16")
    results["env_f32"] = env_case("f32")
    results["policy_bf16"] = policy_case("bf16")
    results["policy_f32"] = policy_case("f32")

    rb, rf = results["run_bf16"], results["run_f32"]
    line = {
        "metric": METRIC,
        "value": round(rb["value"], 1),
        "unit": "agent-env steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(rb["wall_ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded LBF episodes, random-init MLP weights N(0, 1/fan_in))",
        "config": {"workload": "LBF 8x8, 2 agents, 3 food, 4096 envs x 128 steps, MLP 192-128-128-6 bf16",
                   "n_envs": E, "n_agents": A, "steps_per_rollout": T, "parallelism": "single GPU"},
        "env_steps_per_s": round(rb["env_steps_s"], 1),
        "roofline": roofline("hbm", rb["gbs"], HBM_PEAK_GBS, "GB/s", load_traffic("lbf8_4096_run_bf16:run")),
        "kernel_ms": round(rb["kern_ms"], 4),
        "f32": {"value": round(rf["value"], 1), "ms_per_step": round(rf["wall_ms"], 4),
                "kernel_ms": round(rf["kern_ms"], 4),
                "roofline": roofline("mfma", rf["tflops"], MFMA_PEAK_TFLOPS["f32"], "TFLOP/s",
                                     load_traffic("lbf8_4096_run_f32:run"))},
        "env_only": {dt: {"env_steps_per_s": round(results[f"env_{dt}"]["env_steps_s"], 1),
                          "kernel_ms": round(results[f"env_{dt}"]["kern_ms"], 4),
                          "roofline": roofline("hbm", results[f"env_{dt}"]["gbs"], HBM_PEAK_GBS, "GB/s",
                                               load_traffic(f"lbf8_4096_env_{dt}:env"))}
                     for dt in ("bf16", "f32")},
        "policy_forward": {dt: {"rows": results[f"policy_{dt}"]["rows"],
                                "kernel_ms": round(results[f"policy_{dt}"]["kern_ms"], 4),
                                "roofline": roofline("mfma", results[f"policy_{dt}"]["tflops"],
                                                     MFMA_PEAK_TFLOPS[dt], "TFLOP/s",
                                                     load_traffic(f"lbf8_4096_policy_{dt}:policy"))}
                           for dt in ("bf16", "f32")},
        "csrc_hash": csrc_hash(),
    }
    if not args.no_workloads:
        # the other workloads at full size, bf16, a few timed launches each
        line["workloads"] = {n: measure_workload(R, workloads, n, "bf16", min(args.steps, 5), 1)
                             for n in ("lbf12_16k", "oc_4096", "hn_4096", "hn_mini_4096", "lbf7_const_4096",
                                       "lbf7_teams_4096")}
        line["workloads"]["lbf8_4096_ac"] = measure_actor_critic(R, workloads, "lbf8_4096_ac", "bf16",
                                                                 min(args.steps, 5), 1)
        line["workloads"]["lbf8_4096_pop"] = measure_population(R, workloads, "lbf8_4096_pop", "bf16",
                                                                min(args.steps, 5), 1)
        line["workloads"]["lbf8_4096_s5"] = measure_s5(R, workloads, "lbf8_4096_s5", "bf16", min(args.steps, 3), 1)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
