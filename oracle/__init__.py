"""CPU oracle for the batched multi-agent rollout (test infrastructure only).

This package is a plain, slow, single-threaded reference of what the GPU
rollout computes: the Dec-POMDP step of the paper's problem setting (Section 3:
transition P(s'|s,a), shared team reward r(s,a), per-agent observation,
initial-state distribution rho), the counter-based random draws that drive it,
the categorical action sampler and the per-agent MLP policy.

It is test infrastructure.  Only the test suite, the package smoke check and
the CPU-baseline leg of the benchmark may import it.  The GPU library never
calls it, links it or reads anything it produces, and it imports nothing from
the GPU package: the two implementations share no code.  Inputs that both
sides consume (policy weights, injected actions, seeds) are drawn by a
separate generator module that holds none of the method's arithmetic.

Modules
-------
philox    Philox4x64-10 block function and the derived integer draws.
sampling  Gumbel-max categorical sampling over masked fp32 logits.
mlp       Per-agent tanh MLP in fp64, with bf16 rounding emulation.
lbf       Level-Based Foraging: reset, step, observation.
overcooked  Overcooked-style two-agent kitchen: layout, reset, step, observation.
hanabi    Two-player Hanabi: deal, legality, step, observation.
rollout   The rollout loop: observe, act, step, auto-reset.
actor_critic  log pi(a) of sampled actions and generalised advantage estimates.

Environment rules that the paper leaves open (it names the environments and
their sources, Section 4 "Environments" and the environment table, but does
not restate their dynamics) follow one fixed reading each; every reading is
stated in the docstring of the function that implements it.
"""
