"""MI355X-native batched multi-agent rollout (Level-Based Foraging on gfx950).

The compute path is the HIP library ``librollout.so`` (sources in ``csrc/``,
C ABI in ``include/rollout.h``); ``rollout`` is its Python binding and
``workloads`` draws the seeded synthetic inputs.  Build with
``python -m paper_2609_13716_amd.build``.
"""
