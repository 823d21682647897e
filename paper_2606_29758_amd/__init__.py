"""MI355X-native hot path of a PS-PPO policy update (prefix-truncated, importance-weighted
PPO loss through the LM head, with its gradient), as HIP kernels for gfx950 behind a C ABI.

Submodules:
  synth     -- seeded synthetic workloads (inputs only)
  pspo      -- ctypes binding of libpspo.so (sample_cutoffs, pack_prefixes, loss_fwd_bwd)
  pipeline  -- one device-resident pass of the three calls
  build     -- builds libpspo.so with hipcc for gfx950
"""
