"""MI355X-native speculative sampling (Chen et al., 2023).

Submodules:
  sps      ctypes binding of libsps.so (the HIP library); importing it fails
           loudly when the library has not been built.
  configs  the named model shapes and workloads.
  synth    seeded synthetic input generators (weights, prompts, KV, probs).
  build    compiles libsps.so for gfx950 with hipcc.
"""
