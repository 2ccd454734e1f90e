"""MI355X-native online e-prop: the per-timestep hot path of gradient-based
synaptic plasticity (arxiv 2501.11407) as hand-written HIP kernels for gfx950
behind a C ABI, with a thin ctypes binding."""
