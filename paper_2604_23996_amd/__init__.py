"""MI355X-native SMoES MoE layer: HIP kernels for gfx950 behind a C ABI.

Import `paper_2604_23996_amd.smoes` for the binding (it loads libsmoes.so and
fails loudly if the library has not been built); `workloads` holds the seeded
synthetic inputs.
"""
__version__ = "0.1.0"
