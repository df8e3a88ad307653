"""MI355X-native Pr^2 MoE-layer hot path: HIP kernels behind a C ABI."""
