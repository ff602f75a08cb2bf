"""MI355X-native AVQ-Attention forward pass (HIP kernels behind a C ABI)."""
