"""MI355X-native parallel-window neural decoder (HIP kernels behind a C ABI)."""
