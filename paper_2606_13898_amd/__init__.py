"""MI355X-native HiLo-Token compressed DiT block: HIP kernels behind a C ABI (libhilo.so)."""
