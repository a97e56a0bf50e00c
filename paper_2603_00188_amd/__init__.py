"""MI355X-native ST-Lite KV-cache compression pass (HIP kernels behind a C ABI)."""
