"""MI355X-native OffQ W4A4KV4 online path (HIP kernels behind a C ABI)."""
