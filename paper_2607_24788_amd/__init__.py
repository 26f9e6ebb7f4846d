"""GLIDE hybrid-attention step for AMD Instinct MI355X (gfx950).

The compute lives in libglide.so (HIP kernels behind the C ABI of
include/glide.h); ``glide`` is its ctypes binding and ``workload`` the
synthetic input generator."""
