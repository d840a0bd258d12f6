"""Single-GPU Speculative Pipeline Decoding step for MI355X (gfx950).

libspd.so (built from csrc/ by build.py) holds the HIP kernels and the C ABI of include/spd.h;
`binding` marshals its calls; `engine` provides device memory and streams through PyTorch."""
