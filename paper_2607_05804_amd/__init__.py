"""MI355X-native fused turn-aware reverse-KL distillation loss (TurnOPD hot path).

The compute lives in libturnkl.so (HIP kernels for gfx950, C ABI declared in
include/turnkl.h); paper_2607_05804_amd.turnkl is its thin Python binding.
"""
