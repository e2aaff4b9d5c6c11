"""MI355X-native MoE-layer training step (the hot path Lancet overlaps with
all-to-all communication): HIP kernels behind a C ABI (include/lancet_moe.h),
with a thin ctypes binding in ``lancet_moe``."""
