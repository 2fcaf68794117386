"""MI355X-native hot path of EMA's memory slice.

The work lives in libema_slice.so (C ABI in include/ema_slice.h, HIP kernels
for gfx950 in csrc/); ``ema`` is its thin Python binding. Build with
``python -m paper_2609_27040_amd.build``.
"""
