"""MI355X-native denoising step of a masked-diffusion transformer.

``dlm`` is the ctypes binding of the C ABI in include/dlm.h (libdlm.so, HIP
kernels for gfx950); ``engine`` is the host-side block/request bookkeeping
around it. There is no CPU implementation in this package.
"""
