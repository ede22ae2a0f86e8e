"""MI355X-native decoder-layer shard of Voltron (arXiv 2607.07046).

The compute path is libvoltron.so (HIP kernels for gfx950 behind the C ABI
in include/voltron.h); ``voltron`` is its ctypes binding and ``pack`` the
shard-wise device allocation of weights. Importing the package loads
nothing; the first call into ``voltron`` loads the library and fails loudly
if it has not been built.
"""
