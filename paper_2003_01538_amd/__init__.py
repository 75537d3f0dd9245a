"""MI355X-native ensemble inference (FlexServe's hot path): one shared
transformation of a variable-size image batch, N co-resident CNNs run by
hand-written gfx950 HIP kernels, per-model softmax and an ensemble combine.

The C ABI is declared in include/flexserve.h; ``flexserve`` is its ctypes
binding and ``build`` compiles libflexserve.so in-tree.
"""
