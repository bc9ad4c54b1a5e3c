"""MI355X-native block-swapped inference engine (SwapNet's method on gfx950).

``swapnet`` is the ctypes binding of libswapnet.so; ``workloads`` holds the
seeded synthetic networks; ``build`` compiles the HIP library in-tree.
"""
