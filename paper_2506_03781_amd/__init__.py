"""MI355X-native UniQuan_F fake-quant path (arXiv 2506.03781).

libuniquan.so (HIP, gfx950) is the product; ``uniquan`` is its ctypes binding
and ``layer`` drives one optimisation step of one linear layer through it.
Importing the package does not load the library; the first call does, and
fails loudly if it has not been built.
"""
__all__ = ["uniquan", "layer", "synth", "build"]
