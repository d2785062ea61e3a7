"""MI355X (gfx950) activation-sparse dReLU FFN and top-k MoE decode path
(Turbo Sparse, arXiv 2406.05955).

``paper_2406_05955_amd.binding`` is the ctypes binding of the HIP library
(libturbosparse.so, C ABI in include/turbosparse.h); ``synth`` draws the
seeded synthetic inputs; ``build`` compiles the library in-tree.
"""
import importlib

__all__ = ["binding", "synth", "build"]


def __getattr__(name):
    if name in __all__:
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
