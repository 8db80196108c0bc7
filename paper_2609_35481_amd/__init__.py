"""TopoEP per-layer, per-microbatch load-balancing planner on MI355X (gfx950).

The planner itself is the HIP library ``libtopoep.so`` behind the C ABI of
``include/topoep.h``; ``paper_2609_35481_amd.topoep`` is its thin binding.
The binding is imported lazily so that ``paper_2609_35481_amd.build`` works
before the library exists.
"""
import importlib

__all__ = ["topoep", "build"]


def __getattr__(name):
    if name in __all__:
        return importlib.import_module(__name__ + "." + name)
    raise AttributeError(name)
