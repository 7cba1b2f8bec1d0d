"""MI355X-native multi-tensor LAMB / LARS optimizer step (You et al., Algorithms 1 and 2).

Importing the package loads nothing native. The HIP library is opened on the
first call into ``paper_1904_00962_amd._lib`` (directly or through
``paper_1904_00962_amd.optim.LAMB`` / ``LARS``) and raises if it is missing.
"""

import importlib

__all__ = ["LAMB", "LARS"]


def __getattr__(name):
    if name in ("LAMB", "LARS"):
        return getattr(importlib.import_module(__name__ + ".optim"), name)
    raise AttributeError(name)
