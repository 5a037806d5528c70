"""PQ-HSA decode attention for MI355X (gfx950): HIP kernels behind a C ABI.

    from paper_2609_33746_amd import PQHSA
The binding loads paper_2609_33746_amd/_lib/libpqhsa.so (built by
paper_2609_33746_amd.build); importing the package itself loads nothing.
"""

__all__ = ["PQHSA", "PQHSAError", "load_library"]


def __getattr__(name):
    if name in __all__:
        from . import pqhsa
        return getattr(pqhsa, name)
    raise AttributeError(name)
