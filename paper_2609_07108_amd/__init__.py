"""MI355X (gfx950) draft branch attention under context parallelism.

The computation lives in ``libbranchattn.so`` (HIP kernels + C ABI, declared
in include/branch_attn.h); :mod:`.binding` is its ctypes binding,
:mod:`.rankshare` lays out one rank's share of a packed problem, and
:mod:`.workloads` draws seeded synthetic inputs.  Importing the package does
not load the library; :func:`load` (or any binding call) does, and fails if it
has not been built.
"""

__all__ = ["load", "workloads"]

from . import workloads  # noqa: E402


def load():
    from . import binding
    return binding.lib()
