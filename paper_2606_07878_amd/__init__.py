"""Still compactor forward pass on MI355X (gfx950): C-ABI library + thin binding.

Submodules: ``configs`` (shapes), ``synth`` (seeded synthetic inputs),
``binding`` (ctypes marshalling of libstill.so), ``build`` (hipcc build).
The HIP library is loaded lazily by ``binding.lib()``; it is never replaced by
a CPU path.
"""
from . import configs  # noqa: F401
