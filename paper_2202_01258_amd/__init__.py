"""MI355X (gfx950) implementation of one massively-parallel MAP-Elites
generation: uniform selection, Iso+LineDD variation, batched evaluation,
descriptor-to-cell mapping and per-cell scatter-max insertion, all in HIP
kernels behind the C ABI of include/qd.h (libqd.so)."""
from . import workloads  # noqa: F401
from .qd import Archive, QdError, layout_query, make_config  # noqa: F401
