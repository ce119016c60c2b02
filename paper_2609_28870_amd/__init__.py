"""MI355X-native hot path of trace-driven prefix-cache eviction analysis.

``pc`` binds the HIP library ``libpc.so`` (see ``include/pc.h``): chained
block hashing, prev/next-use indexing, exact LRU stack distance and the
hit-ratio / compute-savings histograms over every capacity at once."""
from . import pc  # noqa: F401

__all__ = ["pc"]
