"""MI355X (gfx950) implementation of ShallowStream's query-time evidence
retrieval over a shallow-layer key index.

The work runs in ``libshallowstream.so`` (HIP kernels behind the C ABI of
``include/shallowstream.h``); this package only marshals arguments.
"""
from ._lib import SSError, lib  # noqa: F401
from .index import (LongClusters, PooledRanker, Retriever, ShallowIndex, assemble_evidence,  # noqa: F401
                    sample_plan, set_profile_events)

__all__ = ["ShallowIndex", "Retriever", "PooledRanker", "LongClusters", "assemble_evidence", "SSError", "sample_plan",
           "set_profile_events", "lib"]
