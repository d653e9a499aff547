"""MI355X (gfx950) implementation of ShallowStream's query-time evidence
retrieval over a shallow-layer key index.

The work runs in ``libshallowstream.so`` (HIP kernels behind the C ABI of
``include/shallowstream.h``); this package only marshals arguments.
"""
from ._lib import SSError, lib  # noqa: F401
from .index import PooledRanker, Retriever, ShallowIndex, assemble_evidence, set_profile_events  # noqa: F401

__all__ = ["ShallowIndex", "Retriever", "PooledRanker", "assemble_evidence", "SSError", "set_profile_events", "lib"]
