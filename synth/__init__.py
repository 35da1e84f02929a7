"""Seeded synthetic inputs for the sparse decode-step hot path.

This package only draws inputs (queries, KV block records, lengths, query
drift, synthetic selection streams).  It contains none of the method's
arithmetic: no metadata, scoring, selection, caching or attention.  Both the
oracle-side tests and the GPU path are fed from it.
"""
from .configs import CONFIGS, Config, get  # noqa: F401
from . import gen  # noqa: F401
