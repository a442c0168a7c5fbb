"""CPU oracle for bounded state staging.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``, never by the product path, and it
imports nothing from the product path.  See ``oracle/staging.py``.
"""
from .staging import (  # noqa: F401
    Model,
    checksum,
    chunk_checksums,
    chunk_spans,
    inverse,
    moment_stream,
    padded_elems,
    reshard,
    rne_bf16,
    rollout_rank,
    rollout_stream,
    rollout_table,
    rollout_tensor,
    rollout_tensors,
    shards,
    split_stream,
    training_offsets,
    training_tensors,
    training_views,
    widen_bf16,
)
