"""Oracle for the decode-maximal hybrid-batch decoder layer (TEST INFRASTRUCTURE).

A plain, slow, float64 CPU implementation of what the GPU path computes.  It
exists to check the HIP library and nothing else: only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  It shares no code with the HIP path and imports nothing from it.

Kind of result: the method (chunked prefills + decode-maximal batching,
Sec. 4.2-4.3) reaches exactly the result of the plain definition -- a
pre-norm decoder layer in which every token attends causally to the tokens of
its own request -- so the oracle is that definition written out, token by
token, with the hybrid batch being only a grouping of rows.

Pins: every function here is pinned by ``tests/test_oracle_pins.py`` against
closed forms, invariants, library routines and brute force.  The absolute
values of a full layer with random weights have no printed counterpart in the
paper; beyond those pins they are pinned only through the invariants
(chunking, batch and concatenation invariance, residual identity).
"""
from .layer import (  # noqa: F401
    OracleBatch, OracleMixedBatch, LayerOut, rms_norm, layer_norm, linear, rope_rotate, silu, gelu,
    attend, layer_forward, model_step, token_positions, chunk_visibility,
)
