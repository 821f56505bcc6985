"""CPU oracle for Attention-Aware Transform Coding (AATC) -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct NumPy implementation of what the AATC hot path
computes: calibration (covariance, eigendecomposition, attention-aware weights, integer
reverse water-filling, per-channel scales), encoding (transform, per-token scale,
quantization, bit packing), and exact softmax attention over the decoded cache.  It also
holds the quantities of the paper's distortion theory (Theorem 1, Lemma 1 and the
softmax ray derivatives) for Monte-Carlo pins.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GPU library never imports, links or calls
it, and it shares no code with the GPU library.

Parity status: every function is pinned by the tests under ``tests/test_oracle_*``
except the items listed as "parity unpinned" in ``oracle/aatc.py``'s header.
"""
from . import aatc, groups, theory  # noqa: F401
