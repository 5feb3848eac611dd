"""Oracle for Autonomy-of-Heads head-mixed attention (CPU, numpy float64).

THIS PACKAGE IS TEST INFRASTRUCTURE. It is the plain, slow, obviously correct
definition that the HIP kernels are checked against. Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it. The product path (``paper_2608_06849_amd``) never imports it, and it
never imports the product path: the two share no code.

Modules
  attention   -- masks and masked-softmax attention (prefill rows, decode steps),
                 the attention-weight matrix, and an explicit-mask brute force.
  cache_model -- where a token lands in the paged cache and in the streaming
                 ring, and the expected cache image after a series of appends.
  accounting  -- visible-pair counts, FLOP/byte counts and the KV-cache bytes
                 formula that reproduces the paper's memory tables.
  classifier  -- the effective-rank head classifier (proxy spectrum, effective
                 rank, group mean, lowest-k retrieval selection).

Parity status of each function is stated in its docstring; every function is
pinned by a ``-m "not gpu"`` test (see tests/test_oracle_*.py).
"""
from . import attention, cache_model, accounting, classifier, h2share  # noqa: F401
