"""CPU oracle -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously correct reference implementations of what the HIP
library computes, written from the paper (Libra, arXiv 2607.23250):

* ``oracle.plan``      -- SH-Tiles (Eq. 5), tile cost (Eq. 6), KV groups
  (Eq. 7), communication increment (Eq. 8) and the communication-aware
  placement of Algorithm 2, in pure Python integers.
* ``oracle.attention`` -- document-masked causal attention (Eq. 1 under the
  block-diagonal causal mask of Sec. 2.3), forward and backward, in float64
  (torch CPU), one sample and one head at a time.
* ``oracle.vrsp``      -- Variance-Reduced Sequence Placement (Algorithm 1,
  Eq. 4) and the inter-pool imbalance R - 1 of Sec. 3.2, in Python integers.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` legs of
``bench.py`` may import this package.  It shares no code with the HIP library
and imports nothing from it; the product path never falls back to it.
"""
