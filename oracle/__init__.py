"""CPU oracle for RadixAttention's hot path -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously correct reference implementations written from the
paper (SGLang, arXiv 2312.07104):

* ``attention``: causal softmax attention in float64, recomputed from scratch
  for every request with no cache (the definition the cached kernels must
  reach; section 3 and Appendix A.1);
* ``radix``: the radix tree with LRU leaf eviction and reference counters,
  and the shared token pool (section 3, Algorithm 1);
* ``replay``: the per-request call sequence of Algorithm 1 run against that
  tree, producing the slot tables a batch attends through;
* ``router``: the data-parallel router's per-worker prefix holdings as plain
  sets (Appendix A.4).

Only the tests, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg
may import this package.  It shares no code with the HIP library and never
imports it; the only inputs both sides share come from ``workload``.
"""
