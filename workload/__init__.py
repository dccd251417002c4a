"""Seeded synthetic inputs shared by the oracle and the GPU harness.

``contentgen``, ``scenarios`` and ``gpu_gen`` compute no attention and
maintain no radix tree: they only produce token sequences, workload recipes
and content-addressed bf16 values, and the oracle may use them.  ``driver``
is the GPU side's workload driver: it runs a scenario through the package
(radix cache, slot tables, kernels) and is never imported by the oracle.
"""
