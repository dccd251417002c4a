"""Seeded synthetic inputs shared by the oracle and the GPU harness.

Nothing here computes attention or maintains a radix tree: this package only
produces token sequences, workload recipes and content-addressed bf16 values.
"""
