"""CPU oracle for the batched decode step -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 NumPy statement of what one forward pass of the
serving engine computes (the paper's dense mode, "Design and
Implementation": every row runs every layer), written from the paper's
description and the standard decoder definition, never from the device
code.  Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's
CPU-baseline leg may import it.  The device library must never call it.

Contents
  numerics   bf16 rounding, RMSNorm, rotary positions, SiLU, softmax attention
  kvcache    block allocator model, slots, paged KV store
  model      weight source and the forward pass (decode and ragged prefill)

Parity status of each function is stated in its docstring; the test files
``tests/test_oracle_*.py`` pin each one to closed forms, textbook library
routines, invariants or brute force.
"""
from . import numerics, kvcache, model  # noqa: F401
