"""CPU oracle for the rollout hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct numpy implementation of what rollout
generation computes (paper section 2.1: the actor produces R0 responses for
each of P0 prompts) for a Qwen2.5-style decoder, of the Philox-keyed
Gumbel-max sampler, and of the tail-batching round policy (section 3).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The HIP library never calls it, and it
shares no code with the HIP library: both sides only consume the seeded
inputs from the ``workloads`` package.

Floating point is fp64 except where a float decides an integer (the sampler's
argmax), which is taken in fp32 like the kernel.  Every function is pinned by
a CPU test against something other than itself (see tests/test_oracle_*.py);
there is no "parity unpinned" function in this package.
"""
from . import model, sampling, schedule  # noqa: F401
