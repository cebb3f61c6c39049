"""CPU oracle: plain, slow, obviously correct reference implementations.

TEST INFRASTRUCTURE ONLY. Nothing under ``oracle/`` is part of the product:
only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import it. It shares no code with the GPU library; the only
common module is ``paper_2609_12075_amd.synth`` (shapes and seeded input
generators, which hold none of the method's arithmetic).
"""
