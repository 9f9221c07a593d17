"""Oracle for the swapped GPT training step.

TEST INFRASTRUCTURE ONLY: plain, slow, obviously correct CPU code.  It may be
imported only by tests/, by the package's smoke() entry and by the CPU-baseline
leg of bench.py.  The product path (the C-ABI library and its Python binding)
never imports, links or runs anything from here, and this package shares no
code with it.  The only module both sides use is `synthetic`, which draws the
seeded inputs and holds none of the method's arithmetic.

* oracle.gpt   - fp64 GPT forward and backward (Section III-B model, Table II
                 shapes), the result every swap schedule must reproduce.
* oracle.adamw - AdamW, the host optimizer step after a global batch.
* oracle.plan  - brute-force enumeration of contiguous partitions of the layer
                 chain under the memory and overlap constraints of Algorithm 1
                 (Section III-D), with the selection rule.
"""
