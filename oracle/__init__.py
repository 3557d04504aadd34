"""CPU oracle for the HetPipe stage step and the Wave Synchronous Parallel update.

TEST INFRASTRUCTURE ONLY.  Only tests/, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The library in
``paper_2005_14038_amd`` never imports it and shares no code with it; the two
meet only through the seeded inputs of the ``seeded_inputs`` module.

Contents
  * ``ops``    -- the stage operators (conv, FC, ReLU, max-pool, batch-norm,
                  residual add, global average pool, softmax cross-entropy),
                  plain double-precision loops in ``oracle.c``.
  * ``nets``   -- the layer graphs of the five workloads (Tiny CNN, VGG-19,
                  ResNet-152 and stages of them) and their flat parameter layout.
  * ``stage``  -- forward and backward of a layer graph built on ``ops``.
  * ``wsp``    -- the WSP algorithm (HetPipe Sec. 4 local staleness and Sec. 5
                  waves, clocks and the clock-distance bound) as a deterministic
                  simulation of several virtual workers.
  * ``bf16``   -- round-to-nearest-even emulation of bfloat16 operands.
"""
