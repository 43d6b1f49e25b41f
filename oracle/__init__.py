"""CPU oracle for the out-of-core training step (test infrastructure only).

Plain, slow, obviously correct implementations of what the product computes,
written from the paper (Hayakawa & Narihira, "Out-of-core training for
extremely large-scale neural networks with adaptive window-based scheduling"):

* ``schedule``  -- the adaptive-window swap scheduler (Section 3, Fig. 2) and
                   the in-core plan;
* ``pool``      -- the virtual-address chunk pool (Section 4, eq. 1 and 2);
* ``naive``     -- the swap-before-and-after-every-layer schedule (Section 1)
                   used as a limiting case;
* ``check``     -- an independent replayer that checks any op list against
                   budget, residency and write-back rules;
* ``lower``     -- network description -> function sequence (Section 2);
* ``ops``       -- float64 NumPy forward/backward/SGD of every layer kind;
* ``interp``    -- runs a function sequence with ``ops`` (one training step).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP path and
never imports it; the only module both sides use is the seeded input
generator ``paper_2010_14109_amd.synth``, which holds none of the method.
"""
