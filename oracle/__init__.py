"""CPU oracle of the integer relative-position attention block (test infrastructure).

Only ``tests/``, the smoke check in ``__graft_entry__`` and the CPU-baseline leg
of ``bench.py`` import this package; the GPU library never does.

* ``core``      -- the C oracle (scalar int64), step by step and whole-block.
* ``fp_block``  -- the floating-point block of Eq. 8-9 on dequantized inputs.
* ``swish``     -- the minimax integer Swish of Eq. 12-13 and its float forms.
"""
