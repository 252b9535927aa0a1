"""Float64 CPU oracle of one entropic-time decode step.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct
NumPy implementation of what the HIP library computes.  Only the test suite,
the smoke check and the benchmark's CPU-baseline leg may import it; the
library and its Python binding never do, and it shares no code with them.

Modules, each following the paper's definitions (section cited per function):

* ``entropy``    -- exact Shannon entropy of the tempered softmax, the top-k
                    and tail-corrected estimates of it, entropic time, and
                    the temperature control law.
* ``blocks``     -- per-block mean keys, block entropic contributions, the
                    entropy-driven block budget and the kept-block set.
* ``attention``  -- decode attention restricted to the kept blocks.
* ``sample``     -- inverse-CDF sampling at the controlled temperature.
* ``append``     -- appending one token to the paged cache.
* ``schedule``   -- entropy-aware selection of the sequences of the next batch.
* ``layout``     -- reading the library's buffer layouts.
* ``step``       -- the whole step for a batch, built from the above.

Readings where the paper is silent or garbled are stated in each function's
docstring; the ones that cannot be pinned to the paper say "parity unpinned".
"""
from . import entropy, blocks, attention, sample, append, layout, step, schedule  # noqa: F401
