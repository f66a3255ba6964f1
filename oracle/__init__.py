"""CPU oracle for Linearized 2-Simplicial Attention (LinSimp).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from this package.  The
GPU product path never calls it, and it shares no code with the HIP library:
it imports nothing from ``paper_2608_09307_amd`` and the library imports nothing
from here.

Everything is plain numpy in float64 (pure-Python loops only in ``brute``).
Each function cites the passage of the paper it writes out:

* ``linsimp``    -- the layer itself: feature map, pair / recurrent /
                    log-space / chunked forms, the exact gradient, the decode
                    step, the exact-kernel operators it approximates.
* ``brute``      -- pure-Python nested loops over tiny inputs (pair sums).
* ``montecarlo`` -- Lemma 1 (unbiasedness) and the closed-form variance of the
                    random-feature kernel estimate.
* ``features``   -- the orthogonal random-feature bank of App. B.1.
* ``layer``      -- the full head around the core: L2 normalisation and the
                    query temperature (Sec. 3.1), the gated RMSNorm output
                    (eq:gated-output) and the channel-wise gate variant.

Reading conventions (where the paper is silent or ambiguous) are listed in
the module docstring of ``linsimp``.
"""

from . import linsimp, brute, montecarlo, features, layer  # noqa: F401
