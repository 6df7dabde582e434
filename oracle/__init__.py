"""CPU oracle for the block-sparse attention path with a reusable block mask.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports this package:
only the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg
of ``bench.py`` may call it.  It shares no code with the HIP library.

Everything here is plain NumPy in float64 (the fp8 codec works on exact
integer/fp32 values), written for a reader who checks it against the paper
(Chorus II, "Cross-Request Sparsity Reuse for Efficient Image-to-Video
Generation"):

* ``attention``  -- block-masked softmax attention, the definition the sparse
  kernel must reproduce (Sec. 3.2, "Efficient block-sparse kernel": pruned
  block pairs are skipped in QK^T, softmax and PV, i.e. carry zero weight).
* ``mask``       -- the mean-pool block-score predictor (Sec. 3.2, Obs. 2) with
  the joint top-p / minimum-top-k selection (Sec. 3.2, "Mask Caching and
  Retrieval" and "Minimum top-k guarantee"; knobs in Sec. 4.1).
* ``fp8``        -- OCP e4m3fn round-to-nearest-even codec and the per-(head,
  64-token block) quantiser feeding the FP8 path (Sec. 3.2, FP8 backend).
* ``mass``       -- the true block attention mass of a request, the top-p /
  top-k mask selected from it (the masks a historical request records, Sec.
  3.2 "Mask Caching and Retrieval") and the coverage of a mask on a request
  (Sec. 3.2, Obs. 1).
* ``fallback``   -- block-pair visit refreshing over a layer group, the first
  safeguard of Sec. 3.2 "Safety fallback against information loss".
* ``guidance``   -- the first-frame key enhancement of Eq. (1) (Sec. 3.4),
  applied to K before any of the above.

Every function is pinned by ``tests/test_oracle_*.py`` against brute force,
closed forms, library routines and invariants.  The one part with no outside
pin is agreement with the paper's own numbers: the paper prints no mask,
output or worked example for this path ("parity unpinned" against the paper
itself; pinned against the mathematics).
"""

from . import attention, fallback, fp8, guidance, mask, mass  # noqa: F401
