"""CPU oracle for the GIFT gradient codec -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 numpy implementation of what the codec computes,
written from the paper (GIFT: Geometry-Informed Low-precision Gradient
Communication).  It exists to check the GPU library and is never part of the
product path: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no code with
the GPU library (``paper_2607_07494_amd``) and neither imports the other.

Modules
-------
``e4m3``      OCP FP8 E4M3 decode table and the saturating round-to-nearest-even
              quantizer (the FP8 format of the communication core, Sec. IV-A).
``codec``     factor statistics, the low-rank transform, scaling, quantization,
              the local rank sum, the inverse transform and the reconstruction
              metrics (Sec. II-B, IV-A, V-A, V-B, Algorithm 1).
``subspace``  the iterative rank-r eigen-step the GPU uses for the factor
              refresh, mirrored in float64, and the counter-based random
              generator that seeds it.

Every function is pinned by ``tests/test_oracle_*.py`` against closed forms,
invariants, brute force on tiny inputs or library routines; see the pins listed
in each function's docstring.
"""

from . import e4m3, codec, subspace  # noqa: F401
