"""CPU oracle for the World-Model dream rollout and MDN-NLL pass.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library (no kernels, headers, helpers or constant tables); the two meet only
on the seeded inputs drawn by ``paper_2205_01435_amd.workloads``.

Everything is plain float64 numpy, written from the paper (Parker, Alabed,
Yoneki, "RLFlow: Optimising Neural Network Subgraph Transformation with World
Models", arXiv 2205.01435):

* ``philox``  Philox4x32-10 counter RNG (Salmon et al., SC'11), uint64 numpy.
* ``bf16``    round-to-nearest-even emulation of bfloat16 storage.
* ``wm``      the vectorised oracle: controller (section 3.4), MDN-RNN step and
              temperature-scaled mixture sampling (section 3.3.2), rollout,
              controller step and teacher-forced NLL.
* ``brute``   the same method as scalar Python loops (own Philox, own bf16),
              for tiny shapes only; it pins ``wm`` by agreement.

Every function is pinned by a CPU test (``tests/test_oracle_*.py``) against a
closed form, a library routine, a published known-answer vector, a
distributional test, or the brute-force loops.  The end-to-end values of a
*trained* world model are "parity unpinned": the paper publishes no weights,
data or per-step numbers.
"""

from . import bf16, philox, wm  # noqa: F401
