"""CPU oracle for the LVSA hot path.

TEST INFRASTRUCTURE ONLY: a plain, slow restatement of what the LVSA paper
defines (Sec. 2: Def. 1-2, Eq. 1-3, Alg. 1), used to check the HIP library.
Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it.  The library never imports it and it imports
nothing from the library.

  oracle.mask       LVSA frame sets and the block CSR (integer, exact)
  oracle.attention  Eq. 1 / Eq. 2 masked softmax attention (numpy)
"""
from . import mask, attention  # noqa: F401
