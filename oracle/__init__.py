"""Oracle for the block-sparse attention path.

TEST INFRASTRUCTURE ONLY.  Plain, slow, obviously-correct CPU code written
from the paper's definitions (fp64 masked attention, Eq. 1; block-CSR, mask
statistics and physical-plan enumeration, Sections 4-5; offline table
compilation and online selection, Algorithms 1-2; the mean-pooled top-k
sparsifier that supplies the mask, Section 2.1).  It shares no code with
the HIP library.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import it; the library never does.
"""
