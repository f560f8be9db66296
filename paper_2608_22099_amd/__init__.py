"""Structure-aware banded LU on MI355X (gfx950).

The path of "When Structure is Silent" (Sec. II-A three steps, Listing 2):
identify the bandwidths of a dense-stored matrix, convert it to the xGBTRF
band layout, and factor it with banded LU with partial pivoting; then solve.

Every step runs in hand-written HIP kernels in ``libbandlu.so``; the Python
module :mod:`paper_2608_22099_amd.bandlu` is a thin ctypes binding over the
C ABI declared in ``include/bandlu.h``.  Import it explicitly:

    from paper_2608_22099_amd import bandlu

:mod:`paper_2608_22099_amd.inputs` holds the seeded synthetic generators.
"""
