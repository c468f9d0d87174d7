"""fp64 CPU oracle for the revisit-consistency hot path. TEST INFRASTRUCTURE ONLY.

This package is the plain, slow, obviously correct statement of what the
GPU library computes. Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it; the library itself never
does, and it shares no code, header, table or constant with the HIP
kernels. Inputs are numpy arrays (the same fp32 / bf16-valued arrays the
GPU receives); all arithmetic is float64.

Modules, each citing the passage of the paper it writes out:

* ``retrieval``    -- the retrieval score and admissible set (Sec. 4.2,
  Eq. retrieval);
* ``reprojection`` -- unprojection, relative SE(3), projection and the
  occlusion-aware visibility test (Sec. 4.3, Eq. reprojection and
  Eq. visibility, with design choice (iii));
* ``attention``    -- scaled dot-product attention with the Gaussian
  correspondence bias on retrieved-frame key columns (Sec. 4.3, Eq. bias,
  design choices (ii) and (iii));
* ``kvpack``       -- reinstating retrieved chunks into the cache: gather
  of their keys and values and re-rotation of the keys' temporal position
  embedding to the packed positions (Sec. 4.2, cache layout and cache
  packing);
* ``stream``       -- the cache layout run chunk by chunk over a trajectory:
  history ring, retrieval, slot table, correspondence, packing and biased
  attention composed as the method runs them (Sec. 4.2, Sec. 4.3);
* ``brute``        -- pure-Python loop versions of the first three, for tiny
  inputs, used to pin the vectorised ones.

Every function here has pins in ``tests/test_oracle_*.py`` (closed forms,
invariants, library reductions, brute force); none is "parity unpinned".
"""

from . import attention, brute, kvpack, reprojection, retrieval, stream  # noqa: F401
