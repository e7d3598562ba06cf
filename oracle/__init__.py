"""CPU oracle for the function-level KV grafting hot path.  TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or run anything in this package.  The product path
(the HIP library and its Python binding) never imports it and shares no code
with it.

What it computes, in plain float64 NumPy, following the paper's statement of
the method:

* ``numerics`` - storage dtypes (fp32, bf16) and their round-to-nearest-even
  narrowing.
* ``rope``     - the rotary position encoding the cached keys carry, and the
  re-alignment of a cached key to a new position (a rotation by the position
  delta).  The paper composes cached function modules "not tied to fixed
  prefix positions" (Sec. 4.1, two-tier code cache) while keeping each
  module's internal token order (App. B.1, module-level cache reuse; App. C.7).
* ``layout``   - where every grafted segment and every fresh token lands in the
  composite cache: offsets, deltas, the contiguous or paged slot map, and the
  validation rules of the library boundary.
* ``graft``    - the composite cache itself: the interface KV states of the
  retrieved functions concatenated as context (Sec. 4.2, Eq. 4), keys
  re-rotated, values copied.
* ``attention``- causal grouped-query softmax attention of the patch tokens and
  of each decode step over the grafted cache (Sec. 4.2, Eq. 6: the prefix KV is
  reused and only the new span is computed).

Parity status of each function is stated in its module header; every function
here is pinned by a ``-m "not gpu"`` test against closed forms, invariants,
brute force or an independent library routine.
"""
