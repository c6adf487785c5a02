"""CPU oracle for target-side KV-cache reconstruction.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
link this package: only the tests, the smoke check and the benchmark's CPU
baseline leg use it.  It is a plain, slow, float64 numpy statement of what the
reconstruction computes, written from the paper:

* ``footprint`` -- per-token KV footprint and transfer volume (Eq. 1).
* ``numerics``  -- bf16 round-to-nearest-even from float64.
* ``model``     -- the decoder forward that builds a KV cache by prefill and
                   extends it by one decode step (Sections 2.1 and 4.3).
* ``paged``     -- the paged KV layout, suffix-block extraction, assembly into
                   a new block table, the coverage and epoch checks
                   (Sections 4.3 and 5).
* ``scheduler`` -- the prefetching-window model and its online selection,
                   admission, rate smoothing and the stale-preparation bound
                   (Sections 4.1, 4.2 and 4.4).

It shares no code with the HIP library or its Python binding.  Inputs
(weights, ids, tables) come from the seeded generators in ``workloads``.
"""
from . import footprint, numerics, model, paged, scheduler  # noqa: F401
