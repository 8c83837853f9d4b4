"""CPU oracle for the best-matching-unit search -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously correct fp64 numpy code written from the paper's
definition of the search.  Only the tests, the package's smoke check and the
benchmark's CPU-baseline leg may import it; the product path never does, and
this package imports nothing from the product (the HIP library or its
binding).  It shares no code, tables or helpers with the GPU path.

Parity status of each function is stated in its module docstring.
"""

from .bmu import (  # noqa: F401
    codebook_norms,
    codebook_norms_blocks,
    doc_distances,
    bmu_search,
    bmu_search_exact,
    bmu_search_dense,
    bmu_search_tiled,
    tile_union,
    cluster_order,
    accept_bmu,
    accept_top2,
)
from .update import (  # noqa: F401
    neighbourhood,
    neighbourhood_radius,
    update_accumulate,
    update_finish,
    update_finish_at,
)
