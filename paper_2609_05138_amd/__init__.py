"""MI355X-native best-matching-unit (BMU) search for sparse binary documents.

The compute lives in ``libsom.so`` (HIP kernels for gfx950 behind the C ABI
of ``include/som.h``); ``paper_2609_05138_amd.som`` is the ctypes binding
with the same function names.  Build with ``python -m
paper_2609_05138_amd.build``.
"""

from .som import (  # noqa: F401
    SomError,
    load,
    som_abi_version,
    Plan,
    som_bmu_search,
    som_bmu_search_planned,
    som_bmu_search_top2,
    som_bmu_search_top2_planned,
    som_bmu_search_unfused,
    som_bmu_search_unfused_workspace_bytes,
    som_bmu_search_planned_workspace_bytes,
    som_bmu_workspace_bytes,
    som_group_plan,
    som_plan,
    som_cluster_order,
    som_cluster_workspace_bytes,
    som_codebook_ldw,
    som_codebook_norms,
    som_last_error,
    som_probe_read,
    som_probe_lds,
    som_tile_plan,
    som_update_accumulate,
    som_update_finish,
    som_update_workspace_bytes,
)
