"""Seeded synthetic inputs for the best-matching-unit (BMU) search.

This package only draws random numbers: codebooks and sparse binary document
batches shaped like the workloads of the paper (Zipfian term frequencies over a
fixed vocabulary, binary term vectors, map sizes 32^2 to 512^2).  It holds none
of the search's arithmetic.  Both the CPU oracle tests and the GPU benchmark
consume its output, so neither side can bias the inputs the other sees.
"""

from .corpus import (  # noqa: F401
    CONFIGS,
    Config,
    batch_sizes,
    codebook,
    codebook_rows,
    documents,
    zipf_cdf,
    topic_subsets,
)
