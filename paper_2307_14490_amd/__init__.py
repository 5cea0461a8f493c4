"""MI355X-native training step of HUGE (KDD'23): skip-gram negative sampling
over (source_id, destination_id, co_counts) batches, in hand-written HIP
kernels behind the C ABI of ``include/huge.h``, the random-walk sampler
that produces those batches on the GPU, and the unsupervised evaluation of
the trained embeddings (edge SNR, distance percentiles, sampled recall).

``binding`` is the ctypes layer; ``build`` compiles ``libhuge.so`` in-tree.
"""
from .binding import (  # noqa: F401
    EXPORTED,
    Evaluator,
    HUGE_NEG_ALIAS,
    HUGE_NEG_UNIFORM,
    HUGE_SCATTER_ATOMIC,
    HUGE_SCATTER_SORTED,
    HugeConfig,
    HugeError,
    HugeWalkConfig,
    Trainer,
    build_alias,
    cocount_weights,
    load,
    make_config,
    sample_walks,
    status_string,
    walk_config,
    workspace_bytes,
)
