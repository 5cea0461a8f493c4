"""Seeded synthetic inputs for the HUGE training step.

This package produces graphs, random walks and the (source_id, destination_id,
co_counts) triples that the paper's sampler emits (Sec. 3.2), plus the node
weights that define a negative distribution.  It holds none of the training
step's arithmetic: no Philox, no alias table, no loss.  Both the product path
(through the benchmark and the tests) and the CPU oracle consume its output.

Workloads (sizes from the benchmark configurations; the real-world graphs of
the paper are replaced by random graphs of the kind it uses, Sec. 4.1.1):

* ``tiny``      exact SBM, 10k nodes, whole epoch of globally aggregated pairs;
* ``medium``    exact SBM, 1M nodes, pairs from walks on the realised graph;
* ``powerlaw``  Chung-Lu, 10M nodes, exponent 2.1, annealed walks;
* ``sbm100m``   SBM, 100M nodes, annealed walks;
* ``hubstress`` Chung-Lu, 50M nodes, exponent 1.9, i.i.d. endpoint pairs,
                Zipf(1.5) co_counts capped at 1000;
* ``sbm100m_k31`` the SBM-100M graph with 31 negatives per positive (the
                number of negatives of the paper's TPU runs, Table 2).
"""
from .gen import (  # noqa: F401
    CONFIGS,
    Workload,
    aggregate_pairs,
    annealed_sbm_step,
    chung_lu_weights,
    csr_from_edges,
    make_workload,
    relabel,
    sbm_edges,
    tuples_from_walks,
    walk_csr,
    window_pairs,
)
