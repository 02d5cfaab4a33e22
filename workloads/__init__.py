"""Seeded synthetic DNN-shaped training graphs (inputs only, no method arithmetic).

Both the oracle side and the HIP side read the arrays these generators return;
nothing here computes levels, t/b-levels, paths or label sums.
"""
from .graphs import (  # noqa: F401
    SEED_BASE,
    SynthGraph,
    MoveSchedule,
    config0,
    config1,
    config2,
    config3,
    config4_moves,
    make_config,
    materialize_placements,
    random_dag,
    chain_graph,
    layered_dag,
    long_edge_dag,
    node_kinds,
    path_clusters,
)
