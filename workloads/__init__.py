"""Seeded synthetic inputs: graphs, features, GCN parameters and target nodes.

This module is shared by the tests, the benchmark and the oracle's callers.
It holds none of the explained method's arithmetic (no sampling of
coalitions, no GCN evaluation, no least squares): it only draws random
inputs with the shapes and distributions of the paper's workloads.

Graphs are simple (no self loops, no duplicate edges) and symmetric (both
directions of every undirected pair are stored), as the paper's datasets are.
They are returned as an in-CSR: the sources of the edges u -> w are
``indices[indptr[w]:indptr[w+1]]``, ascending; ``indptr`` is int64 and
``indices`` int32.  Node ids are a seeded permutation of the generation order,
so that degree does not correlate with id.
"""
from .graphs import (chung_lu_pairs, dcsbm_pairs, in_csr_from_pairs,  # noqa: F401
                     in_csr_from_directed, random_digraph)
from .params import (binary_features, tfidf_features, gaussian_features,  # noqa: F401
                     glorot_gcn, glorot_gat)
from .configs import CONFIGS, make_config, player_count  # noqa: F401
