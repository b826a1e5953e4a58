"""Plain fp64 CPU oracle for the GNNShap coalition-evaluation path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
library (``paper_2401_04829_amd``) never imports it and shares no code with it.

Every function follows a passage of the GNNShap paper (Akkas & Azad, arXiv
2401.04829) and is written for a reader to check by eye, not for speed:

* ``philox``   - Philox4x32-10 counter-based generator (Salmon et al., SC'11).
* ``sampler``  - the coalition sampler: size classes and quotas (eq. 4-6),
                 surplus redistribution and enumeration of small sizes
                 (Sec. 3.3.1, Alg. 2), lexicographic unranking and random
                 c-subsets (Sec. 3.3.2, Alg. 3), complement pairing (App. C.1).
* ``subgraph`` - the pruned computational graph (Sec. 3.2, App. A).
* ``gcn``      - the coalition game f(S): a GCN run on the computational graph
                 with only the coalition's edges present (Sec. 2.2, 3.4, 4.2);
                 ``values_many`` evaluates the same formula over a batch of
                 coalitions for the large workloads.
* ``wls``      - the constrained Kernel-SHAP weighted least squares
                 (eq. 2-3, Alg. 1 step 5, Sec. 3.5); ``kernel_shap_normal``
                 solves the same problem through its normal equations when
                 the rows are too many for the SVD.
* ``shapley``  - exact Shapley values by eq. 1 (brute force, small games).
* ``explain``  - Alg. 1 end to end for one target node.

All floating point is fp64.  Inputs (graph, features, weights) are fp32 values
produced by ``workloads`` and are widened to fp64 here.
"""
from . import philox, sampler, subgraph, gcn, wls, shapley, explain  # noqa: F401
