"""CPU oracle for sketched multioutput split search (SketchBoost, arXiv 2211.12858).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run anything in this package.
The product path (``paper_2211_12858_amd``) never imports it, and this package
imports nothing from the product path: the two share no code, headers, tables
or helpers.  Inputs come from ``workloads`` (seeded generators holding none of
the method's arithmetic) or from the tests themselves.

Everything here is plain, slow and meant to be checked by eye against the
paper.  Floating point is accumulated in fp64 unless a step is defined to round
(the sketch columns are stored in fp32, as the device path stores them).

Modules
-------
``sketch``  column norms, Top Outputs, Random Sampling, Random Projections,
            identity (full-output) sketch and the fp32 materialisation
            (Section 3.1-3.3).
``split``   per-node histograms, split scores, best split, partition and the
            depth-wise level loop (Section 2 "Finding the tree structure",
            eq. 4; Section 3 S_G; Section 3.4 histogram algorithm).
``brute``   exact-rational brute force over every candidate split of tiny
            inputs, independent of histograms and prefix sums.
``leaf``    leaf values of a grown tree from the full gradient matrix
            (Section 2 "Finding the leaf values", eq. 3) and the per-leaf
            objective they minimise.
``boost``   loss derivatives (eq. 2) of softmax and sigmoid cross-entropy,
            the prediction update and the boosting loop (Section 2).

Parity status: every function is pinned by the non-GPU tests
(``tests/test_oracle_*.py``) except the exact values of the random draws
themselves (uniforms and projection matrices are inputs, not oracle output).
"""
from .sketch import (  # noqa: F401
    column_norms2,
    top_outputs,
    random_sampling,
    identity_sketch,
    materialise,
    random_projection,
    sparse_pi_matrix,
    sparse_projection,
    sketch,
)
from .split import (  # noqa: F401
    node_histograms,
    split_scores,
    best_split,
    partition,
    grow_tree,
    sketch_score,
)
from .brute import brute_best_split, brute_tree, exact_region_score  # noqa: F401
from .leaf import leaf_rows, leaf_values, leaf_objective  # noqa: F401
from . import boost  # noqa: F401
