"""Pins of the oracle's Backbone Expansion tree (Section 2.2): hand-worked
golden cases and structural invariants over random candidate lists."""
import json
import os

import numpy as np
import pytest

from tests.treecheck import check_tree

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tree_backbone_n3_k2.json")


def test_golden_trees(feo):
    for case in json.load(open(GOLDEN))["cases"]:
        N, k = case["n_layers"], case["topk"]
        tr = feo.build_tree(N, k, np.array([case["root_token"]]),
                            np.array([case["topk_ids"]]), np.array([case["prefix_len"]]))
        for key in ("tokens", "parents", "depth", "positions", "mask", "retrieve"):
            np.testing.assert_array_equal(tr[key][0], np.array(case[key]), err_msg=key)


@pytest.mark.parametrize("N,k", [(1, 1), (1, 5), (2, 3), (5, 8), (7, 8), (5, 10), (4, 1), (3, 16)])
def test_tree_invariants(feo, N, k):
    rng = np.random.default_rng(N * 100 + k)
    B = 3
    roots = rng.integers(0, 1000, B).astype(np.int32)
    ids = np.stack([np.stack([rng.choice(1000, k, replace=False) for _ in range(N)])
                    for _ in range(B)]).astype(np.int32)
    P = rng.integers(0, 9000, B).astype(np.int32)
    tr = feo.build_tree(N, k, roots, ids, P)
    T = 1 + N * k
    assert tr["tokens"].shape == (B, T)
    for b in range(B):
        check_tree(tr, b, N, k, roots[b], ids[b], P[b])
