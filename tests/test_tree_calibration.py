"""Greedy sparse-tree calibration and breadth-first packing (Sec. 2.2, Fig. 2), on the CPU.

The greedy tree is checked against brute force over every tree of the same size on
small acceptance tables (the largest sum of path probabilities), and the packing
against the Fig. 2 example."""
import itertools
import json
import os

import numpy as np
import pytest

from paper_2609_37007_amd import tree as T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _all_trees(K, R, N):
    nodes = [p for d in range(1, K + 1) for p in itertools.product(range(R), repeat=d)]
    for sub in itertools.combinations(nodes, N):
        s = set(sub)
        if all(len(p) == 1 or p[:-1] in s for p in sub):
            yield sub


@pytest.mark.parametrize("seed", range(6))
def test_greedy_tree_is_the_best_tree_of_its_size(seed):
    rng = np.random.default_rng(seed)
    K, R = 3, 3
    P = np.sort(rng.random((K, R)) * 0.6, axis=1)[:, ::-1]  # rank 0 likeliest, as a draft's ranks are
    for N in range(1, 7):
        g = T.greedy_tree(P, N, K)
        assert len(g) == N and len(set(g)) == N
        best = max(T.expected_accepted(P, t) for t in _all_trees(K, R, N))
        assert abs(T.expected_accepted(P, g) - best) < 1e-12
        parents, ranks = T.pack(g)
        assert sorted(T.unpack(parents, ranks)) == sorted(g)


def test_greedy_respects_the_depth_cap_and_budget():
    P = [[0.9, 0.5], [0.9, 0.5], [0.9, 0.5], [0.9, 0.5]]
    g = T.greedy_tree(P, 5, K=2)
    assert max(len(p) for p in g) <= 2 and len(g) == 5
    assert T.greedy_tree(P, 100, K=2) and len(T.greedy_tree(P, 100, K=2)) == 2 + 4


def test_packing_reproduces_fig2():
    with open(os.path.join(GOLDEN, "fig2_sparse_tree.json")) as fh:
        g = json.load(fh)
    # Fig. 2's tree as rank paths: t1 = (0), t2 = (1), t3 = (0,0), t4 = (0,1), t3 = (1,0),
    # t5 = (0,0,0), t5 = (1,0,0), t6 = (1,0,1)
    paths = [(1, 0, 1), (0,), (1, 0, 0), (0, 1), (1,), (0, 0), (1, 0), (0, 0, 0)]
    parents, ranks = T.pack(paths)
    anc = [[0]]
    for r, p in enumerate(parents, start=1):
        anc.append(sorted(set(anc[p]) | {r}))
    assert anc == g["ancestors"]
    assert ranks == [0, 1, 0, 1, 0, 0, 0, 1]


def test_pack_rejects_orphans_and_duplicates():
    with pytest.raises(ValueError):
        T.pack([(0, 1)])
    with pytest.raises(ValueError):
        T.pack([(0,), (0,)])
