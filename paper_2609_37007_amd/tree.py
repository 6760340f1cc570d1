"""Sparse draft trees: greedy calibration and packing (Sec. 2.2, Fig. 2).

A tree node is a path of candidate ranks (r_1, ..., r_d): the rank-r_j candidate
of depth j's draft distribution under the rank-r_{j-1} candidate of depth j - 1,
and so on; the candidates of a depth are shared by every parent. The paper grows
the tree greedily from per-depth, per-rank acceptance statistics measured on a
calibration set: at each step it adds the node with the largest expected
contribution to the accepted prefix length, until the node budget N, with depth
at most K. A node's contribution is the probability that its whole path is
accepted, the product of P[depth][rank] along the path (acceptances taken as
independent, the usual calibration approximation). Since a child never
contributes more than its parent, the N best nodes form a tree, and greedy
growth finds them.

Packing (Fig. 2): the root (the committed token's row) is row 0, then the nodes
breadth first -- by depth, then by parent row, then by rank -- so that parents
precede children and a frame's end truncates the rows to a prefix. The packed
form is (parents, ranks) for rows 1..N, as the library's tree configuration and
the oracle take it.

This module is offline tooling: it produces the tree a model is created with.
"""
from __future__ import annotations

import heapq
import json
import math

import numpy as np


def greedy_tree(P, N: int, K: int | None = None):
    """The N-node tree of largest sum of path acceptance probabilities.

    P[d - 1][r]: probability that the rank-r candidate at depth d is accepted when its
    parent was. Ties go to the shallower node, then the lexicographically smaller rank
    path. Returns the rank paths in the order they were added."""
    P = [list(map(float, row)) for row in P]
    K = len(P) if K is None else min(K, len(P))
    heap = [(-P[0][r], 1, (r,)) for r in range(len(P[0]))] if K >= 1 else []
    heapq.heapify(heap)
    chosen = []
    while heap and len(chosen) < N:
        negv, d, path = heapq.heappop(heap)
        chosen.append(path)
        if d < K:
            for r in range(len(P[d])):
                heapq.heappush(heap, (negv * P[d][r], d + 1, path + (r,)))
    return chosen


def path_value(P, path) -> float:
    return math.prod(float(P[d][r]) for d, r in enumerate(path))


def pack(paths):
    """Breadth-first packing of rank paths: (parents, ranks) of rows 1..N."""
    paths = [tuple(p) for p in paths]
    have = set(paths)
    for p in paths:
        if len(p) == 0 or (len(p) > 1 and p[:-1] not in have):
            raise ValueError(f"path {p} has no parent in the tree")
    if len(have) != len(paths):
        raise ValueError("duplicate path")
    row_of = {(): 0}
    order = []
    for d in range(1, max((len(p) for p in paths), default=0) + 1):
        level = sorted((p for p in paths if len(p) == d), key=lambda p: (row_of[p[:-1]], p[-1]))
        for p in level:
            row_of[p] = len(order) + 1
            order.append(p)
    parents = [row_of[p[:-1]] for p in order]
    ranks = [p[-1] for p in order]
    return parents, ranks


def unpack(parents, ranks):
    """Rank paths of packed rows 1..N."""
    paths = [()]
    for par, r in zip(parents, ranks):
        paths.append(paths[par] + (int(r),))
    return paths[1:]


def expected_accepted(P, paths) -> float:
    """Expected accepted nodes per round under the calibration approximation."""
    return sum(path_value(P, p) for p in paths)


def rank_statistics(dec, hs, codes, offsets, topk: int, T: float, K: int, R: int):
    """P[d - 1][r] estimated from teacher-forced samples: the share of anchors k (1 <= k,
    k + d <= n) at which the code that followed at k + d was the rank-r candidate of
    q_{k+d} = topk-softmax(LMH_{k+d}(h_k + b_d) / T). dec: paper_2609_37007_amd.offsets.Decoder;
    hs: final-normed hidden states [F][n + 1][H]; codes [F][n + 1] (c_0 .. c_n)."""
    torch = dec.torch
    n = dec.s.n_codes
    b = torch.as_tensor(np.ascontiguousarray(offsets, dtype=np.float32), device=hs.device)
    hits = np.zeros((K, R))
    tot = np.zeros(K)
    with torch.no_grad():
        for d in range(1, K + 1):
            for k in range(1, n - d + 1):
                lg = (hs[:, k] + b[d - 1]) @ dec.W[f"lmh{k + d}"].T
                order = torch.argsort(-lg, dim=-1, stable=True)[:, :min(R, topk)]
                match = (order == codes[:, k + d][:, None]).cpu().numpy()
                hits[d - 1, :match.shape[1]] += match.sum(0)
                tot[d - 1] += match.shape[0]
    return hits / np.maximum(tot, 1)[:, None]


def save(path, parents, ranks, **meta):
    with open(path, "w") as fh:
        json.dump(dict(n_nodes=len(parents), parents=list(map(int, parents)), ranks=list(map(int, ranks)), **meta),
                  fh, indent=1)


def load(path):
    with open(path) as fh:
        d = json.load(fh)
    return d["parents"], d["ranks"]


def calibrate(workload: str = "mcd1024", frames: int = 2048, depth: int = 4, ranks: int = 8, nodes=(16,),
              offsets: str = "seed", seed: int = 0, device=None, log=print, head_scale: float = 1.0):
    """Rank statistics of the model's own top-k samples (the stand-in for the paper's
    calibration set) and the greedy tree of every node budget in `nodes`."""
    import torch

    from paper_2609_37007_amd import offsets as OF
    from paper_2609_37007_amd import synth as S

    shape_name, topk = OF.WORKLOADS[workload]
    s = getattr(S, shape_name)
    if offsets == "seed":
        blob = S.make_weights(s, seed=0, head_scale=head_scale)
    elif offsets == "zero":
        blob = S.make_weights(s, seed=0, head_scale=head_scale, offsets=np.zeros((s.max_draft, s.hidden)))
    else:
        blob = S.make_weights(s, seed=0, head_scale=head_scale, offsets=np.load(offsets, allow_pickle=False))
    dev = torch.device(device or ("cuda" if torch.cuda.is_available() else "cpu"))
    dec = OF.Decoder(s, blob, dev)
    f, c0 = S.frame_inputs(s, frames, seed_hidden=seed + 60, seed_c0=seed + 61)
    gen = torch.Generator(device=dev).manual_seed(seed + 62)
    with torch.no_grad():
        fT = torch.from_numpy(f).to(dev)
        cT = torch.from_numpy(c0.astype(np.int64)).to(dev)
        codes, hs = [], []
        for a in range(0, frames, 512):
            c = dec.sample_frames(fT[a:a + 512], cT[a:a + 512], topk, 0.9, gen)
            codes.append(c)
            hs.append(dec.forward(dec.inputs(fT[a:a + 512], c[:, :-1])))
        codes, hs = torch.cat(codes), torch.cat(hs)
    P = rank_statistics(dec, hs, codes, S.unpack_weights(s, blob)["offsets"], topk, 0.9, depth, ranks)
    log("acceptance by depth (rows) and rank (columns):\n" + np.array2string(P, precision=4))
    trees = {}
    for N in nodes:
        paths = greedy_tree(P, N, depth)
        parents, rks = pack(paths)
        trees[N] = dict(parents=parents, ranks=rks, expected_accepted=expected_accepted(P, paths))
    return P, trees


def main(argv=None):
    import argparse
    import os
    ap = argparse.ArgumentParser(description="Greedy sparse-tree calibration from the model's own samples")
    ap.add_argument("--workload", default="mcd1024")
    ap.add_argument("--frames", type=int, default=2048)
    ap.add_argument("--depth", type=int, default=4)
    ap.add_argument("--ranks", type=int, default=8)
    ap.add_argument("--nodes", default="4,8,16,32,48,64")
    ap.add_argument("--offsets", default="seed")
    ap.add_argument("--head-scale", type=float, default=1.0)
    ap.add_argument("--out-dir", required=True)
    a = ap.parse_args(argv)
    nodes = [int(x) for x in a.nodes.split(",")]
    P, trees = calibrate(a.workload, a.frames, a.depth, a.ranks, nodes, a.offsets, head_scale=a.head_scale)
    os.makedirs(a.out_dir, exist_ok=True)
    for N, t in trees.items():
        tag = "" if a.head_scale == 1.0 else f"_h{a.head_scale:g}"
        path = os.path.join(a.out_dir, f"tree_{a.workload}{tag}_n{N}.json")
        save(path, t["parents"], t["ranks"], workload=a.workload, depth=a.depth, frames=a.frames,
             offsets=a.offsets, head_scale=a.head_scale, expected_accepted=t["expected_accepted"],
             acceptance=P.tolist())
        print(f"N = {N}: expected accepted nodes per round {t['expected_accepted']:.4f} -> {path}")
    return 0


if __name__ == "__main__":
    import sys
    sys.exit(main())
