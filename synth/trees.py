"""Seeded sparse candidate trees with prompt-token chains.

A tree has a root (node 0: the last verified token, not yet in the KV cache),
candidate ("guess") nodes below it, and a chain of `n_prompt` prompt tokens
hung off every leaf candidate (Section 4.1: each guess token carries a sequence
of prompt tokens; the chain length bounds the next step's tree depth).  Chain
position j (1-based) uses prompt embedding j-1, i.e. the prompt token whose
token distance is j (Section 3.1).  A prompt node's id is vocab + prompt index.

Node order is topological: candidates in breadth-first order (depth, then
creation), then the chains in leaf order, so parent[i] < i for every i > 0 and
parent[0] == -1.  Sibling candidates carry distinct tokens, as top-k candidate
generation would produce.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List

import numpy as np


@dataclass
class Tree:
    parent: np.ndarray        # int32 [T]
    ids: np.ndarray           # int32 [T]; ids >= vocab are prompt tokens
    n_candidates: int         # candidates incl. the root occupy nodes [0, n_candidates)

    @property
    def T(self) -> int:
        return int(self.parent.shape[0])


def _shape_random_parents(rng, n_cand: int, max_depth: int, max_fanout: int):
    """Parent array over n_cand candidate nodes (node 0 = root), creation order."""
    parent = [-1]
    depth = [0]
    kids = [0]
    while len(parent) < n_cand:
        elig = [i for i in range(len(parent)) if depth[i] < max_depth and kids[i] < max_fanout]
        p = elig[int(rng.integers(len(elig)))]
        parent.append(p)
        depth.append(depth[p] + 1)
        kids.append(0)
        kids[p] += 1
    return parent, depth


def _shape_exact_total(rng, total: int, n_prompt: int, max_depth: int, max_fanout: int):
    """Grow candidates until candidates + n_prompt * leaves == total exactly.

    Adding a child to a leaf moves that leaf's chain to the child (+1 node);
    adding a child to an inner node adds the child and a new chain
    (+1 + n_prompt).  With remaining budget < 1 + n_prompt only leaves are
    eligible.  A dead end restarts from the root, continuing the same RNG stream.
    """
    if total < 1 + n_prompt:
        raise ValueError("total too small for a root with its prompt chain")
    while True:
        parent, depth, kids = [-1], [0], [0]
        size = 1 + n_prompt
        while size < total:
            rem = total - size
            elig = [i for i in range(len(parent))
                    if depth[i] < max_depth and kids[i] < max_fanout
                    and (kids[i] == 0 or rem >= 1 + n_prompt)]
            if not elig:
                break
            p = elig[int(rng.integers(len(elig)))]
            size += 1 if kids[p] == 0 else 1 + n_prompt
            parent.append(p)
            depth.append(depth[p] + 1)
            kids.append(0)
            kids[p] += 1
        if size == total:
            return parent, depth


def _finish(rng, parent: List[int], depth: List[int], vocab: int, n_prompt: int,
            root_token: int) -> Tree:
    n = len(parent)
    order = sorted(range(n), key=lambda i: (depth[i], i))      # BFS, root first
    new_of = {old: new for new, old in enumerate(order)}
    cparent = [-1] + [new_of[parent[old]] for old in order[1:]]
    # distinct tokens among siblings
    ids = [int(root_token)]
    used = {}
    for i in range(1, n):
        p = cparent[i]
        s = used.setdefault(p, set())
        while True:
            t = int(rng.integers(vocab))
            if t not in s:
                s.add(t)
                break
        ids.append(t)
    has_child = [False] * n
    for i in range(1, n):
        has_child[cparent[i]] = True
    par = list(cparent)
    for leaf in range(n):
        if has_child[leaf]:
            continue
        prev = leaf
        for j in range(n_prompt):
            par.append(prev)
            ids.append(vocab + j)
            prev = len(par) - 1
    return Tree(np.asarray(par, np.int32), np.asarray(ids, np.int32), n)


def make_tree(spec: str, vocab: int, n_prompt: int, max_depth: int, seed: int,
              root_token: int, max_fanout: int = 4) -> Tree:
    """spec: "candidates:<n>" (n candidates incl. root) or "total:<T>" (exact size)
    or "chain:<n>" (root + n-1 candidates in a line, plus one prompt chain)."""
    kind, val = spec.split(":")
    n = int(val)
    rng = np.random.Generator(np.random.PCG64(seed))
    if kind == "candidates":
        parent, depth = _shape_random_parents(rng, n, max_depth, max_fanout)
    elif kind == "total":
        parent, depth = _shape_exact_total(rng, n, n_prompt, max_depth, max_fanout)
    elif kind == "chain":
        parent = [-1] + list(range(n - 1))
        depth = list(range(n))
    else:
        raise ValueError(spec)
    return _finish(rng, parent, depth, vocab, n_prompt, root_token)


def tree_from_parents(parent, ids, vocab: int) -> Tree:
    parent = np.asarray(parent, np.int32)
    ids = np.asarray(ids, np.int32)
    return Tree(parent, ids, int(np.sum(ids < vocab)))


# ---------------------------------------------------------------------------
# sparse-tree templates for the next step's tree (candidate generation)

# candidate rank paths of a 15-candidate template (depth <= 3): rank r at
# depth d means "the r-th best guess for the token at depth d"
RANK_PATHS_15 = [(0,), (1,), (2,), (3,), (4,), (5,),
                 (0, 0), (0, 1), (0, 2), (1, 0), (1, 1), (2, 0),
                 (0, 0, 0), (0, 0, 1), (0, 1, 0)]


@dataclass
class Template:
    parent: np.ndarray  # int32 [T]
    kind: np.ndarray    # int32 [T]: rank (>= 0) of a candidate, or -1 - prompt id

    @property
    def T(self) -> int:
        return int(self.parent.shape[0])


def make_template(rank_paths=RANK_PATHS_15, n_prompt: int = 3, n_ept: int = 1) -> Template:
    """Root, then the candidates of `rank_paths` (each path's prefix must come
    earlier), then under the root and under every candidate n_ept parallel
    chains of n_prompt prompt tokens (chain g: prompt ids j * n_ept + g for
    j = 0 .. n_prompt - 1), in node order.  Every node carries chains, so
    whichever node is accepted, the next tree's guesses come from its own
    prompt tokens.  Default: 1 + 15 candidates, 16 chains of 3 -> T = 64."""
    parent, kind = [-1], [0]
    node_of = {(): 0}
    for path in rank_paths:
        path = tuple(path)
        parent.append(node_of[path[:-1]])
        kind.append(path[-1])
        node_of[path] = len(parent) - 1
    n_cand = len(parent)
    for c in range(n_cand):
        for g in range(n_ept):
            prev = c
            for j in range(n_prompt):
                parent.append(prev)
                kind.append(-1 - (j * n_ept + g))
                prev = len(parent) - 1
    return Template(np.asarray(parent, np.int32), np.asarray(kind, np.int32))


def template_tree(tpl: Template, ids) -> Tree:
    """The tree of a template with the given token ids."""
    n_cand = int(np.sum(tpl.kind[1:] >= 0)) + 1
    return Tree(tpl.parent.copy(), np.asarray(ids, np.int32), n_cand)


# Synthetic acceptance table for tree sizing: p[d][r] = probability that the
# true token at token distance d + 1 is the rank-r guess there.  Anchored on
# the paper's prediction accuracies with one EPT (EPT appendix, accuracy
# table: distance 1 top-1 0.472, top-5 0.771; distance 2 top-1 0.248, top-5
# 0.576).  Within a distance, ranks 1-4 share top-5 minus top-1 geometrically
# (ratio 0.6) and ranks 5-15 continue the same geometric tail; each further
# distance is the previous row scaled by the distance-2 / distance-1 top-1
# ratio.  Synthetic: no dataset is used.
PAPER_TOP1 = (0.472, 0.248)
PAPER_TOP5 = (0.771, 0.576)


def synthetic_accept_table(depth: int = 3, k: int = 16, ratio: float = 0.6):
    w = sum(ratio ** i for i in range(4))
    table = []
    for d in range(depth):
        if d < len(PAPER_TOP1):
            a = (PAPER_TOP5[d] - PAPER_TOP1[d]) / w
            row = [PAPER_TOP1[d]] + [a * ratio ** i for i in range(k - 1)]
        else:
            row = [x * PAPER_TOP1[1] / PAPER_TOP1[0] for x in table[-1]]
        table.append(row)
    return np.asarray(table, np.float64)
