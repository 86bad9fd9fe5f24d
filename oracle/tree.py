"""Flattening drafted beams into one sequence with a tree attention mask.

Tree-based attention (Sec. 3.3 and its implementation appendix): the beam
sequences of every drafted step are flattened by appending, level by level,
the tokens that are new at that level, so shared prefixes appear once (the
appendix example: beams a1 | a2, a1 b1 | a2 b2, a1 b1 c1 | a1 b1 c2 flatten to
"a1 a2 b1 b2 c1 c2").  Each row of the mask belongs to one beam sequence and
marks its own last token and the tokens preceding it in that beam.

Parity: pinned by the appendix's worked example (tests/golden/tree_example.json).
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

Path = Tuple[int, ...]


def flatten(paths: Sequence[Sequence]) -> Tuple[List[Path], List[int], List[int]]:
    """Distinct prefixes of ``paths`` ordered by depth, then first appearance.

    Returns (nodes, parent index (-1 for depth 1), depth).
    """
    first: Dict[Path, int] = {}
    order = 0
    for p in paths:
        p = tuple(p)
        for d in range(1, len(p) + 1):
            if p[:d] not in first:
                first[p[:d]] = order
                order += 1
    nodes = sorted(first, key=lambda q: (len(q), first[q]))
    index = {q: i for i, q in enumerate(nodes)}
    parent = [index[q[:-1]] if len(q) > 1 else -1 for q in nodes]
    depth = [len(q) for q in nodes]
    return nodes, parent, depth


def ancestor_mask(parent: Sequence[int]) -> np.ndarray:
    """mask[i, j] = 1 iff node j is node i or one of its ancestors."""
    n = len(parent)
    m = np.zeros((n, n), dtype=np.int8)
    for i in range(n):
        j = i
        while j >= 0:
            m[i, j] = 1
            j = parent[j]
    return m
