"""Prefix trie of valid item identifiers (constrained generation, Sec. 3.1).

Every item is a fixed-length tuple of L codes; a partial sequence may only be
extended by a code that keeps it a prefix of some catalog item.  Plain Python:
a dict from each valid prefix (tuple of codes) to the sorted list of codes that
extend it.

Parity: pinned by tests/test_oracle_search.py (children sets against brute
force over the catalog).
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np


class Trie:
    def __init__(self, codes: np.ndarray):
        codes = np.asarray(codes)
        self.L = codes.shape[1]
        kids: Dict[Tuple[int, ...], set] = {}
        for row in codes.tolist():
            for l in range(self.L):
                kids.setdefault(tuple(row[:l]), set()).add(row[l])
        self._kids: Dict[Tuple[int, ...], List[int]] = {k: sorted(v) for k, v in kids.items()}
        self.items = {tuple(r) for r in codes.tolist()}

    def children(self, prefix: Sequence[int]) -> List[int]:
        return self._kids.get(tuple(prefix), [])

    def is_prefix(self, prefix: Sequence[int]) -> bool:
        return len(prefix) == 0 or tuple(prefix) in self._kids or tuple(prefix) in self.items
