"""Constrained beam search, drafting and strict top-K verification (fp64).

Definitions followed:

* Target-only constrained beam search (task formulation, Sec. 2): start from
  the empty sequence with score 0; at each of the L levels extend every beam by
  every trie-valid code, score a sequence by its cumulative log-probability
  S(s·c) = S(s) + log p(c | x, s), keep the K best.  Ties are broken by the
  lexicographically smaller code sequence (the paper is silent on ties).
* Drafting (Eq. 1): the draft runs the same beam search with width N for
  gamma levels, starting from the current target beams Y_t scored by the
  draft; level j keeps TopN of the extensions of level j-1.
* Strict top-K verification (Algorithm 1, Sec. 2): at level j the target's
  TopK is taken over the extensions of the target beams accepted at level j-1
  (reading: only these keep the result identical to target beam search, the
  losslessness claim of Sec. 4.2); the level is accepted when that TopK is a
  subset of the drafted level; verification stops at the first rejection and
  outputs the target's TopK of that level.  If every drafted level is
  accepted and the item is not complete, one more level is taken from the
  target (the p_{gamma+1} term of Algorithm 1).  The level that completes the
  item is the target's whatever the test says.
* Log-probabilities are normalised over the item-token columns of the
  vocabulary; trie-invalid codes are dropped without renormalising.

Scores are fp64.  Every top-n decision records its margin (the n-th score
minus the (n+1)-th) and the two sequences it separates, so that a GPU result
can be compared outside ties.

Parity: beam search pinned by brute-force enumeration of the catalog and a
hand-worked table example; the speculative loop pinned by the losslessness
invariant (equal to target beam search for any draft) and by the all-accept
special cases (tests/test_oracle_search.py).  Accepted lengths and the level
reached are pinned against their definition through the enumeration-pinned
beam search: level t+i is accepted while the target's own TopK at that level
lies inside drafted level i, then one target level follows (up to L); checked
under natural drafts and under drafts that drop one target path at a chosen
level, the item-completing level included.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

from .model import Decoder, PrefixCache, item_log_softmax

Path = Tuple[int, ...]
Beam = Tuple[Path, float]


class Scorer:
    """Memoised item log-probs of one model for one user: lp(path) -> [n_item]."""

    def __init__(self, fn: Callable[[List[Path]], np.ndarray]):
        self._fn = fn
        self._memo: Dict[Path, np.ndarray] = {}
        self.calls = 0

    def __call__(self, paths: Sequence[Path]) -> List[np.ndarray]:
        miss = [p for p in dict.fromkeys(paths) if p not in self._memo]
        if miss:
            self.calls += 1
            out = self._fn(miss)
            for p, row in zip(miss, out):
                self._memo[p] = row
        return [self._memo[p] for p in paths]


def model_scorer(dec: Decoder, cache: PrefixCache, item_base: int, codebook: int) -> Scorer:
    def fn(paths):
        toks = [tuple(item_base + codebook * l + c for l, c in enumerate(p)) for p in paths]
        return item_log_softmax(dec.path_logits(cache, toks))
    return Scorer(fn)


def table_scorer(table: Dict[Path, np.ndarray]) -> Scorer:
    return Scorer(lambda paths: np.stack([np.asarray(table[p], dtype=np.float64) for p in paths]))


@dataclasses.dataclass
class Decision:
    kind: str      # "target_topk", "draft_topn"
    level: int     # item level (1-based depth of the selected sequences)
    margin: float  # n-th minus (n+1)-th score; inf if no (n+1)-th candidate
    pair: Optional[Tuple[Path, Path]] = None   # (n-th selected, (n+1)-th) sequences


def extend(beams: Sequence[Beam], lp: Scorer, trie, codebook: int) -> List[Beam]:
    """All trie-valid one-code extensions of ``beams`` with cumulative scores."""
    rows = lp([p for p, _ in beams])
    out = []
    for (p, s), row in zip(beams, rows):
        col0 = codebook * len(p)
        for c in trie.children(p):
            out.append((p + (c,), s + float(row[col0 + c])))
    return out


def top_boundary(cands: List[Beam], n: int) -> Tuple[List[Beam], float, Optional[Tuple[Path, Path]]]:
    """The n best by score (ties: lexicographically smaller path first), the
    margin and the pair of sequences the margin separates."""
    srt = sorted(cands, key=lambda b: (-b[1], b[0]))
    if len(srt) > n:
        return srt[:n], srt[n - 1][1] - srt[n][1], (srt[n - 1][0], srt[n][0])
    return srt[:n], float("inf"), None


def top(cands: List[Beam], n: int) -> Tuple[List[Beam], float]:
    """The n best by score (ties: lexicographically smaller path first) and the margin."""
    sel, margin, _ = top_boundary(cands, n)
    return sel, margin


def beam_search(lp: Scorer, trie, K: int, L: int, codebook: int,
                log: Optional[List[Decision]] = None) -> List[List[Beam]]:
    """Target-only constrained beam search; returns the beams of every level 1..L."""
    beams: List[Beam] = [((), 0.0)]
    levels = []
    for lvl in range(1, L + 1):
        beams, m, pr = top_boundary(extend(beams, lp, trie, codebook), K)
        if log is not None:
            log.append(Decision("target_topk", lvl, m, pr))
        levels.append(beams)
    return levels


def path_score(lp: Scorer, path: Path, codebook: int) -> float:
    rows = lp([path[:i] for i in range(len(path))])
    return float(sum(row[codebook * i + path[i]] for i, row in enumerate(rows)))


def draft_levels(lq: Scorer, trie, Y: Sequence[Path], J: int, N: int, codebook: int,
                 log: Optional[List[Decision]] = None) -> List[List[Beam]]:
    """Eq. 1: J levels of draft beam search of width N from the target beams Y."""
    cur: List[Beam] = [(p, path_score(lq, p, codebook)) for p in Y]
    t = len(Y[0]) if Y else 0
    out = []
    for j in range(1, J + 1):
        cands = extend(cur, lq, trie, codebook)
        cur, m, pr = top_boundary(cands, N)
        if log is not None:
            log.append(Decision("draft_topn", t + j, m, pr))
        out.append(cur)
    return out


@dataclasses.dataclass
class VerifyResult:
    accepted: int                 # levels accepted before the first rejection
    t_after: int
    beams: List[Beam]             # new target beams (paths at depth t_after, target scores)
    levels: List[List[Beam]]      # target TopK of every level examined


def verify_strict(lp: Scorer, trie, Y: Sequence[Beam], drafted: Sequence[Sequence[Path]],
                  K: int, L: int, codebook: int, log: Optional[List[Decision]] = None) -> VerifyResult:
    """Algorithm 1 from level t = len(path of Y) with drafted levels t+1..t+J."""
    t = len(Y[0][0])
    J = len(drafted)
    T: List[Beam] = list(Y)
    levels = []
    for j in range(1, J + 1):
        Tj, m, pr = top_boundary(extend(T, lp, trie, codebook), K)
        if log is not None:
            log.append(Decision("target_topk", t + j, m, pr))
        levels.append(Tj)
        ok = {p for p, _ in Tj} <= set(drafted[j - 1])
        if t + j == L:
            return VerifyResult(j if ok else j - 1, L, Tj, levels)
        if not ok:
            return VerifyResult(j - 1, t + j, Tj, levels)
        T = Tj
    # every drafted level accepted and the item is not complete: one target level more
    Tn, m, pr = top_boundary(extend(T, lp, trie, codebook), K)
    if log is not None:
        log.append(Decision("target_topk", t + J + 1, m, pr))
    levels.append(Tn)
    return VerifyResult(J, t + J + 1, Tn, levels)


@dataclasses.dataclass
class SDStep:
    t: int
    Y: List[Beam]                  # target beams entering the step (target scores)
    drafted: List[List[Beam]]      # draft levels t+1..t+J (draft scores)
    result: VerifyResult


def sd_decode_strict(lp: Scorer, lq: Scorer, trie, K: int, N: int, gamma: int, L: int, codebook: int,
                     log: Optional[List[Decision]] = None,
                     drafter: Optional[Callable] = None) -> Tuple[List[Beam], List[SDStep]]:
    """Speculative decoding with strict verification until the items are complete.

    ``drafter(Y_paths, J)`` may replace the draft beam search (it must return J
    levels of (path, draft score) beams, each level's parents in the previous
    level).
    """
    t = 0
    Y: List[Beam] = [((), 0.0)]
    steps = []
    while t < L:
        J = min(gamma, L - t)
        if drafter is None:
            D = draft_levels(lq, trie, [p for p, _ in Y], J, N, codebook, log)
        else:
            D = drafter([p for p, _ in Y], J)
        res = verify_strict(lp, trie, Y, [[p for p, _ in lvl] for lvl in D], K, L, codebook, log)
        steps.append(SDStep(t, list(Y), D, res))
        Y, t = res.beams, res.t_after
    return Y, steps
