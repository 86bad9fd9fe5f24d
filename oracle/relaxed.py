"""Relaxed sampling verification (Sec. 3.2, Eq. 6, Algorithm 2), fp64.

Per drafted sequence y the target accepts with probability min(1, p(y)/q(y))
(accept iff r <= p(y)/q(y), r ~ U(0,1)); a rejected one is replaced by a draw
from norm(max(0, p - q)).  p and q are the sequence distributions of the
current beam-search level: for a set S of parent beams and a model M,
pi_M(c) = exp(S_M(c)/tau) / sum_{c' in ext(S)} exp(S_M(c')/tau) over the
trie-valid one-code extensions ext(S), with S_M the cumulative log-probability.

Algorithm 2 cannot be read literally (it samples K sequences but loops over K
and keeps them when more than K are accepted; Y_out is never reset; there is no
break after a rejection).  Two explicit readings are implemented:

RELAXED_EXACT (the with-replacement theory of Sec. 3.2 and its appendix):
  a level has K slots; slot k's draft y_k is drawn from pi_q over ext(S^q) where
  S^q is the distinct set of the previous level's slots (level 1: the current
  beams Y_t).  Slot k is accepted iff log u_k <= log pi_p(y_k) - log pi_q(y_k).
  If every slot is accepted the level is accepted with beams distinct(y).
  Otherwise every rejected slot is redrawn from norm(max(0, pi_p - pi_q)), the
  level's beams are the distinct slots, and the step stops.  Each slot is then
  exactly pi_p-distributed; a level is accepted with probability b^K,
  b = sum_c min(pi_p(c), pi_q(c)) = 1 - TVD (Eq. 6).

RELAXED_PAPER (Algorithm 2 with the draft keeping width N, as in the paper's
experiments):
  level j draws N distinct sequences from pi_q over ext(D_{j-1}) (Gumbel-top-N);
  each is accepted iff log u_i <= log pi_p(y_i) - log pi_q(y_i), with pi_p over
  ext(T_{j-1}) (zero outside it).  If at least K are accepted (">" read as
  ">="), K of them are kept uniformly at random and the level is accepted;
  otherwise B = K - #accepted distinct sequences are drawn from
  norm(max(0, pi_p - pi_q)) with the accepted ones zeroed (Gumbel-top-B; all
  positive ones if fewer), the level's beams are accepted + redrawn, and the
  step stops.

In both modes the level that completes the item is final whatever the test
says; when every drafted level is accepted and the item is incomplete, the next
level is drawn from pi_p (EXACT: K i.i.d. slots; PAPER: Gumbel-top-K).

Logging (paper reading): every acceptance test is recorded with its margin
|log u - (log pi_p - log pi_q)|, its Philox counter and both values, and every
Gumbel-top-k draw (drafting, the uniform K-subset, the residual redraw, the
target's bonus level) with its k + 1 best keyed candidates and their counters,
so that a GPU result that differs can be checked against the oracle with one
near-tie decision taken the other way.

Randomness: every uniform comes from Philox4x32-10 (oracle.philox) at counter
(user, step, level * 2^16 + draw, cand * 4 + tag), tag 0 draft, 1 accept,
2 subset, 3 target draw / residual; cand = (rank of the parent among the
parents of the candidate set in lexicographic order) * codebook + code, or 0 for
per-draw uniforms.  Categorical and without-replacement draws are Gumbel-max and
Gumbel-top-k (Kool et al., 2019) over log-weights.

Parity: RELAXED_EXACT is pinned by chi-square tests of its per-slot output
against pi_p, of its acceptance frequency against 1 - TVD (Eq. 6) and of its
level acceptance against (1 - TVD)^K (tests/test_oracle_relaxed.py).
RELAXED_PAPER is only approximately pi_p by construction (its accepted draws
follow min(p, q)); its parts are pinned where they reduce to a known law: with
N = K = 1 it is Leviathan et al.'s speculative sampling, whose output follows
pi_p exactly; with q = p every draft passes and the kept K are a uniform subset
of the N drafts; q = p accepts every level.  The composite law with 0 < passes
< K is pinned by its exact enumeration on a six-code level (every ordered draft
set, acceptance pattern, kept subset and residual redraw weighed by its
probability), against which the oracle's outcomes pass a chi-square test.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .philox import gumbel, philox4x32_10, uniform
from .search import Beam, Path, Scorer, VerifyResult, extend, path_score

TAG_DRAFT, TAG_ACCEPT, TAG_SUBSET, TAG_TARGET = 0, 1, 2, 3


class Streams:
    """Philox draws of one user: key (k0, k1), counter (user, step, level*2^16+draw, cand*4+tag)."""

    def __init__(self, key: Sequence[int], user: int):
        self.key = (int(key[0]), int(key[1]))
        self.user = user

    def word(self, step: int, level: int, draw: int, cand: int, tag: int) -> int:
        return philox4x32_10((self.user, step, level * 65536 + draw, cand * 4 + tag), self.key)[0]

    def u(self, step, level, draw, cand, tag) -> float:
        return uniform(self.word(step, level, draw, cand, tag))

    def g(self, step, level, draw, cand, tag) -> float:
        return gumbel(self.word(step, level, draw, cand, tag))


def cand_index(parents: Sequence[Path], codebook: int) -> Dict[Path, int]:
    """Canonical index of every one-code extension of the parents: lexicographic parent rank * codebook + code."""
    rank = {p: i for i, p in enumerate(sorted(set(parents)))}
    return {p: rank[p] * codebook for p in rank}


def level_dist(beams: Sequence[Beam], lm: Scorer, trie, codebook: int, tau: float
               ) -> Tuple[List[Path], np.ndarray, Dict[Path, float]]:
    """Candidates ext(beams), their log pi (normalised over them) and cumulative scores."""
    cands = extend(beams, lm, trie, codebook)
    paths = [c for c, _ in cands]
    s = np.array([v for _, v in cands], dtype=np.float64) / tau
    m = s.max()
    logz = m + math.log(np.exp(s - m).sum())
    return paths, s - logz, {c: v for c, v in cands}


def gumbel_argmax(paths, logw, noise) -> Path:
    """argmax of log-weight + Gumbel noise (log-weight -inf excluded); ties -> smaller path."""
    best, bv = None, -math.inf
    for p, lw in zip(paths, logw):
        if lw == -math.inf:
            continue
        v = lw + noise(p)
        if v > bv or (v == bv and best is not None and p < best):
            best, bv = p, v
    return best


def gumbel_keys(paths, logw, rs: "Streams", ctr) -> list:
    """Every candidate of positive weight as (log-weight + Gumbel, path, counter,
    Gumbel), best first (ties -> smaller path); ``ctr(path)`` is the Philox
    counter (step, level, draw, cand, tag) of its Gumbel noise.  The first k
    paths are the Gumbel-top-k draw without replacement."""
    out = []
    for p, lw in zip(paths, logw):
        if lw == -math.inf:
            continue
        c = ctr(p)
        g = rs.g(*c)
        out.append((lw + g, p, c, g))
    out.sort(key=lambda x: (-x[0], x[1]))
    return out


def _log_topk(log, kind, lvl, k, keyed):
    # the draw's decisions: the k best and the first one left out
    if log is not None:
        log.append((kind, lvl, k, keyed[:k + 1]))


# ---------------------------------------------------------------- drafting
def draft_exact(lq: Scorer, trie, Y: Sequence[Path], Yq: Sequence[float], J: int, K: int, codebook: int,
                tau: float, rs: Streams, step: int) -> List[List[Path]]:
    """J levels of K i.i.d. slots from pi_q; returns the slot lists (with repeats)."""
    t = len(Y[0]) if Y else 0
    parents: List[Beam] = list(zip(Y, Yq))
    out = []
    for j in range(1, J + 1):
        lvl = t + j
        paths, logq, _ = level_dist(parents, lq, trie, codebook, tau)
        ci = cand_index([p for p, _ in parents], codebook)
        slots = []
        for k in range(K):
            slots.append(gumbel_argmax(paths, logq, lambda c: rs.g(step, lvl, k, ci[c[:-1]] + c[-1], TAG_DRAFT)))
        out.append(slots)
        distinct = sorted(set(slots))
        parents = [(p, path_score(lq, p, codebook)) for p in distinct]
    return out


def draft_paper(lq: Scorer, trie, Y: Sequence[Path], Yq: Sequence[float], J: int, N: int, codebook: int,
                tau: float, rs: Streams, step: int, log: Optional[list] = None) -> List[List[Beam]]:
    """J levels of N distinct draws (Gumbel-top-N) from pi_q; beams carry draft scores, in draw order."""
    t = len(Y[0]) if Y else 0
    parents: List[Beam] = list(zip(Y, Yq))
    out = []
    for j in range(1, J + 1):
        lvl = t + j
        paths, logq, sq = level_dist(parents, lq, trie, codebook, tau)
        ci = cand_index([p for p, _ in parents], codebook)
        keyed = gumbel_keys(paths, logq, rs, lambda c: (step, lvl, 0, ci[c[:-1]] + c[-1], TAG_DRAFT))
        _log_topk(log, "draft", lvl, N, keyed)
        pick = [p for _, p, _, _ in keyed[:N]]
        lvl_beams = [(p, sq[p]) for p in pick]
        out.append(lvl_beams)
        parents = lvl_beams
    return out


# ---------------------------------------------------------------- verification
def _residual(paths, logp, logq_of, zero: set) -> np.ndarray:
    r = np.array([max(0.0, math.exp(lp) - math.exp(logq_of(c))) if c not in zero else 0.0
                  for c, lp in zip(paths, logp)])
    with np.errstate(divide="ignore"):
        return np.where(r > 0, np.log(np.maximum(r, 1e-300)), -math.inf)


def verify_exact(lp: Scorer, lq: Scorer, trie, Y: Sequence[Beam], Yq: Sequence[float],
                 slots: Sequence[Sequence[Path]], K: int, L: int, codebook: int, tau: float,
                 rs: Streams, step: int, log: Optional[list] = None) -> VerifyResult:
    t = len(Y[0][0])
    J = len(slots)
    T: List[Beam] = list(Y)
    Tq: List[float] = list(Yq)
    levels = []
    for j in range(1, J + 1):
        lvl = t + j
        paths, logp, sp = level_dist(T, lp, trie, codebook, tau)
        _, logq, _ = level_dist(list(zip([p for p, _ in T], Tq)), lq, trie, codebook, tau)
        ip = dict(zip(paths, logp))
        iq = dict(zip(paths, logq))
        ci = cand_index([p for p, _ in T], codebook)
        ok_all = True
        final = []
        for k, y in enumerate(slots[j - 1]):
            a = ip.get(y, -math.inf) - iq[y]
            lu = math.log(rs.u(step, lvl, k, 0, TAG_ACCEPT))
            if log is not None:
                log.append(("accept", lvl, k, abs(lu - a)))
            if lu <= a:
                final.append(y)
            else:
                ok_all = False
                final.append(None)
        if not ok_all:
            res = _residual(paths, logp, lambda c: iq[c], set())
            for k in range(len(final)):
                if final[k] is None:
                    y = gumbel_argmax(paths, res, lambda c: rs.g(step, lvl, k, ci[c[:-1]] + c[-1], TAG_TARGET))
                    final[k] = y if y is not None else slots[j - 1][k]
        if log is not None:
            log.append(("slots", lvl, list(final), ok_all))
        Tj = [(p, sp[p]) for p in sorted(set(final))]
        levels.append(Tj)
        if lvl == L:
            return VerifyResult(j if ok_all else j - 1, L, Tj, levels)
        if not ok_all:
            return VerifyResult(j - 1, lvl, Tj, levels)
        T = Tj
        Tq = [path_score(lq, p, codebook) for p, _ in T]
    lvl = t + J + 1
    paths, logp, sp = level_dist(T, lp, trie, codebook, tau)
    ci = cand_index([p for p, _ in T], codebook)
    draws = [gumbel_argmax(paths, logp, lambda c: rs.g(step, lvl, k, ci[c[:-1]] + c[-1], TAG_TARGET))
             for k in range(K)]
    Tn = [(p, sp[p]) for p in sorted(set(draws))]
    levels.append(Tn)
    return VerifyResult(J, lvl, Tn, levels)


def verify_paper(lp: Scorer, lq: Scorer, trie, Y: Sequence[Beam], Yq: Sequence[float],
                 drafted: Sequence[Sequence[Beam]], K: int, L: int, codebook: int, tau: float,
                 rs: Streams, step: int, log: Optional[list] = None) -> VerifyResult:
    t = len(Y[0][0])
    J = len(drafted)
    T: List[Beam] = list(Y)
    Dprev: List[Beam] = list(zip([p for p, _ in Y], Yq))
    levels = []
    for j in range(1, J + 1):
        lvl = t + j
        paths, logp, sp = level_dist(T, lp, trie, codebook, tau)
        qpaths, logq, _ = level_dist(Dprev, lq, trie, codebook, tau)
        ip = dict(zip(paths, logp))
        iq = dict(zip(qpaths, logq))
        acc = []
        for i, (y, _) in enumerate(drafted[j - 1]):
            a = ip.get(y, -math.inf) - iq[y]
            ctr = (step, lvl, i, 0, TAG_ACCEPT)
            lu = math.log(rs.u(*ctr))
            if log is not None:
                log.append(("accept", lvl, i, abs(lu - a) if a > -math.inf else math.inf, ctr, a, lu))
            if lu <= a:
                acc.append((i, y))
        if len(acc) >= K:
            # K of the accepted, uniformly: Gumbel-top-K over equal weights
            draw_of = {y: i for i, y in acc}
            keyed = gumbel_keys([y for _, y in acc], [0.0] * len(acc), rs,
                                lambda y: (step, lvl, draw_of[y], 0, TAG_SUBSET))
            _log_topk(log, "subset", lvl, K, keyed)
            Tj = [(p, sp[p]) for p in sorted(y for _, y, _, _ in keyed[:K])]
            ok = True
        else:
            ci = cand_index([p for p, _ in T], codebook)
            zero = {y for _, y in acc}
            res = _residual(paths, logp, lambda c: iq.get(c, -math.inf), zero)
            keyed = gumbel_keys(paths, res, rs, lambda c: (step, lvl, 0, ci[c[:-1]] + c[-1], TAG_TARGET))
            _log_topk(log, "residual", lvl, K - len(acc), keyed)
            extra = [p for _, p, _, _ in keyed[:K - len(acc)]]
            Tj = [(p, sp[p]) for p in sorted(zero | set(extra))]
            ok = False
        levels.append(Tj)
        if lvl == L:
            return VerifyResult(j if ok else j - 1, L, Tj, levels)
        if not ok:
            return VerifyResult(j - 1, lvl, Tj, levels)
        T = Tj
        Dprev = list(drafted[j - 1])
    lvl = t + J + 1
    paths, logp, sp = level_dist(T, lp, trie, codebook, tau)
    ci = cand_index([p for p, _ in T], codebook)
    keyed = gumbel_keys(paths, logp, rs, lambda c: (step, lvl, 0, ci[c[:-1]] + c[-1], TAG_TARGET))
    _log_topk(log, "target_draw", lvl, K, keyed)
    Tn = [(p, sp[p]) for p in sorted(p for _, p, _, _ in keyed[:K])]
    levels.append(Tn)
    return VerifyResult(J, lvl, Tn, levels)


def sd_decode_relaxed(mode: str, lp: Scorer, lq: Scorer, trie, K: int, N: int, gamma: int, L: int,
                      codebook: int, tau: float, key, user: int, log: Optional[list] = None):
    """Speculative decoding with relaxed verification until the items are complete."""
    rs = Streams(key, user)
    t, step = 0, 0
    Y: List[Beam] = [((), 0.0)]
    steps = []
    while t < L:
        J = min(gamma, L - t)
        Yp = [p for p, _ in Y]
        Yq = [path_score(lq, p, codebook) for p in Yp]
        if mode == "relaxed_exact":
            D = draft_exact(lq, trie, Yp, Yq, J, K, codebook, tau, rs, step)
            res = verify_exact(lp, lq, trie, Y, Yq, D, K, L, codebook, tau, rs, step, log)
        else:
            D = draft_paper(lq, trie, Yp, Yq, J, N, codebook, tau, rs, step)
            res = verify_paper(lp, lq, trie, Y, Yq, D, K, L, codebook, tau, rs, step, log)
        steps.append((t, D, res))
        Y, t = res.beams, res.t_after
        step += 1
    return Y, steps
