"""The tie-zone rule the GPU parity tests apply (CPU): a result that differs
from the oracle's is accepted only if taking one near-tie oracle decision the
other way reproduces it.  Checked here on the oracle itself: the flip of a
decision is found when (and only when) it is inside the zone, and a result
that needs no flip, or a different one, is not explained by it."""
import numpy as np

from _gpu_common import (FlipStreams, flipped_scorer, relaxed_flips, relaxed_tie, strict_tie, env,
                         oracle_user)
from synth import philox_key
from oracle.relaxed import draft_paper, verify_paper
from oracle.search import Decision, table_scorer, verify_strict
from oracle.trie import Trie


def _table_case():
    # codebook 3, L 2, full catalog; level-1 candidates (0), (1) 1e-5 apart at the K = 1 boundary
    cb, L = 3, 2
    cat = np.array([[a, b] for a in range(cb) for b in range(cb)])
    rows = {(): np.log(np.array([0.4, 0.4 - 1e-5, 0.2 - 1e-5 + 1e-5, 1, 1, 1]))}
    rng = np.random.default_rng(0)
    for a in range(cb):
        rows[(a,)] = np.log(rng.uniform(0.1, 1.0, 2 * cb))
    return cb, L, Trie(cat), rows


def test_strict_flip_reproduces_only_near_ties():
    cb, L, trie, rows = _table_case()
    lp = table_scorer(rows)
    D = [[(0,), (1,)], [(0, 0), (1, 1)]]
    log = []
    base = verify_strict(lp, trie, [((), 0.0)], D, 1, L, cb, log)
    d0 = log[0]
    assert d0.pair == ((0,), (1,)) and 0 < d0.margin < 1e-3
    other = verify_strict(flipped_scorer(lp, d0, cb), trie, [((), 0.0)], D, 1, L, cb)
    assert [p for p, _ in other.beams] != [p for p, _ in base.beams]

    def rerun(d):
        return verify_strict(flipped_scorer(lp, d, cb), trie, [((), 0.0)], D, 1, L, cb)

    def same_as(r):
        return lambda x: [p for p, _ in x.beams] == [p for p, _ in r.beams] and x.t_after == r.t_after
    assert strict_tie(log, rerun, same_as(other)) is d0
    assert strict_tie(log, rerun, same_as(other), tie=1e-6) is None      # outside a narrower zone
    # a result no single near-tie flip produces is not explained
    fake = Decision("target_topk", 1, 0.0, ((0,), (2,)))
    third = verify_strict(flipped_scorer(lp, fake, cb), trie, [((), 0.0)], D, 1, L, cb)
    assert strict_tie(log, rerun, same_as(third)) is None


def test_relaxed_flip_finds_the_decision():
    e = env("tiny")
    w = e["w"]
    o = oracle_user("tiny", 0)
    k = philox_key(w)
    key = [int(k[0]), int(k[1])]
    rs = FlipStreams(key, 0)
    D = draft_paper(o["lq"], e["trie"], [()], [0.0], 4, w.N, w.codebook, 1.0, rs, 0)
    log = []
    base = verify_paper(o["lp"], o["lq"], e["trie"], [((), 0.0)], [0.0], D, w.K, w.L, w.codebook, 1.0, rs, 0, log)

    def rerun(uo, go):
        return verify_paper(o["lp"], o["lq"], e["trie"], [((), 0.0)], [0.0], D, w.K, w.L, w.codebook, 1.0,
                            FlipStreams(key, 0, uo, go), 0)

    def sig(r):
        return (r.t_after, r.accepted, [p for p, _ in r.beams])
    # natural margins lie outside the zone: nothing to flip
    assert list(relaxed_flips(log)) == []
    # with a zone wide enough to hold every decision, the first flip that changes
    # the result is found again from that result
    flips = list(relaxed_flips(log, tie=1e9))
    assert flips
    target = None
    for m, uo, go in flips:
        r = rerun(uo, go)
        if sig(r) != sig(base):
            target = r
            break
    assert target is not None
    assert relaxed_tie(log, rerun, lambda r: sig(r) == sig(target), tie=1e9) is not None
    assert relaxed_tie(log, rerun, lambda r: sig(r) == sig(target)) is None
