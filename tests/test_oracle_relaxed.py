"""Pins for the oracle's relaxed sampling verification (CPU).

Output law (speculative sampling, Leviathan et al. A.1, as restated in the
relaxed-verification appendix): every RELAXED_EXACT slot is distributed as the
target's level distribution pi_p; a slot is accepted with probability
b = sum min(pi_p, pi_q) = 1 - TVD (Eq. 6); a level with K slots is accepted with
probability b^K.  Small table scorers keep the Philox-driven runs fast.
"""
import math

import numpy as np
import pytest

from oracle.relaxed import Streams, draft_exact, draft_paper, level_dist, verify_exact, verify_paper
from oracle.search import table_scorer
from oracle.trie import Trie

CB, L = 4, 2


def _tables(seed, same=False):
    rng = np.random.default_rng(seed)
    def tab():
        t = {(): np.log(rng.dirichlet(np.ones(CB)))}
        for c in range(CB):
            t[(c,)] = np.concatenate([np.full(CB, -50.0), np.log(rng.dirichlet(np.ones(CB) * 0.7))])
        for k in t:
            if len(t[k]) == CB:
                t[k] = np.concatenate([t[k], np.full(CB, -50.0)])
        return t
    tp = tab()
    tq = tp if same else tab()
    return table_scorer(tp), table_scorer(tq)


def _run_exact(lp, lq, trie, K, runs):
    slots1, acc_slots, acc_levels, n_slots = [], 0, 0, 0
    for r in range(runs):
        rs = Streams((r, 12345), 0)
        D = draft_exact(lq, trie, [()], [0.0], 2, K, CB, 1.0, rs, 0)
        log = []
        verify_exact(lp, lq, trie, [((), 0.0)], [0.0], D, K, L, CB, 1.0, rs, 0, log)
        lvl1 = [e for e in log if e[0] == "slots" and e[1] == 1][0]
        slots1.extend(lvl1[2])
        acc_levels += int(lvl1[3])
        n_slots += K
    return slots1, acc_levels


def test_exact_slots_follow_target_distribution():
    trie = Trie(np.array([[a, b] for a in range(CB) for b in range(CB)]))
    lp, lq = _tables(1)
    K, runs = 2, 6000
    paths, logp, _ = level_dist([((), 0.0)], lp, trie, CB, 1.0)
    _, logq, _ = level_dist([((), 0.0)], lq, trie, CB, 1.0)
    p, q = np.exp(logp), np.exp(logq)
    slots1, acc_levels = _run_exact(lp, lq, trie, K, runs)
    counts = np.array([sum(1 for s in slots1 if s == c) for c in paths], dtype=float)
    n = counts.sum()
    chi2 = float(((counts - n * p) ** 2 / (n * p)).sum())
    # chi-square with 3 dof, alpha = 1e-3: 16.27
    assert chi2 < 16.27, (counts / n, p)
    # the draft is not the target: without the correction the slots would follow q
    chi2_q = float(((counts - n * q) ** 2 / (n * q)).sum())
    assert chi2_q > 16.27
    # level acceptance = b^K with b = sum min(p, q) = 1 - TVD (Eq. 6); 99.9% normal interval
    b = float(np.minimum(p, q).sum())
    assert abs(b - (1 - 0.5 * np.abs(p - q).sum())) < 1e-12
    pk = b ** K
    se = math.sqrt(pk * (1 - pk) / runs)
    assert abs(acc_levels / runs - pk) < 3.3 * se, (acc_levels / runs, pk)


def test_exact_slot_acceptance_rate_is_one_minus_tvd():
    trie = Trie(np.array([[a, b] for a in range(CB) for b in range(CB)]))
    lp, lq = _tables(2)
    paths, logp, _ = level_dist([((), 0.0)], lp, trie, CB, 1.0)
    _, logq, _ = level_dist([((), 0.0)], lq, trie, CB, 1.0)
    b = float(np.minimum(np.exp(logp), np.exp(logq)).sum())
    runs, K, acc = 4000, 3, 0
    for r in range(runs):
        rs = Streams((r, 777), 1)
        D = draft_exact(lq, trie, [()], [0.0], 1, K, CB, 1.0, rs, 0)
        for k, y in enumerate(D[0]):
            i = paths.index(y)
            acc += math.log(rs.u(0, 1, k, 0, 1)) <= logp[i] - logq[i]
    n = runs * K
    se = math.sqrt(b * (1 - b) / n)
    assert abs(acc / n - b) < 3.3 * se, (acc / n, b)


def test_identical_draft_accepts_every_level():
    trie = Trie(np.array([[a, b] for a in range(CB) for b in range(CB)]))
    lp, _ = _tables(3)
    for r in range(50):
        rs = Streams((r, 1), 0)
        D = draft_exact(lp, trie, [()], [0.0], 2, 3, CB, 1.0, rs, 0)
        res = verify_exact(lp, lp, trie, [((), 0.0)], [0.0], D, 3, L, CB, 1.0, rs, 0)
        assert res.accepted == 2 and res.t_after == 2
        # PAPER mode: with N = K the kept beams are the drafted ones, so pi_p and
        # pi_q share their candidate sets and q = p accepts every level
        Dp = draft_paper(lp, trie, [()], [0.0], 2, 2, CB, 1.0, rs, 0)
        res = verify_paper(lp, lp, trie, [((), 0.0)], [0.0], Dp, 2, L, CB, 1.0, rs, 0)
        assert res.accepted == 2 and res.t_after == 2


def test_paper_mode_outputs_valid_distinct_beams():
    trie = Trie(np.array([[a, b] for a in range(CB) for b in range(CB) if (a + b) % 3]))
    lp, lq = _tables(4)
    for r in range(200):
        rs = Streams((r, 9), 2)
        D = draft_paper(lq, trie, [()], [0.0], 2, 3, CB, 1.0, rs, 0)
        assert all(len(set(p for p, _ in lvl)) == len(lvl) for lvl in D)
        res = verify_paper(lp, lq, trie, [((), 0.0)], [0.0], D, 2, L, CB, 1.0, rs, 0)
        paths = [p for p, _ in res.beams]
        assert len(paths) == len(set(paths)) <= 2
        assert all(trie.is_prefix(p) for p in paths)
        assert res.t_after == len(paths[0]) and 0 <= res.accepted <= res.t_after


def test_paper_mode_with_one_draft_is_speculative_sampling():
    """RELAXED_PAPER with N = K = 1 and one drafted level is the speculative
    sampling of Leviathan et al.: one draft from pi_q, kept with probability
    min(1, pi_p / pi_q), else one draw from norm(max(0, pi_p - pi_q)).  Its output
    then follows pi_p exactly (their Theorem), and not pi_q.  A flipped
    acceptance ratio, a residual of pi_q - pi_p or a draft from pi_p each break
    one of the two chi-square checks."""
    trie = Trie(np.array([[a, b] for a in range(CB) for b in range(CB)]))
    lp, lq = _tables(1)
    paths, logp, _ = level_dist([((), 0.0)], lp, trie, CB, 1.0)
    _, logq, _ = level_dist([((), 0.0)], lq, trie, CB, 1.0)
    p, q = np.exp(logp), np.exp(logq)
    runs = 6000
    counts = np.zeros(len(paths))
    for r in range(runs):
        rs = Streams((r, 4242), 0)
        D = draft_paper(lq, trie, [()], [0.0], 1, 1, CB, 1.0, rs, 0)
        res = verify_paper(lp, lq, trie, [((), 0.0)], [0.0], D, 1, L, CB, 1.0, rs, 0)
        lvl1 = res.levels[0]
        assert len(lvl1) == 1
        counts[paths.index(lvl1[0][0])] += 1
    chi2_p = float(((counts - runs * p) ** 2 / (runs * p)).sum())
    chi2_q = float(((counts - runs * q) ** 2 / (runs * q)).sum())
    # chi-square with 3 dof, alpha = 1e-3: 16.27
    assert chi2_p < 16.27, (counts / runs, p)
    assert chi2_q > 16.27, (counts / runs, q)


def test_paper_mode_keeps_a_uniform_subset_when_k_pass():
    """With q = p every one of the N distinct drafts passes (pi_p / pi_q = 1), so
    the reading of Alg. 2 keeps K of them uniformly at random: over the C(N, K)
    subsets of draft positions the counts are uniform (keeping the first K
    drawn, or the K best-scored, fails)."""
    trie = Trie(np.array([[a, b] for a in range(CB) for b in range(CB)]))
    lp, _ = _tables(5)
    N, K, runs = 3, 2, 3000
    counts = {}
    for r in range(runs):
        rs = Streams((r, 99), 0)
        D = draft_paper(lp, trie, [()], [0.0], 1, N, CB, 1.0, rs, 0)
        res = verify_paper(lp, lp, trie, [((), 0.0)], [0.0], D, K, L, CB, 1.0, rs, 0)
        assert res.accepted == 1
        drafted = [p for p, _ in D[0]]
        kept = frozenset(drafted.index(p) for p, _ in res.levels[0])
        assert len(kept) == K
        counts[kept] = counts.get(kept, 0) + 1
    assert len(counts) == math.comb(N, K)
    exp = runs / math.comb(N, K)
    chi2 = sum((c - exp) ** 2 / exp for c in counts.values())
    # chi-square with 2 dof, alpha = 1e-3: 13.82
    assert chi2 < 13.82, counts


def _paper_level_law(p, q, N, K):
    """Exact output law of one RELAXED_PAPER level (Algorithm 2 read with N
    distinct drafts) by enumeration: the N drafts as every ordered draw without
    replacement from q (probability prod q(y_i) / (1 - q(y_1) - ... - q(y_{i-1}))),
    each accepted independently with probability min(1, p/q); with at least K
    accepted, each K-subset of them equally likely and the level accepted;
    otherwise the accepted ones plus K - #accepted distinct ordered draws without
    replacement from max(0, p - q) with the accepted ones zeroed (all of its
    support if that holds fewer), the level rejected.  Returns
    {(accepted, frozenset of beams): probability}."""
    import itertools
    C = len(p)
    law = {}

    def add(key, pr):
        law[key] = law.get(key, 0.0) + pr

    for perm in itertools.permutations(range(C), N):
        pd, rest = 1.0, 1.0
        for y in perm:
            pd *= q[y] / rest
            rest -= q[y]
        for mask in itertools.product((0, 1), repeat=N):
            pr = pd
            for y, m in zip(perm, mask):
                a = min(1.0, p[y] / q[y])
                pr *= a if m else 1.0 - a
            if pr == 0.0:
                continue
            A = [y for y, m in zip(perm, mask) if m]
            if len(A) >= K:
                subs = list(itertools.combinations(A, K))
                for s in subs:
                    add((True, frozenset(s)), pr / len(subs))
                continue
            r = [0.0 if c in A else max(0.0, p[c] - q[c]) for c in range(C)]
            pos = [c for c in range(C) if r[c] > 0.0]
            B = K - len(A)
            if len(pos) <= B:
                add((False, frozenset(A) | frozenset(pos)), pr)
                continue
            for draw in itertools.permutations(pos, B):
                pw, rest = 1.0, sum(r)
                for c in draw:
                    pw *= r[c] / rest
                    rest -= r[c]
                add((False, frozenset(A) | frozenset(draw)), pr * pw)
    return law


def _explicit_tables(p, q, cb):
    """Scorers whose level-1 distributions are exactly p (target) and q (draft)
    over cb codes, with a uniform second level."""
    def tab(d):
        t = {(): np.concatenate([np.log(np.asarray(d, dtype=np.float64)), np.full(cb, -50.0)])}
        for c in range(cb):
            t[(c,)] = np.concatenate([np.full(cb, -50.0), np.full(cb, -math.log(cb))])
        return table_scorer(t)
    return tab(p), tab(q)


LAW_CASES = {
    # the draft favours what the target does not: most drafts fail, a few pass
    "reversed": ([0.30, 0.25, 0.20, 0.12, 0.08, 0.05], [0.05, 0.10, 0.15, 0.20, 0.22, 0.28]),
    # partly aligned: passes of one to all four drafts all carry weight
    "shifted": ([0.22, 0.20, 0.18, 0.16, 0.14, 0.10], [0.10, 0.28, 0.12, 0.25, 0.05, 0.20]),
}


@pytest.mark.parametrize("case", list(LAW_CASES))
def test_paper_mode_level_law_matches_enumeration(case):
    """The composite law of a RELAXED_PAPER level, where some but fewer than K
    of the N drafts pass: over many Philox streams the oracle's (accepted,
    level-1 beam set) outcomes follow the law enumerated exactly from pi_p and
    pi_q (chi-square).  Mistakes that leave the special cases N = K = 1 and
    q = p intact -- not zeroing the accepted drafts in the residual, ">" instead
    of ">=", keeping the first K accepted, a residual drawn with replacement --
    move this law."""
    p0, q0 = LAW_CASES[case]
    cb = len(p0)
    trie = Trie(np.array([[a, b] for a in range(cb) for b in range(cb)]))
    lp, lq = _explicit_tables(p0, q0, cb)
    paths, logp, _ = level_dist([((), 0.0)], lp, trie, cb, 1.0)
    _, logq, _ = level_dist([((), 0.0)], lq, trie, cb, 1.0)
    p, q = np.exp(logp), np.exp(logq)
    assert np.allclose(p, p0) and np.allclose(q, q0)
    N, K, runs = 4, 3, 12000
    law = _paper_level_law(p, q, N, K)
    assert abs(sum(law.values()) - 1.0) < 1e-12
    # the composite regime carries weight: some but fewer than K drafts pass
    assert sum(v for (ok, s), v in law.items() if not ok) > 0.2
    counts = {}
    for r in range(runs):
        rs = Streams((r, 31337), 0)
        D = draft_paper(lq, trie, [()], [0.0], 1, N, cb, 1.0, rs, 0)
        res = verify_paper(lp, lq, trie, [((), 0.0)], [0.0], D, K, 2, cb, 1.0, rs, 0)
        key = (res.accepted == 1, frozenset(paths.index(b) for b, _ in res.levels[0]))
        counts[key] = counts.get(key, 0) + 1
    assert set(counts) <= set(law), set(counts) - set(law)
    # bins with an expected count below 5 pooled into one
    exp_, obs_ = [], []
    small_e = small_o = 0.0
    for key, pr in law.items():
        if runs * pr < 5:
            small_e += runs * pr
            small_o += counts.get(key, 0)
        else:
            exp_.append(runs * pr)
            obs_.append(counts.get(key, 0))
    if small_e > 0:
        exp_.append(small_e)
        obs_.append(small_o)
    exp_, obs_ = np.array(exp_), np.array(obs_, dtype=float)
    chi2 = float(((obs_ - exp_) ** 2 / exp_).sum())
    from scipy.stats import chi2 as chi2_dist
    crit = float(chi2_dist.ppf(1 - 1e-3, len(exp_) - 1))
    assert chi2 < crit, (chi2, crit, counts, law)
