"""Pins for the oracle's beam search and strict speculative decoding (CPU)."""
import itertools
import json
import math
import os

import numpy as np
import pytest

from synth import ModelDims, Workload, make_catalog, make_prefixes, make_weights
from oracle.model import Decoder, item_log_softmax
from oracle.search import (beam_search, draft_levels, model_scorer, sd_decode_strict,
                           table_scorer, top, verify_strict)
from oracle.trie import Trie

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _wl(codebook=5, n_items=150, seed=0, dtype="fp32", K=3, N=4):
    V = 4 * codebook + 7
    return Workload(name="s", dtype=dtype, target=ModelDims(2, 32, 4, 64, V, 7),
                    draft=ModelDims(1, 16, 2, 32, V, 7), n_items=n_items, batch=2, hist_items=3,
                    prompt_len=2, hist_dist="uniform", K=K, N=N, gamma=4, codebook=codebook, seed=seed)


def _setup(w, user=0):
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    tgt = Decoder(w.target, make_weights(w, "target"), w.dtype)
    dft = Decoder(w.draft, make_weights(w, "draft"), w.dtype)
    lp = model_scorer(tgt, tgt.prefill(pre[user]), w.target.item_base, w.codebook)
    lq = model_scorer(dft, dft.prefill(pre[user]), w.draft.item_base, w.codebook)
    return cat, pre, tgt, lp, lq


def test_catalog_distinct_and_in_range():
    w = _wl()
    cat = make_catalog(w)
    assert cat.shape == (150, 4)
    assert len({tuple(r) for r in cat.tolist()}) == 150
    assert cat.min() >= 0 and cat.max() < 5


def test_trie_children_brute_force():
    cat = make_catalog(_wl())
    tr = Trie(cat)
    items = [tuple(r) for r in cat.tolist()]
    for l in range(4):
        for pre in {it[:l] for it in items}:
            want = sorted({it[l] for it in items if it[:l] == pre})
            assert tr.children(pre) == want


def test_beam_search_hand_example():
    with open(os.path.join(GOLDEN, "beam_example.json")) as f:
        g = json.load(f)
    cb = g["codebook"]
    tr = Trie(np.array(g["catalog"]))
    table = {}
    for key, pr in g["probs"].items():
        path = tuple(int(c) for c in key.split(",")) if key else ()
        row = np.full(g["L"] * cb, -50.0)
        row[cb * len(path): cb * len(path) + cb] = np.log(pr)
        table[path] = row
    for kname, want in g["expected"].items():
        K = int(kname.split("=")[1])
        levels = beam_search(table_scorer(table), tr, K, g["L"], cb)
        assert [[list(p) for p, _ in lvl] for lvl in levels] == want
    # beam search is not exhaustive: the exact best pair was pruned at level 1 for K=2
    full = beam_search(table_scorer(table), tr, 100, g["L"], cb)[-1]
    assert [list(p) for p, _ in full[:2]] == g["exhaustive_top2"]


class _TableLogits:
    """Stand-in decoder: raw item logits per path, read back through model_scorer."""

    def __init__(self, masses, item_base, codebook):
        self.rows = {k: np.log(np.asarray(v, dtype=np.float64)) for k, v in masses.items()}
        self.base, self.cb = item_base, codebook

    def path_logits(self, cache, toks):
        keys = [",".join(str(t - self.base - self.cb * l) for l, t in enumerate(tk)) for tk in toks]
        return np.stack([self.rows[k] for k in keys])


def test_item_log_softmax_is_normalised_over_all_item_columns():
    rng = np.random.default_rng(11)
    z = rng.standard_normal((5, 1024)) * np.array([[1.0], [10.0], [100.0], [0.01], [300.0]])
    lp = item_log_softmax(z)
    np.testing.assert_allclose(np.exp(lp).sum(axis=-1), 1.0, rtol=0, atol=1e-12)
    # a log-softmax is a shift of the logits by one constant per row
    d = z - lp
    np.testing.assert_allclose(d, np.broadcast_to(d[:, :1], d.shape), rtol=0, atol=1e-9)


def test_normaliser_hand_example():
    # Beams and scores of the hand-worked example in tests/golden/normaliser_example.json,
    # scored through model_scorer exactly as the oracle's searches score a model.
    with open(os.path.join(GOLDEN, "normaliser_example.json")) as f:
        g = json.load(f)
    cb, L = g["codebook"], g["L"]
    tr = Trie(np.array(g["catalog"]))
    for base in (0, 5):
        lp = model_scorer(_TableLogits(g["masses"], base, cb), None, base, cb)
        for kname, want in g["expected"].items():
            K = int(kname.split("=")[1])
            final = beam_search(lp, tr, K, L, cb)[-1]
            assert [list(p) for p, _ in final] == want["beams"]
            np.testing.assert_allclose([s for _, s in final], [math.log(a / b) for a, b in want["prob"]],
                                       rtol=0, atol=1e-12)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_exhaustive_beam_search_equals_enumeration(dtype):
    # Score every catalog item with ONE causal forward over prefix || item
    # (log-probs read at all four positions), rank them, and compare with beam
    # search whose width keeps every candidate.
    w = _wl(codebook=4, n_items=120, dtype=dtype)
    cat, pre, tgt, lp, _ = _setup(w)
    P = pre.shape[1]
    toks = w.target.item_base + w.codebook * np.arange(4)[None, :] + cat
    full = np.concatenate([np.broadcast_to(pre[0], (len(cat), P)), toks], axis=1)
    logits, _ = tgt.forward(full, np.arange(P + 4))
    lps = item_log_softmax(logits[:, P - 1: P + 3])                       # [n, 4, n_item]
    score = lps[np.arange(len(cat))[:, None], np.arange(4)[None, :], w.codebook * np.arange(4)[None, :] + cat].sum(1)
    order = sorted(range(len(cat)), key=lambda i: (-score[i], tuple(cat[i])))
    beams = beam_search(lp, Trie(cat), 10_000, 4, w.codebook)[-1]
    assert [p for p, _ in beams] == [tuple(cat[i]) for i in order]
    np.testing.assert_allclose([s for _, s in beams], score[order], rtol=0, atol=1e-10)


def test_k1_is_greedy():
    w = _wl()
    cat, pre, tgt, lp, _ = _setup(w)
    tr = Trie(cat)
    path = ()
    for l in range(4):
        row = lp([path])[0]
        kids = tr.children(path)
        path = path + (max(kids, key=lambda c: (row[w.codebook * l + c], -c)),)
    assert beam_search(lp, tr, 1, 4, w.codebook)[-1][0][0] == path


@pytest.mark.parametrize("seed,K,N", [(0, 3, 4), (1, 5, 5), (2, 2, 7), (3, 4, 12)])
def test_strict_sd_is_lossless(seed, K, N):
    # Strict top-K verification returns exactly the target beam search lists.
    w = _wl(seed=seed, K=K, N=N)
    cat, pre, tgt, lp, lq = _setup(w, user=seed % 2)
    tr = Trie(cat)
    want = beam_search(lp, tr, K, 4, w.codebook)
    got, steps = sd_decode_strict(lp, lq, tr, K, N, 4, 4, w.codebook)
    assert [p for p, _ in got] == [p for p, _ in want[-1]]
    np.testing.assert_allclose([s for _, s in got], [s for _, s in want[-1]], rtol=0, atol=1e-12)
    # each step's output is the target's beam set of the level it stopped at
    for st in steps:
        assert [p for p, _ in st.result.beams] == [p for p, _ in want[st.result.t_after - 1]]


def test_strict_sd_lossless_with_adversarial_draft():
    w = _wl(seed=4, K=3, N=5)
    cat, pre, tgt, lp, lq = _setup(w)
    tr = Trie(cat)
    rng = np.random.default_rng(0)

    def drafter(Y, J):
        cur, out = list(Y), []
        for _ in range(J):
            ext = [p + (c,) for p in cur for c in tr.children(p)]
            pick = rng.permutation(len(ext))[:w.N]
            cur = [ext[i] for i in sorted(pick)]
            out.append([(p, 0.0) for p in cur])
        return out

    got, _ = sd_decode_strict(lp, lq, tr, 3, 5, 4, 4, w.codebook, drafter=drafter)
    want = beam_search(lp, tr, 3, 4, w.codebook)[-1]
    assert [p for p, _ in got] == [p for p, _ in want]


def test_identical_draft_with_n_equal_k_accepts_everything():
    w = _wl(seed=5, K=4, N=4)
    cat, pre, tgt, lp, _ = _setup(w)
    tr = Trie(cat)
    got, steps = sd_decode_strict(lp, lp, tr, 4, 4, 4, 4, w.codebook)
    assert len(steps) == 1 and steps[0].result.accepted == 4 and steps[0].result.t_after == 4


def test_full_width_draft_accepts_everything():
    # N >= every candidate set: each drafted level holds all extensions.
    w = _wl(seed=6, K=3, N=10_000)
    cat, pre, tgt, lp, lq = _setup(w)
    got, steps = sd_decode_strict(lp, lq, Trie(cat), 3, 10_000, 4, 4, w.codebook)
    assert len(steps) == 1 and steps[0].result.accepted == 4


def test_bonus_level_when_gamma_short():
    # gamma < L: all drafted levels accepted -> one more level from the target.
    w = _wl(seed=7, K=3, N=3)
    cat, pre, tgt, lp, _ = _setup(w)
    tr = Trie(cat)
    got, steps = sd_decode_strict(lp, lp, tr, 3, 3, 2, 4, w.codebook)
    assert steps[0].result.accepted == 2 and steps[0].result.t_after == 3
    want = beam_search(lp, tr, 3, 4, w.codebook)[-1]
    assert [p for p, _ in got] == [p for p, _ in want]


def test_top_margin_and_ties():
    c = [((1,), 0.5), ((0,), 0.5), ((2,), 0.1)]
    sel, m = top(c, 1)
    assert sel[0][0] == (0,) and m == 0.0
    sel, m = top(c, 2)
    assert [p for p, _ in sel] == [(0,), (1,)] and abs(m - 0.4) < 1e-15
    assert top(c, 3)[1] == float("inf")


def _accepted_by_definition(want, t, levels, L):
    """Algorithm 1's accepted length from its definition: level t+i is accepted
    while the target's TopK at that level (its own beam search, pinned above by
    enumeration) lies inside drafted level i; then one target level follows."""
    a = 0
    for i, lvl in enumerate(levels, start=1):
        if {p for p, _ in want[t + i - 1]} <= set(lvl):
            a = i
        else:
            break
    return a, min(L, t + a + 1)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_accepted_lengths_match_the_subset_definition(seed):
    K, L = 3, 4
    w = _wl(seed=seed, K=K, N=6)
    cat, pre, tgt, lp, lq = _setup(w, user=seed % 2)
    tr = Trie(cat)
    want = beam_search(lp, tr, K, L, w.codebook)
    rng = np.random.default_rng(seed)
    breaks = []

    def make_drafter(last):
        return lambda Y, J: drafter(Y, J, last)

    def drafter(Y, J, last):
        # the target's own levels padded with other children, one target path
        # dropped at a random level (J + 1: none dropped) or at the last one
        # (at t = 0 with gamma = L that is the item-completing level L)
        t = len(Y[0])
        brk = J if last else int(rng.integers(1, J + 2))
        breaks.append((t, brk))
        out, prev = [], list(Y)
        for i in range(1, J + 1):
            lvl = [p for p, _ in want[t + i - 1] if p[:-1] in prev]
            dropped = set()
            if i == brk:
                dropped = {lvl[-1]}
                lvl = lvl[:-1]
            extra = [p + (c,) for p in prev for c in tr.children(p)
                     if p + (c,) not in lvl and p + (c,) not in dropped]
            lvl = lvl + extra[:max(0, w.N - len(lvl))]
            out.append([(p, 0.0) for p in lvl])
            prev = lvl
        return out

    for dr in (None, make_drafter(False), make_drafter(True)):
        breaks.clear()
        got, steps = sd_decode_strict(lp, lq, tr, K, w.N, L, L, w.codebook, drafter=dr)
        assert [p for p, _ in got] == [p for p, _ in want[-1]]
        for n, st in enumerate(steps):
            levels = [[p for p, _ in lvl] for lvl in st.drafted]
            a, t_after = _accepted_by_definition(want, st.t, levels, L)
            assert (st.result.accepted, st.result.t_after) == (a, t_after), (dr, st.t, a, t_after)
            if dr is not None:
                t, brk = breaks[n]
                assert a == min(brk - 1, len(levels))
