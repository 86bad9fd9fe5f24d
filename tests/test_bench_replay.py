"""The bench's forced-acceptance trees (replay-paper-AS profile), checked on the
CPU against the oracle's Algorithm 1: at every step the oracle must accept
exactly the drawn number of levels and move to the drawn level, and the decode
must end on the target beam search lists."""
import numpy as np
import pytest

import bench
from synth import ModelDims, Workload, make_catalog, make_prefixes, make_weights
from oracle.model import Decoder
from oracle.search import beam_search, model_scorer, verify_strict
from oracle.trie import Trie


def _setup(seed, K, N, codebook=6, n_items=300):
    V = 4 * codebook + 7
    w = Workload(name="r", dtype="fp32", target=ModelDims(2, 32, 4, 64, V, 7), draft=ModelDims(1, 16, 2, 32, V, 7),
                 n_items=n_items, batch=1, hist_items=3, prompt_len=2, hist_dist="uniform", K=K, N=N, gamma=4,
                 codebook=codebook, seed=seed)
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    tgt = Decoder(w.target, make_weights(w, "target"), w.dtype)
    lp = model_scorer(tgt, tgt.prefill(pre[0]), w.target.item_base, w.codebook)
    return w, cat, lp


def _levels(want, w):
    """The bench's per-level state records (t, nbeams, paths [B, K, L], scores) for one user."""
    out = []
    for d, beams in enumerate(want, start=1):
        paths = np.zeros((1, w.K, w.L), np.int32)
        sc = np.zeros((1, w.K), np.float32)
        for k, (p, s) in enumerate(beams):
            paths[0, k, :d] = p
            sc[0, k] = s
        out.append((np.array([d]), np.array([len(beams)]), paths, sc))
    return out


@pytest.mark.parametrize("seed,K,N", [(0, 3, 5), (1, 4, 4), (2, 2, 8)])
def test_forced_acceptance_trees_follow_algorithm_1(seed, K, N):
    w, cat, lp = _setup(seed, K, N)
    tr = Trie(cat)
    want = beam_search(lp, tr, K, w.L, w.codebook)
    levels = _levels(want, w)
    kids = bench.catalog_children(cat)
    for draw_seed in range(4):
        steps = bench.replay_as_steps(kids, w, levels, draw_seed)
        Y = [((), 0.0)]
        t = 0
        for trees, acc, after in steps:
            nodes = trees[0]
            D = [[p for p in nodes if len(p) == d] for d in range(t + 1, w.L + 1)]
            while D and not D[-1]:
                D.pop()
            res = verify_strict(lp, tr, Y, D, K, w.L, w.codebook)
            assert res.accepted == acc[0] and res.t_after == after[0], (draw_seed, t, res.accepted, acc[0])
            # the tree holds every current beam path
            assert t == 0 or all(p in nodes for p, _ in Y)
            Y, t = res.beams, res.t_after
        assert t == w.L
        assert [p for p, _ in Y] == [p for p, _ in want[-1]]


def test_forced_acceptance_mean_at_first_step():
    # P(a >= j) = ALPHA^j over four levels: mean 1.64 at t = 0
    a = bench.AS_ALPHA
    assert abs(sum(a ** j for j in range(1, 5)) - 1.64) < 0.01
