"""Pins for the oracle's draft alignment objectives (Sec. 3.1 Align-S, Sec. 3.2 Align-R), CPU."""
import json
import math
import os

import numpy as np
import pytest

from oracle.align import (adamw_step, label_distributions, mixture_beam_search, rec_loss, align_r, align_s, aligned_loss, constrained_topk, context_weights, head_gradient,
                          log_pK_of)
from oracle.search import table_scorer
from oracle.trie import Trie

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_worked_context():
    with open(os.path.join(GOLDEN, "align_example.json")) as f:
        g = json.load(f)
    lq, lp = np.log(g["q"]), np.log(g["p"])
    assert constrained_topk(lq, g["valid_cols"], g["K"]) == g["V_c"]
    ls, _, vc = align_s(lq, lp, g["valid_cols"], g["K"], math.log(g["p_K"]))
    assert vc == g["V_c"]
    assert abs(ls - 0.4 * math.log(1.25)) < 1e-12
    lr, _, _ = align_r(lq, lp, g["valid_cols"], g["K"])
    assert abs(lr - g["loss_R"][0] / g["loss_R"][1]) < 1e-12


@pytest.mark.parametrize("mode", ["S", "R"])
def test_gradients_match_finite_differences(mode):
    rng = np.random.default_rng(3)
    n, cols, K = 24, [1, 3, 4, 8, 9, 12, 17, 20], 4
    for trial in range(5):
        z = rng.standard_normal(n) * 2
        lp = np.log(np.exp(rng.standard_normal(n)) / np.exp(rng.standard_normal(n)).sum())
        lpk = float(rng.normal(-3, 1))

        def f(zz):
            lq = zz - (np.max(zz) + np.log(np.exp(zz - np.max(zz)).sum()))
            return (align_s(lq, lp, cols, K, lpk) if mode == "S" else align_r(lq, lp, cols, K))[:2]
        l0, g = f(z)
        vc0 = constrained_topk(z, cols, K)
        for j in range(n):
            e = np.zeros(n)
            e[j] = 1e-6
            # V_c is piecewise constant: only compare where the step keeps it
            if constrained_topk(z + e, cols, K) != vc0 or constrained_topk(z - e, cols, K) != vc0:
                continue
            fd = (f(z + e)[0] - f(z - e)[0]) / 2e-6
            assert abs(fd - g[j]) < 1e-6 * max(1.0, abs(fd)), (mode, trial, j, fd, g[j])


def test_density_regulariser_sign():
    q = np.array([0.5, 0.3, 0.1, 0.1])
    lp = np.log(np.array([0.4, 0.3, 0.2, 0.1]))
    cols = [0, 1, 2, 3]
    # V_c = {0, 1}; both more probable under the target than p_K = 0.15: negative
    assert align_s(np.log(q), lp, cols, 2, math.log(0.15))[0] < 0
    # both less probable than p_K = 0.5: positive
    assert align_s(np.log(q), lp, cols, 2, math.log(0.5))[0] > 0


def test_tvd_range_and_sum_of_minima():
    rng = np.random.default_rng(5)
    cols = list(range(10))
    for _ in range(20):
        lq = np.log(rng.dirichlet(np.ones(10)))
        lp = np.log(rng.dirichlet(np.ones(10)))
        t, _, vc = align_r(lq, lp, cols, 10)
        qn, pn = np.exp(lq), np.exp(lp)
        assert 0.0 <= t <= 1.0
        assert abs((1 - t) - np.minimum(qn, pn).sum()) < 1e-12     # Eq. 6: b = 1 - TVD
        assert align_r(lq, lq, cols, 4)[0] == 0.0


def test_context_weights_hand_count():
    Y = [[(0, 0), (0, 1), (1, 0)]]
    w = context_weights(Y, 2)[0]
    assert w == {(): 1.5, (0,): 1.0, (1,): 0.5}
    w2 = context_weights([[(0, 0)], [(1, 1), (1, 0)]], 2)
    assert w2[0] == {(): 0.25, (0,): 0.25} and w2[1] == {(): 0.5, (1,): 0.5}


def test_log_pK_is_the_kth_sequence_along_its_own_prefix():
    cb = 3
    rows = {(): np.log([0.5, 0.3, 0.2, 0.1, 0.1, 0.8]), (1,): np.log([0.2, 0.2, 0.6, 0.7, 0.2, 0.1])}
    got = log_pK_of([(0, 2), (1, 0)], lambda p: rows[p], cb)
    assert np.allclose(got, [math.log(0.3), math.log(0.7)])


def test_aggregate_and_head_gradient():
    # two users, one level: the aggregate is the weighted sum of the contexts and
    # the head gradient is the weighted sum of outer products
    cb, L, K = 3, 1, 1
    trie = Trie(np.array([[0], [1], [2]]))
    rng = np.random.default_rng(1)
    lq = {u: np.log(rng.dirichlet(np.ones(3))) for u in range(2)}
    lp = {u: np.log(rng.dirichlet(np.ones(3))) for u in range(2)}
    Y = [[(int(np.argmax(lp[u])),)] for u in range(2)]
    loss, grads = aligned_loss("R", lambda u, p: lq[u], lambda u, p: lp[u], trie, Y, K, L, cb)
    assert abs(loss - sum(0.5 * align_r(lq[u], lp[u], [0, 1, 2], K)[0] for u in range(2))) < 1e-12
    h = {k: rng.standard_normal(4) for k in grads}
    G = head_gradient(grads, h)
    want = sum(grads[k][0] * np.outer(grads[k][1], h[k]) for k in grads)
    assert np.allclose(G, want)


def test_adamw_matches_torch_adamw():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    w0 = rng.standard_normal((5, 4))
    grads = [rng.standard_normal((5, 4)) for _ in range(4)]
    hp = dict(lr=1e-2, beta1=0.8, beta2=0.95, eps=1e-6, weight_decay=0.1)
    p = torch.tensor(w0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([p], lr=hp["lr"], betas=(hp["beta1"], hp["beta2"]), eps=hp["eps"],
                            weight_decay=hp["weight_decay"])
    w, m, v = w0.copy(), np.zeros_like(w0), np.zeros_like(w0)
    for step, g in enumerate(grads, 1):
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        w, m, v = adamw_step(w, m, v, g, step, **hp)
        np.testing.assert_allclose(w, p.detach().numpy(), rtol=0, atol=1e-14)


def test_adamw_first_step_closed_form():
    # step 1 without decay: the bias-corrected moments are g and g^2, so the step
    # is lr * g / (|g| + eps), i.e. lr times the sign for |g| >> eps
    g = np.array([3.0, -0.5, 1e-3, -2e-3])
    w, m, v = adamw_step(np.zeros(4), np.zeros(4), np.zeros(4), g, 1, 0.1, 0.9, 0.999, 1e-12, 0.0)
    np.testing.assert_allclose(w, -0.1 * np.sign(g), rtol=1e-8)
    np.testing.assert_allclose(m, 0.1 * g)
    np.testing.assert_allclose(v, 0.001 * g * g)
    # decay alone shrinks by lr * wd
    w2, _, _ = adamw_step(np.full(4, 2.0), np.zeros(4), np.zeros(4), np.zeros(4), 1, 0.1, 0.9, 0.999, 1e-8, 0.5)
    np.testing.assert_allclose(w2, 2.0 * (1 - 0.05))


def test_rec_loss_matches_torch_cross_entropy():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(4)
    z = rng.standard_normal(12)
    pi = {2: 0.25, 7: 0.5, 11: 0.25}
    lq = z - np.log(np.exp(z).sum())
    loss, grad = rec_loss(lq, pi)
    zt = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    target = torch.zeros(12, dtype=torch.float64)
    for c, v in pi.items():
        target[c] = v
    ce = torch.nn.functional.cross_entropy(zt[None], target[None])
    ce.backward()
    assert abs(loss - ce.item()) < 1e-13
    np.testing.assert_allclose(grad, zt.grad.numpy(), atol=1e-14)


def test_label_distributions_and_weights_of_mixed_lengths():
    # multi-step data: a whole item and a one-code beam
    Y = [(0, 0), (0, 1), (1,)]
    pis = label_distributions(Y, 2)
    assert pis == {(): {0: 0.5, 1: 0.5}, (0,): {2: 0.5, 3: 0.5}}
    w = context_weights([[(0, 0), (1,)]], 2)[0]
    assert w == {(): 1.5, (0,): 0.5}


def test_aggregate_alpha_zero_is_sequence_nll():
    cb, L, K = 3, 2, 2
    cat = np.array([[a, b] for a in range(3) for b in range(3)])
    trie = Trie(cat)
    rng = np.random.default_rng(6)
    lq = {(u, p): np.log(rng.dirichlet(np.ones(6))) for u in range(2) for p in [(), (0,), (1,), (2,)]}
    lp = {k: np.log(rng.dirichlet(np.ones(6))) for k in lq}
    Y = [[(0, 1), (2,), (1, 2)], [(2, 0), (2, 2)]]
    loss, _ = aligned_loss("S", lambda u, p: lq[(u, p)], lambda u, p: lp[(u, p)], trie, Y, K, L, cb, alpha=0.0)
    want = 0.0
    for u, ys in enumerate(Y):
        for y in ys:
            want += sum(-lq[(u, tuple(y[:t]))][cb * t + y[t]] for t in range(len(y))) / len(y)
    assert abs(loss - want / len(Y)) < 1e-12


@pytest.mark.parametrize("mode", ["S", "R"])
def test_aggregate_gradient_finite_differences(mode):
    # the combined per-context gradient times its weight is d(total)/dz of that context
    cb, L, K, alpha = 3, 2, 2, 0.4
    cat = np.array([[a, b] for a in range(3) for b in range(3) if (a + b) % 4 != 3])
    trie = Trie(cat)
    rng = np.random.default_rng(8)
    keys = [(u, p) for u in range(2) for p in [(), (0,), (1,), (2,)]]
    z = {k: rng.standard_normal(6) for k in keys}
    lp = {k: np.log(rng.dirichlet(np.ones(6))) for k in keys}
    Y = [[(0, 1), (2,), (1, 0)], [(2, 0), (0, 0)]]

    def total(zz):
        lq = lambda u, p: zz[(u, p)] - np.log(np.exp(zz[(u, p)]).sum())
        return aligned_loss(mode, lq, lambda u, p: lp[(u, p)], trie, Y, K, L, cb, alpha)
    _, grads = total(z)
    h = 1e-6
    for k, (w, g) in grads.items():
        for j in range(6):
            zp = {kk: v.copy() for kk, v in z.items()}
            zm = {kk: v.copy() for kk, v in z.items()}
            zp[k][j] += h
            zm[k][j] -= h
            fd = (total(zp)[0] - total(zm)[0]) / (2 * h)
            assert abs(fd - w * g[j]) < 1e-7, (k, j, fd, w * g[j])


def _mixture_tables():
    ex = json.load(open(os.path.join(GOLDEN, "mixture_example.json")))
    key = lambda path: "".join(str(c) for c in path)
    lp = lambda path: np.log(np.array(ex["rows"][key(path)]["p"]))
    lq = lambda path: np.log(np.array(ex["rows"][key(path)]["q"]))
    return ex, lp, lq


def test_mixture_search_hand_example():
    ex, lp, lq = _mixture_tables()
    trie = Trie(np.array([[0, 0], [0, 1], [1, 0], [1, 1]]))
    for case in ex["cases"]:
        levels = mixture_beam_search(lp, lq, trie, case["K"], ex["L"], ex["codebook"], case["lambda"])
        for got, want in zip(levels, (case["level1"], case["level2"])):
            assert [p for p, _ in got] == [tuple(p) for p, _ in want], case
            np.testing.assert_allclose([s for _, s in got], [math.log(v) for _, v in want], rtol=0, atol=1e-12)


def test_mixture_search_reduces_to_each_model_and_to_enumeration():
    from oracle.search import beam_search
    rng = np.random.default_rng(11)
    cb, L = 3, 3
    cat = np.array([[a, b, c] for a in range(3) for b in range(3) for c in range(3) if (a * 7 + b * 3 + c) % 5 != 2])
    trie = Trie(cat)
    paths = {()} | {tuple(r[:t]) for r in cat.tolist() for t in range(1, L)}
    P = {p: np.log(rng.dirichlet(np.ones(cb * L))) for p in paths}
    Q = {p: np.log(rng.dirichlet(np.ones(cb * L))) for p in paths}
    lp, lq = (lambda p: P[p]), (lambda p: Q[p])
    for lam, table in ((1.0, P), (0.0, Q)):
        want = beam_search(table_scorer(table), trie, 4, L, cb)
        got = mixture_beam_search(lp, lq, trie, 4, L, cb, lam)
        for g, wv in zip(got, want):
            assert [p for p, _ in g] == [p for p, _ in wv]
            np.testing.assert_allclose([s for _, s in g], [s for _, s in wv], rtol=0, atol=1e-12)
    # width at least the catalog: the last level ranks every item by its mixed
    # sequence log-probability, summed here in probability space per token
    lam = 0.3
    got = mixture_beam_search(lp, lq, trie, len(cat), L, cb, lam)[-1]
    score = {}
    for item in map(tuple, cat.tolist()):
        score[item] = sum(math.log((1 - lam) * math.exp(Q[item[:t]][cb * t + item[t]])
                                   + lam * math.exp(P[item[:t]][cb * t + item[t]])) for t in range(L))
    want = sorted(score.items(), key=lambda kv: (-kv[1], kv[0]))
    assert [p for p, _ in got] == [p for p, _ in want]
    np.testing.assert_allclose([s for _, s in got], [s for _, s in want], rtol=0, atol=1e-12)
