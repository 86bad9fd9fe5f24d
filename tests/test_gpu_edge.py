"""Edge cases of the verify path on the GPU, through the C ABI.

* malformed caller trees are rejected with ATSPEED_E_INVALID (the device-side
  validation keeps every kernel inside its buffers: a user whose tree fails it
  forwards nothing) and leave the context usable;
* ragged and empty trees: users with no nodes, only depth-1 nodes, one chain,
  and a full drafted tree, in one batch (fp32, so logits and selections are
  exact against the oracle);
* finished users (t = L) are no-ops;
* degenerate and maximal widths: K = N = 1 (greedy) and K = N = 128 (the
  largest the selection kernels hold), decoded end to end against the oracle's
  target-only beam search.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from _gpu_common import LOGIT_TOL, env, flipped_scorer, logit_table, strict_tie, tree_arrays  # noqa: E402
from oracle.model import Decoder  # noqa: E402
from oracle.search import beam_search, draft_levels, model_scorer, verify_strict  # noqa: E402

DEV = "cuda:0"


def _engine(w, e):
    from paper_2410_05165_amd.binding import Engine
    return Engine(w, e["tw"], e["dw"], e["cat"])


def _prefill(eng, e):
    w = e["w"]
    prefix = torch.from_numpy(e["pre"]).to(DEV)
    root = torch.zeros((w.batch, w.L * w.codebook), dtype=torch.float32, device=DEV)
    eng.atspeed_prefill(prefix, root)
    torch.cuda.synchronize()
    return prefix, root


def _put(eng, B, n, tok, par, dep):
    tn, tt, tp, td, tq = eng.tree_tensors(B)
    tn.copy_(torch.from_numpy(np.ascontiguousarray(n, np.int32)))
    tt.copy_(torch.from_numpy(np.ascontiguousarray(tok, np.int32)))
    tp.copy_(torch.from_numpy(np.ascontiguousarray(par, np.int32)))
    td.copy_(torch.from_numpy(np.ascontiguousarray(dep, np.int32)))
    tq.zero_()
    torch.cuda.synchronize()


def _oracle_users(e, users):
    w = e["w"]
    out = {}
    for u in users:
        tgt, dft = Decoder(w.target, e["tw"], w.dtype), Decoder(w.draft, e["dw"], w.dtype)
        tc, dc = tgt.prefill(e["pre"][u]), dft.prefill(e["pre"][u])
        out[u] = dict(tgt=tgt, tc=tc, lp=model_scorer(tgt, tc, w.target.item_base, w.codebook),
                      lq=model_scorer(dft, dc, w.draft.item_base, w.codebook))
    return out


def _drafted(e, o, J):
    w = e["w"]
    return draft_levels(o["lq"], e["trie"], [()], J, w.N, w.codebook)


def test_malformed_trees_are_rejected():
    from paper_2410_05165_amd.binding import AtspeedError
    e = env("tiny")
    w = e["w"]
    eng = _engine(w, e)
    try:
        _prefill(eng, e)
        o = _oracle_users(e, [0])[0]
        D = _drafted(e, o, min(w.gamma, w.L))
        good = tree_arrays([[p for lvl in D for p, _ in lvl]], w, eng.max_nodes)[:4]
        n, tok, par, dep = (np.array(a) for a in good)
        i1 = int(np.flatnonzero(dep[0] == 1)[0])
        i2 = int(np.flatnonzero(dep[0] == 2)[0])
        i3 = int(np.flatnonzero(dep[0] == 3)[0])
        bad_code = next(c for c in range(w.codebook) if c not in set(e["trie"].children(
            (int(tok[0, i1] - w.target.item_base),))))

        def case(f):
            a = [x.copy() for x in (n, tok, par, dep)]
            f(*a)
            return a

        cases = {
            "n_nodes above the tree capacity": case(lambda n_, t_, p_, d_: n_.__setitem__(0, eng.max_nodes + 1)),
            "negative n_nodes": case(lambda n_, t_, p_, d_: n_.__setitem__(0, -1)),
            "depth 0": case(lambda n_, t_, p_, d_: d_.__setitem__((0, i1), 0)),
            "depth above L": case(lambda n_, t_, p_, d_: d_.__setitem__((0, i3), w.L + 1)),
            "parent after the node": case(lambda n_, t_, p_, d_: p_.__setitem__((0, i2), i2 + 1)),
            "parent out of range": case(lambda n_, t_, p_, d_: p_.__setitem__((0, i2), 10 ** 6)),
            "depth-1 node with a parent": case(lambda n_, t_, p_, d_: p_.__setitem__((0, i1), 0)),
            "token outside the item range": case(lambda n_, t_, p_, d_: t_.__setitem__((0, i1), 10 ** 6)),
            "path not in the catalog": case(lambda n_, t_, p_, d_: (
                p_.__setitem__((0, i2), i1),
                t_.__setitem__((0, i2), w.target.item_base + w.codebook + bad_code))),
            "node is its own parent": case(lambda n_, t_, p_, d_: (
                d_.__setitem__((0, i1), 2), p_.__setitem__((0, i1), i1))),
            "levels out of order": case(lambda n_, t_, p_, d_: d_.__setitem__((0, i3), 1)),
        }
        for name, arrs in cases.items():
            print(f"[edge] malformed tree: {name}", flush=True)
            _put(eng, w.batch, *arrs)
            with pytest.raises(AtspeedError) as ex:
                eng.atspeed_verify()
            assert ex.value.status == 1 and "malformed tree" in str(ex.value), (name, str(ex.value))
        # the context still verifies a valid tree, with the oracle's result
        _put(eng, w.batch, n, tok, par, dep)
        acc = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
        ta = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
        eng.atspeed_verify(acc, ta)
        log = []
        res = verify_strict(o["lp"], e["trie"], [((), 0.0)], [[p for p, _ in lvl] for lvl in D], w.K, w.L,
                            w.codebook, log)
        t, nb, paths, sc = eng.atspeed_get_state(w.batch)
        got = [tuple(int(c) for c in paths[0, k, :t[0]]) for k in range(nb[0])]

        def same(r):
            return [p for p, _ in r.beams] == got and r.accepted == int(acc[0]) and r.t_after == int(ta[0])
        if not same(res):
            Dp = [[p for p, _ in lvl] for lvl in D]
            assert strict_tie(log, lambda d: verify_strict(flipped_scorer(o["lp"], d, w.codebook), e["trie"],
                                                           [((), 0.0)], Dp, w.K, w.L, w.codebook), same) is not None
        # a beam of Y_t missing from the caller's tree (t = 1)
        eng.atspeed_prefill(torch.from_numpy(e["pre"]).to(DEV))
        top1 = sorted(((p, s) for p, s in res.levels[0]))[:w.K]
        paths1 = np.zeros((w.batch, w.K, w.L), np.int32)
        for k, (p, _) in enumerate(top1):
            paths1[0, k, 0] = p[0]
        eng.atspeed_set_state(np.array([1]), np.array([len(top1)]), paths1,
                              np.array([[s for _, s in top1] + [0.0] * (w.K - len(top1))], np.float32))
        arrs = tree_arrays([[p for p, _ in top1[1:]]], w, eng.max_nodes)[:4]
        print("[edge] malformed tree: beam of Y_t missing", flush=True)
        _put(eng, w.batch, *arrs)
        with pytest.raises(AtspeedError) as ex:
            eng.atspeed_verify()
        assert ex.value.status == 1
    finally:
        eng.close()


def test_ragged_and_empty_trees():
    e = env("tiny", batch=4)
    w = e["w"]
    eng = _engine(w, e)
    try:
        _, root = _prefill(eng, e)
        os_ = _oracle_users(e, range(w.batch))
        J = min(w.gamma, w.L)
        full = [_drafted(e, os_[u], J) for u in range(w.batch)]
        trees = [
            [],                                                   # empty
            [p for p, _ in full[1][0]],                           # depth 1 only
            [p for p, _ in full[2][J - 1][:1]],                   # one chain of depth J
            [p for lvl in full[3] for p, _ in lvl],               # the whole drafted tree
        ]
        # the chain of user 2 needs its ancestors as nodes
        chain = trees[2][0]
        trees[2] = [chain[:d] for d in range(1, len(chain) + 1)]
        n, tok, par, dep, nodes = tree_arrays(trees, w, eng.max_nodes)
        _put(eng, w.batch, n, tok, par, dep)
        T = eng.max_nodes
        logits = torch.full((w.batch, T, w.L * w.codebook), float("nan"), dtype=torch.float32, device=DEV)
        print(f"[edge] ragged trees, nodes per user {n.tolist()}", flush=True)
        eng.atspeed_tree_logits(logits)
        torch.cuda.synchronize()
        lg = logits.cpu().numpy()
        for u in range(w.batch):
            fwd = [i for i, p in enumerate(nodes[u]) if len(p) < w.L]
            if not fwd:
                continue
            toks = [tuple(w.target.item_base + w.codebook * l + c for l, c in enumerate(nodes[u][i])) for i in fwd]
            want = os_[u]["tgt"].path_logits(os_[u]["tc"], toks)
            err = np.abs(lg[u, fwd] - want).max()
            print(f"[edge] user {u}: {len(fwd)} forwarded nodes, logits max|err| {err:.2e}")
            assert err <= LOGIT_TOL[w.dtype]
        acc = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
        ta = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
        eng.atspeed_accept(logits.nan_to_num(0.0), root, acc, ta)
        t, nb, paths, sc = eng.atspeed_get_state(w.batch)
        r = root.cpu().numpy()
        for u in range(w.batch):
            lp = logit_table(nodes[u], lg[u], r[u])
            D = [[p for p in trees[u] if len(p) == d] for d in range(1, J + 1)]
            log = []
            res = verify_strict(lp, e["trie"], [((), 0.0)], D, w.K, w.L, w.codebook, log)
            got = [tuple(int(c) for c in paths[u, k, :t[u]]) for k in range(nb[u])]
            print(f"[edge] user {u}: accepted {int(acc[u])} (oracle {res.accepted}), t -> {int(ta[u])}")

            def same(r):
                return [p for p, _ in r.beams] == got and r.accepted == int(acc[u]) and r.t_after == int(ta[u])
            if not same(res):
                assert strict_tie(log, lambda d: verify_strict(flipped_scorer(lp, d, w.codebook), e["trie"],
                                                               [((), 0.0)], D, w.K, w.L, w.codebook),
                                  same) is not None
                continue
            np.testing.assert_allclose(sc[u, :nb[u]], [s for _, s in res.beams], rtol=0, atol=1e-4)
        assert int(acc[0]) == 0 and int(ta[0]) == 1          # empty tree: level 1 rejected, target level taken
    finally:
        eng.close()


def test_finished_users_are_noops():
    e = env("tiny", batch=2)
    w = e["w"]
    eng = _engine(w, e)
    try:
        _prefill(eng, e)
        o = _oracle_users(e, [0])[0]
        done = beam_search(o["lp"], e["trie"], w.K, w.L, w.codebook)[-1]
        paths = np.zeros((w.batch, w.K, w.L), np.int32)
        scores = np.zeros((w.batch, w.K), np.float32)
        for k, (p, s) in enumerate(done):
            paths[0, k] = p
            scores[0, k] = s
        eng.atspeed_set_state(np.array([w.L, 0]), np.array([len(done), 1]), paths, scores)
        before = eng.atspeed_get_state(w.batch)
        # user 0's tree arrays hold garbage: a finished user's tree is not read
        n = np.array([eng.max_nodes + 7, 0])
        z = np.zeros((w.batch, eng.max_nodes), np.int32)
        _put(eng, w.batch, n, z, z - 1, z)
        acc = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
        ta = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
        print("[edge] verify with user 0 finished", flush=True)
        eng.atspeed_verify(acc, ta)
        after = eng.atspeed_get_state(w.batch)
        assert int(acc[0]) == -1 and int(ta[0]) == w.L
        assert after[0][0] == w.L and after[1][0] == before[1][0]
        np.testing.assert_array_equal(after[2][0], before[2][0])
        np.testing.assert_array_equal(after[3][0], before[3][0])
        assert int(ta[1]) == 1 and int(acc[1]) == 0
    finally:
        eng.close()


@pytest.mark.parametrize("K", [1, 128])
def test_extreme_widths_decode(K):
    """K = N = 1 is greedy decoding; K = N = 128 fills the selection kernels.
    fp32, so the decoded lists equal the oracle's target-only beam search (up to
    one near-tie decision, margin below 1e-3, taken the other way)."""
    e = env("tiny", K=K, N=K)
    w = e["w"]
    eng = _engine(w, e)
    try:
        prefix = torch.from_numpy(e["pre"]).to(DEV)
        items = torch.zeros((w.batch, w.K, w.L), dtype=torch.int32, device=DEV)
        scores = torch.zeros((w.batch, w.K), dtype=torch.float32, device=DEV)
        nn = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
        print(f"[edge] decode_topk K = N = {K}", flush=True)
        eng.atspeed_decode_topk(prefix, items, scores, nn, None)
        torch.cuda.synchronize()
        it, sc, nn = items.cpu().numpy(), scores.cpu().numpy(), nn.cpu().numpy()
        o = _oracle_users(e, [0])[0]
        log = []
        want = beam_search(o["lp"], e["trie"], w.K, w.L, w.codebook, log)[-1]
        got = [tuple(int(c) for c in it[0, k]) for k in range(nn[0])]
        if got != [p for p, _ in want]:
            d = strict_tie(log, lambda d: beam_search(flipped_scorer(o["lp"], d, w.codebook), e["trie"], w.K, w.L,
                                                      w.codebook), lambda lv: [p for p, _ in lv[-1]] == got)
            assert d is not None
            print(f"[edge] K={K}: the level-{d.level} TopK decision (margin {d.margin:.2e}) taken the other way "
                  f"gives the GPU's list")
        else:
            np.testing.assert_allclose(sc[0, :nn[0]], [s for _, s in want], rtol=0, atol=1e-4)
        assert nn[0] == min(K, len(want))
    finally:
        eng.close()
