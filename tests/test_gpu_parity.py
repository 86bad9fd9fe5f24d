"""GPU parity of the verify path against the CPU oracle (through the C ABI).

Workloads: "tiny" (fp32, 2-layer target) and "small" (bf16, 8-layer target,
16 users, tree sizes that span several GEMM tiles and ragged tails).
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from _gpu_common import (LOGIT_TOL, SCORE_TOL, SCORE_TOL_BF16_E2E, SEL_TIE, env, flipped_scorer, logit_table,  # noqa: E402
                         oracle_user, strict_tie, upload_tree)
from oracle.search import draft_levels, path_score, verify_strict  # noqa: E402

USERS = {"tiny": [0], "small": [0, 7, 15]}
_ENG = {}


def engine(name):
    from paper_2410_05165_amd.binding import Engine
    if name not in _ENG:
        e = env(name)
        _ENG[name] = Engine(e["w"], e["tw"], e["dw"], e["cat"])
    return _ENG[name]


def _prefill(name):
    e, eng = env(name), engine(name)
    w = e["w"]
    dev = torch.device("cuda:0")
    prefix = torch.from_numpy(e["pre"]).to(dev)
    root = torch.zeros((w.batch, w.L * w.codebook), dtype=torch.float32, device=dev)
    print(f"[{name}] prefill B={w.batch} P={w.prefix_len}", flush=True)
    eng.atspeed_prefill(prefix, root)
    torch.cuda.synchronize()
    return e, eng, prefix, root


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_prefill_root_logits(name):
    e, eng, prefix, root = _prefill(name)
    r = root.cpu().numpy()
    for u in USERS[name]:
        want = oracle_user(name, u)["tcache"].last_logits
        err = np.abs(r[u] - want).max()
        print(f"[{name}] user {u} root logits max|err| = {err:.3e}")
        assert err <= LOGIT_TOL[e["w"].dtype]


def _oracle_step0_trees(name):
    e = env(name)
    w = e["w"]
    trees = []
    for u in range(w.batch):
        o = oracle_user(name, u)
        D = draft_levels(o["lq"], e["trie"], [()], min(w.gamma, w.L), w.N, w.codebook)
        trees.append([p for lvl in D for p, _ in lvl])
    return trees


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_tree_logits_and_accept(name):
    """Tree forward on the oracle's drafted tree == per-path causal forwards;
    then selection + strict acceptance on those logits == Algorithm 1."""
    e, eng, prefix, root = _prefill(name)
    w = e["w"]
    trees = _oracle_step0_trees(name)
    nodes = upload_tree(eng, trees, w.batch)
    T = eng.max_nodes
    logits = torch.full((w.batch, T, w.L * w.codebook), float("nan"), dtype=torch.float32, device="cuda:0")
    print(f"[{name}] tree logits, nodes/user = {[len(n) for n in nodes][:4]}...", flush=True)
    eng.atspeed_tree_logits(logits)
    torch.cuda.synchronize()
    lg = logits.cpu().numpy()
    for u in USERS[name]:
        o = oracle_user(name, u)
        fwd = [i for i, p in enumerate(nodes[u]) if len(p) < w.L]
        toks = [tuple(w.target.item_base + w.codebook * l + c for l, c in enumerate(nodes[u][i])) for i in fwd]
        want = o["tgt"].path_logits(o["tcache"], toks)
        err = np.abs(lg[u, fwd] - want).max()
        print(f"[{name}] user {u}: {len(fwd)} forwarded nodes, logits max|err| = {err:.3e}")
        assert err <= LOGIT_TOL[w.dtype]
    # acceptance on the same fp32 logits
    acc = torch.zeros(w.batch, dtype=torch.int32, device="cuda:0")
    ta = torch.zeros(w.batch, dtype=torch.int32, device="cuda:0")
    eng.atspeed_accept(logits.nan_to_num(0.0), root, acc, ta)
    t, nb, paths, sc = eng.atspeed_get_state(w.batch)
    r = root.cpu().numpy()
    acc, ta = acc.cpu().numpy(), ta.cpu().numpy()
    for u in range(w.batch):
        lp = logit_table(nodes[u], lg[u], r[u])
        D = [[p for p in trees[u] if len(p) == d] for d in range(1, min(w.gamma, w.L) + 1)]
        log = []
        res = verify_strict(lp, e["trie"], [((), 0.0)], D, w.K, w.L, w.codebook, log)
        got = [tuple(int(c) for c in paths[u, k, :t[u]]) for k in range(nb[u])]

        def same(r):
            return [p for p, _ in r.beams] == got and r.accepted == acc[u] and r.t_after == ta[u]
        if not same(res):
            d = strict_tie(log, lambda d: verify_strict(flipped_scorer(lp, d, w.codebook), e["trie"], [((), 0.0)],
                                                        D, w.K, w.L, w.codebook), same)
            assert d is not None, (u, got, [p for p, _ in res.beams], acc[u], res.accepted)
            print(f"[{name}] user {u}: the level-{d.level} TopK decision (margin {d.margin:.2e}) taken the "
                  f"other way gives the GPU's selection")
            continue
        np.testing.assert_allclose(sc[u, :nb[u]], [s for _, s in res.beams], rtol=0, atol=1e-4)


def _gpu_paths(tn, tt, tp, td, u, w):
    paths = []
    for i in range(tn[u]):
        code = tt[u, i] - w.target.item_base - w.codebook * (td[u, i] - 1)
        paths.append((paths[tp[u, i]] if tp[u, i] >= 0 else ()) + (int(code),))
    return paths


def _consistent_top(chosen, cands, score, n, eps):
    """``chosen`` is the exact top-n of ``cands`` under ``score`` (ties: smaller
    path), or differs from it only between candidates whose scores are within eps."""
    want = sorted(cands, key=lambda c: (-score[c], c))[:n]
    if list(chosen) == want:
        return 0.0
    assert len(set(chosen)) == len(chosen) == min(n, len(cands))
    assert set(chosen) <= set(cands)
    rest = [score[c] for c in cands if c not in set(chosen)]
    gap = (max(rest) - min(score[c] for c in chosen)) if rest else 0.0
    assert gap <= eps, (gap, eps)
    return gap


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_draft_tree(name):
    """GPU drafting (Eq. 1) at t = 0: every drafted level is the TopN of the
    extensions of the previous level under the oracle's draft scores -- exactly,
    or within the score error that the forward tolerance allows (bf16)."""
    e, eng, prefix, root = _prefill(name)
    w = e["w"]
    eng.atspeed_draft()
    torch.cuda.synchronize()
    tn, tt, tp, td, tq = (x.cpu().numpy() for x in eng.tree_tensors(w.batch))
    for u in USERS[name]:
        o = oracle_user(name, u)
        paths = _gpu_paths(tn, tt, tp, td, u, w)
        J = min(w.gamma, w.L)
        prev = [()]
        score = {}
        err = 0.0
        for i, p in enumerate(paths):
            score[p] = path_score(o["lq"], p, w.codebook)
            err = max(err, abs(float(tq[u, i]) - score[p]))
        print(f"[{name}] user {u}: draft cumulative log-prob max|err| = {err:.3e}")
        assert err <= (SCORE_TOL if w.dtype == "fp32" else SCORE_TOL_BF16_E2E)
        for j in range(1, J + 1):
            cands = [p + (c,) for p in prev for c in e["trie"].children(p)]
            for c in cands:
                if c not in score:
                    score[c] = path_score(o["lq"], c, w.codebook)
            got = [p for p, d in zip(paths, td[u]) if d == j]
            eps = 2e-6 if w.dtype == "fp32" else 2 * err + SEL_TIE
            gap = _consistent_top(got, cands, score, w.N, eps)
            if gap:
                print(f"[{name}] user {u} level {j}: differs from exact TopN within {gap:.2e} (eps {eps:.2e})")
            prev = got


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_decode_topk_lossless(name):
    """Speculative decode on the GPU (draft + verify) returns bitwise the lists of
    the GPU's own target-only beam search (verify on trees without drafted
    levels), and every level of that search is the oracle's TopK of the same
    extensions (exactly, or within the bf16 score error)."""
    e = env(name)
    eng = engine(name)
    w = e["w"]
    from paper_2410_05165_amd.binding import Stats
    import ctypes as C
    dev = torch.device("cuda:0")
    prefix = torch.from_numpy(e["pre"]).to(dev)
    items = torch.zeros((w.batch, w.K, w.L), dtype=torch.int32, device=dev)
    scores = torch.zeros((w.batch, w.K), dtype=torch.float32, device=dev)
    n = torch.zeros(w.batch, dtype=torch.int32, device=dev)
    acc = np.zeros((w.L, w.batch), np.int32)
    ta = np.zeros((w.L, w.batch), np.int32)
    st = Stats()
    st.accepted = acc.ctypes.data_as(C.POINTER(C.c_int32))
    st.t_after = ta.ctypes.data_as(C.POINTER(C.c_int32))
    print(f"[{name}] decode_topk B={w.batch}", flush=True)
    eng.atspeed_decode_topk(prefix, items, scores, n, st)
    torch.cuda.synchronize()
    it, sc, nn = items.cpu().numpy(), scores.cpu().numpy(), n.cpu().numpy()
    print(f"[{name}] steps={st.n_steps} accepted={acc[:st.n_steps, :4].tolist()} prefill={st.ms_prefill:.2f}ms "
          f"draft={st.ms_draft:.2f}ms verify={st.ms_verify:.2f}ms")
    # GPU target-only beam search: verify on Y_t-only trees, one level per call
    eng.atspeed_prefill(prefix)
    levels = []
    for lvl in range(w.L):
        t, nb, paths, bsc = eng.atspeed_get_state(w.batch)
        trees = [[tuple(int(c) for c in paths[u, k, :t[u]]) for k in range(nb[u])] if t[u] > 0 else []
                 for u in range(w.batch)]
        upload_tree(eng, trees, w.batch)
        eng.atspeed_verify()
        levels.append(eng.atspeed_get_state(w.batch))
    t, nb, paths, bsc = levels[-1]
    assert (t == w.L).all()
    np.testing.assert_array_equal(nb, nn)
    for u in range(w.batch):
        np.testing.assert_array_equal(paths[u, :nb[u]], it[u, :nn[u]])
        np.testing.assert_array_equal(bsc[u, :nb[u]], sc[u, :nn[u]])
    # each GPU level against the oracle's scores of the same candidates
    for u in USERS[name]:
        o = oracle_user(name, u)
        prev = [()]
        for lvl, (t, nb, paths, bsc) in enumerate(levels):
            got = [tuple(int(c) for c in paths[u, k, :lvl + 1]) for k in range(nb[u])]
            cands = [p + (c,) for p in prev for c in e["trie"].children(p)]
            score = {c: path_score(o["lp"], c, w.codebook) for c in cands}
            err = max(abs(float(bsc[u, k]) - score[g]) for k, g in enumerate(got))
            assert err <= (SCORE_TOL if w.dtype == "fp32" else SCORE_TOL_BF16_E2E), err
            eps = 2e-6 if w.dtype == "fp32" else 2 * err + SEL_TIE
            gap = _consistent_top(got, cands, score, w.K, eps)
            print(f"[{name}] user {u} level {lvl + 1}: score max|err| {err:.2e}" +
                  (f", differs within {gap:.2e}" if gap else ", exact TopK"))
            prev = got
