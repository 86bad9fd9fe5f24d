"""Relaxed sampling verification (the paper's reading of Algorithm 2, Sec. 3.2)
in bf16 at the small shape and at the full 7B shape the relaxed benchmark line
runs (32 users, K = 20, N = 40, tau = 1).

Step parity: every speculative step of sampled users is replayed by the oracle
on the GPU's own inputs -- its draft and target log-probs (atspeed_logprobs),
its drafted tree and the same Philox key -- and must give the GPU's drafted
levels (in draw order), accepted levels, level reached and beams exactly; a
difference is accepted only where taking one oracle decision of margin below
1e-3 (an acceptance test or a Gumbel-top-k boundary) the other way reproduces
it.  This pins the reading's list shortfall to the oracle: a level that rejects
fills its missing draws without replacement from max(0, pi_p - pi_q), and that
residual can hold fewer candidates than the draws it owes, so a user can end
with fewer than K lists.

Properties of the whole decode at the 7B shape: deterministic; tree-KV reuse
leaves the lists, scores and counts bitwise unchanged while forwarding no more
target rows; every user gets 1..K distinct catalog items with finite,
non-positive cumulative log-probs.
"""
import ctypes as C

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from _gpu_common import FlipStreams, env, relaxed_tie  # noqa: E402
from synth import get_workload, make_catalog, make_prefixes, make_weights, philox_key  # noqa: E402
from oracle.relaxed import draft_paper, verify_paper  # noqa: E402
from oracle.search import path_score, table_scorer  # noqa: E402
from oracle.trie import Trie  # noqa: E402

DEV = "cuda:0"


@pytest.fixture(scope="module")
def b7r():
    w = get_workload("b7_relaxed")
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    print("[b7_relaxed] generating weights", flush=True)
    return dict(w=w, cat=cat, pre=pre, tw=make_weights(w, "target"), dw=make_weights(w, "draft"))


def _gpu_paths(tn, tt, tp, td, u, w):
    paths = []
    for i in range(tn[u]):
        code = tt[u, i] - w.target.item_base - w.codebook * (td[u, i] - 1)
        paths.append((paths[tp[u, i]] if tp[u, i] >= 0 else ()) + (int(code),))
    return paths


def _steps_vs_oracle(eng, w, pre, trie, key, users, label):
    """Runs prefill and draft/verify steps on the GPU until every user is done;
    replays each step of ``users`` with the oracle on the GPU's own inputs."""
    B, K, L, cb, tau = w.batch, w.K, w.L, w.codebook, w.temperature
    T, nitem = eng.max_nodes, w.n_item_tokens
    eng.atspeed_prefill(torch.from_numpy(pre).to(DEV))
    acc = torch.zeros(B, dtype=torch.int32, device=DEV)
    ta = torch.zeros(B, dtype=torch.int32, device=DEV)
    tlp = torch.empty((B, T, nitem), dtype=torch.float32, device=DEV)
    dlp = torch.empty_like(tlp)
    troot = torch.empty((B, nitem), dtype=torch.float32, device=DEV)
    droot = torch.empty_like(troot)
    live, compared, ties = set(users), 0, 0
    for step in range(L):
        t0, nb0, paths0, sc0 = eng.atspeed_get_state(B)
        if (t0 >= L).all():
            break
        print(f"[{label}] step {step}: draft + verify on the GPU", flush=True)
        eng.atspeed_draft()
        tn, tt, tp, td, tq = (x.cpu().numpy() for x in eng.tree_tensors(B))
        eng.atspeed_verify(acc, ta)
        eng.atspeed_logprobs(0, tlp, troot)
        eng.atspeed_logprobs(1, dlp, droot)
        t1, nb1, paths1, sc1 = eng.atspeed_get_state(B)
        A, TA = acc.cpu().numpy(), ta.cpu().numpy()
        TL, TR, DL, DR = (x.cpu().numpy().astype(np.float64) for x in (tlp, troot, dlp, droot))
        for u in sorted(live):
            t = int(t0[u])
            if t >= L:
                continue
            J = min(w.gamma, L - t)
            nodes = _gpu_paths(tn, tt, tp, td, u, w)
            lp_tab, lq_tab = {(): TR[u]}, {(): DR[u]}
            for i, p in enumerate(nodes):
                if len(p) < L:
                    lp_tab[p] = TL[u, i]
                if len(p) < min(t + J, L):       # the draft forwards all but its deepest level
                    lq_tab[p] = DL[u, i]
            lp, lq = table_scorer(lp_tab), table_scorer(lq_tab)
            Y = ([(tuple(int(c) for c in paths0[u, k, :t]), float(sc0[u, k])) for k in range(nb0[u])]
                 if t > 0 else [((), 0.0)])
            Yq = [path_score(lq, p, cb) for p, _ in Y]
            gpu_levels = [[(p, float(tq[u, i])) for i, p in enumerate(nodes) if len(p) == lvl]
                          for lvl in range(t + 1, t + J + 1)]
            want_draft = [[p for p, _ in lvl] for lvl in gpu_levels]

            def draft(uo=None, go=None, log=None):
                try:
                    D = draft_paper(lq, trie, [p for p, _ in Y], Yq, J, w.N, cb, tau, FlipStreams(key, u, uo, go),
                                    step, log)
                except KeyError:                  # a draft that needs rows the GPU never forwarded
                    return None
                return [[p for p, _ in lvl] for lvl in D]
            log = []
            if draft(log=log) != want_draft:
                m = relaxed_tie(log, draft, lambda d: d == want_draft)
                assert m is not None, (label, u, step, "drafted levels differ outside the tie zone")
                print(f"[{label}] user {u} step {step}: drafting differs at a near-tie (margin {m:.2e})")
                ties += 1
                live.discard(u)
                continue
            got = (int(TA[u]), int(A[u]), [tuple(int(c) for c in paths1[u, k, :t1[u]]) for k in range(nb1[u])])

            def verify(uo=None, go=None, log=None):
                return verify_paper(lp, lq, trie, Y, Yq, gpu_levels, K, L, cb, tau, FlipStreams(key, u, uo, go),
                                    step, log)

            def same(r):
                return (r.t_after, r.accepted, [p for p, _ in r.beams]) == got
            log = []
            res = verify(log=log)
            if not same(res):
                m = relaxed_tie(log, verify, same)
                assert m is not None, (label, u, step, got, (res.t_after, res.accepted, [p for p, _ in res.beams]))
                print(f"[{label}] user {u} step {step}: verification differs at a near-tie (margin {m:.2e})")
                ties += 1
                live.discard(u)
                continue
            np.testing.assert_allclose(sc1[u, :nb1[u]], [s for _, s in res.beams], rtol=0, atol=1e-4)
            compared += 1
            print(f"[{label}] user {u} step {step}: t {t} -> {got[0]}, accepted {got[1]}, {len(got[2])} beams "
                  f"(oracle equal)")
    t, nb, _, _ = eng.atspeed_get_state(B)
    assert (t == L).all()
    print(f"[{label}] {compared} user-steps equal to the oracle, {ties} decided at a near-tie; lists per "
          f"compared user {[int(nb[u]) for u in users]} of K = {K}; batch mean {nb.mean():.1f}")
    return compared


def test_small_relaxed_paper_steps_match_oracle():
    from paper_2410_05165_amd.binding import Engine
    e = env("small", mode="relaxed_paper")
    w = e["w"]
    k = philox_key(w)
    key = [int(k[0]), int(k[1])]
    eng = Engine(w, e["tw"], e["dw"], e["cat"], mode=2, seed=key[0] | (key[1] << 32))
    try:
        assert _steps_vs_oracle(eng, w, e["pre"], e["trie"], key, [0, 3, 6, 9, 12, 15], "small relaxed") > 0
    finally:
        eng.close()


def test_b7_relaxed_steps_match_oracle(b7r):
    from paper_2410_05165_amd.binding import Engine
    w = b7r["w"]
    k = philox_key(w)
    key = [int(k[0]), int(k[1])]
    eng = Engine(w, b7r["tw"], b7r["dw"], b7r["cat"], mode=2, seed=key[0] | (key[1] << 32))
    try:
        print("[b7_relaxed] oracle trie of 100k items", flush=True)
        trie = Trie(b7r["cat"])
        assert _steps_vs_oracle(eng, w, b7r["pre"], trie, key, [0, 10, 21, 31], "b7 relaxed") > 0
    finally:
        eng.close()


def _decode(eng, w, prefix):
    from paper_2410_05165_amd.binding import Stats
    items = torch.zeros((w.batch, w.K, w.L), dtype=torch.int32, device=DEV)
    scores = torch.zeros((w.batch, w.K), dtype=torch.float32, device=DEV)
    n = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
    acc = np.full((w.L, w.batch), -9, np.int32)
    st = Stats()
    st.accepted = acc.ctypes.data_as(C.POINTER(C.c_int32))
    eng.atspeed_decode_topk(prefix, items, scores, n, st)
    torch.cuda.synchronize()
    return (items.cpu().numpy(), scores.cpu().numpy(), n.cpu().numpy(), acc[:st.n_steps].copy()), st


def test_b7_relaxed_decode_properties(b7r):
    from paper_2410_05165_amd.binding import Engine
    w, cat, pre, tw, dw = b7r["w"], b7r["cat"], b7r["pre"], b7r["tw"], b7r["dw"]
    prefix = torch.from_numpy(pre).to(DEV)
    eng0 = Engine(w, tw, dw, cat, mode=2, seed=7)
    eng1 = Engine(w, tw, dw, cat, mode=2, seed=7, reuse_tree_kv=1)
    try:
        print("[b7_relaxed] decode twice without reuse, once with", flush=True)
        a, st_a = _decode(eng0, w, prefix)
        b, _ = _decode(eng0, w, prefix)
        c, st_c = _decode(eng1, w, prefix)
        print(f"[b7_relaxed] steps {st_a.n_steps}, target rows {st_a.rows_target} -> {st_c.rows_target}")
        for x, y, z in zip(a, b, c):
            np.testing.assert_array_equal(x, y)
            np.testing.assert_array_equal(x, z)
        assert 0 < st_c.rows_target <= st_a.rows_target
        items, scores, n, _ = a
        assert ((n >= 1) & (n <= w.K)).all(), n
        print(f"[b7_relaxed] lists per user: min {n.min()}, mean {n.mean():.1f}, max {n.max()}")
        key = lambda rows: ((rows[..., 0] * 256 + rows[..., 1]) * 256 + rows[..., 2]) * 256 + rows[..., 3]
        catalog = set(key(cat.astype(np.int64)).tolist())
        for u in range(w.batch):
            ks = key(items[u, :n[u]].astype(np.int64)).tolist()
            assert len(set(ks)) == n[u], u
            assert all(k in catalog for k in ks), u
            assert np.isfinite(scores[u, :n[u]]).all() and (scores[u, :n[u]] <= 0).all(), u
    finally:
        eng1.close()
        eng0.close()
