"""Draft alignment on the GPU (AtSpeed-S, Sec. 3.1; AtSpeed-R, Sec. 3.2) against
the oracle, on the small workload (16 users, K = 20, a 2-layer bf16 draft).

The batch is every user's K target lists (a strict decode, lossless: the
target's own top-K, i.e. D' with lambda = 1), or the multi-step data below;
the contexts are the users' roots and the distinct proper prefixes of those
sequences.

* atspeed_align_data: the context tree holds exactly those prefixes, level
  ordered, each node's parent its own prefix; node and root weights equal the
  oracle's dataset weights; log p_K is the target's log-prob of the K-th list's
  code at its own prefix, read from the same target rows; the target rows equal
  the oracle target's log-probs at those contexts (bf16 logit bar, doubled for
  the log-normaliser).
* atspeed_align_step: the loss and the item-head gradient equal the oracle's
  on the GPU's own draft and target log-probs and hidden states; the hidden
  rows reproduce the draft's log-probs through the head (so each row sits at
  its context's slot); the AdamW update equals the oracle's on the GPU's
  gradient; the head the draft reads is the master copy rounded to bf16, bit
  for bit.
* training: the loss falls, the decoded lists stay the target's (strict
  verification is lossless whatever the draft), and acceptance rises (strict
  decoding after AtSpeed-S, relaxed sampling decoding after AtSpeed-R).

Multi-step data (the target's K beams of every beam-search step, which the
paper compares with last-step data) come from atspeed_target_search, the
GPU's target-only beam search, whose lists and per-level beams are checked
against the strict decode and against a host-driven route (verifies of
uploaded trees that hold only the Y_t paths).
"""
import ctypes as C

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from _gpu_common import LOGIT_TOL, env, oracle_user, upload_tree  # noqa: E402
from oracle.align import adamw_step, aligned_loss, head_gradient  # noqa: E402
from oracle.model import item_log_softmax  # noqa: E402
from oracle.numerics import round_bf16  # noqa: E402

DEV = "cuda:0"


def _decode(eng, w, prefix):
    from paper_2410_05165_amd.binding import Stats
    B = prefix.shape[0]
    items = torch.zeros((B, w.K, w.L), dtype=torch.int32, device=DEV)
    scores = torch.zeros((B, w.K), dtype=torch.float32, device=DEV)
    n = torch.zeros(B, dtype=torch.int32, device=DEV)
    acc = np.full((w.L, B), -9, np.int32)
    st = Stats()
    st.accepted = acc.ctypes.data_as(C.POINTER(C.c_int32))
    eng.atspeed_decode_topk(prefix, items, scores, n, st)
    torch.cuda.synchronize()
    return items, n, acc[:st.n_steps].copy()


def _mean_accepted(acc):
    a = acc[acc >= 0]
    return float(a.mean()) if a.size else 0.0


def _py_level_beams(eng, w, prefix):
    """Multi-step data built on the host: per level, the tree of the Y_t paths
    uploaded through the tree pointers and verified (an independent route to
    the target-only beam search)."""
    B, K, L = prefix.shape[0], w.K, w.L
    eng.atspeed_prefill(prefix)
    levels = []
    for _ in range(L):
        t, nb, paths, _ = eng.atspeed_get_state(B)
        trees = [[tuple(int(c) for c in paths[u, k, :t[u]]) for k in range(nb[u])] if t[u] > 0 else []
                 for u in range(B)]
        upload_tree(eng, trees, B)
        eng.atspeed_verify()
        levels.append(eng.atspeed_get_state(B))
    items = np.zeros((B, K * L, L), np.int32)
    lens = np.zeros((B, K * L), np.int32)
    n = np.zeros(B, np.int32)
    for u in range(B):
        for t_, nb, paths, _ in levels:
            for k in range(nb[u]):
                items[u, n[u], :t_[u]] = paths[u, k, :t_[u]]
                lens[u, n[u]] = t_[u]
                n[u] += 1
    return items, lens, n


def _level_beams(eng, w, prefix):
    """Multi-step data: the target's K beams of every beam-search step
    (atspeed_target_search), items [B, K*L, L], lens, n; levels in order."""
    B, K, L = prefix.shape[0], w.K, w.L
    items = torch.zeros((B, K, L), dtype=torch.int32, device=DEV)
    scores = torch.zeros((B, K), dtype=torch.float32, device=DEV)
    n = torch.zeros(B, dtype=torch.int32, device=DEV)
    si = torch.full((B, K * L, L), -1, dtype=torch.int32, device=DEV)
    sl = torch.full((B, K * L), -1, dtype=torch.int32, device=DEV)
    sn = torch.full((B,), -1, dtype=torch.int32, device=DEV)
    eng.atspeed_target_search(prefix, items, scores, n, si, sl, sn)
    return si, sl, sn


def _setup(mode, multistep=False, name="small", **hp):
    from paper_2410_05165_amd.align import AlignTrainer
    from paper_2410_05165_amd.binding import Engine
    e = env(name)
    w = e["w"]
    eng = Engine(w, e["tw"], e["dw"], e["cat"])
    prefix = torch.from_numpy(e["pre"]).to(DEV)
    print(f"[align {mode}] strict decode for the target lists", flush=True)
    items, n, acc = _decode(eng, w, prefix)
    decoded = (items, n)
    lens = None
    if multistep:
        items_l, lens, n_l = _level_beams(eng, w, prefix)
        # the last step's beams are the decoded lists
        whole, ms = _lists((items, None, n)), _lists((items_l, lens, n_l))
        assert all(ms[u][len(ms[u]) - len(whole[u]):] == whole[u] for u in range(len(whole)))
        items, n = items_l, n_l
    eng.atspeed_prefill(prefix)
    tr = AlignTrainer(eng, mode, **hp)
    tr.data(items, n, lens)
    torch.cuda.synchronize()
    return e, eng, prefix, tr, (items, lens, n), acc, decoded


def _contexts(eng, B):
    """Per user: {path: slot} of the context tree (paths rebuilt through the parents)."""
    w = eng.w
    tn, tt, tp, td, _ = (x.cpu().numpy() for x in eng.tree_tensors(B))
    out = []
    for u in range(B):
        paths = []
        for i in range(tn[u]):
            code = tt[u, i] - w.target.item_base - w.codebook * (td[u, i] - 1)
            paths.append((paths[tp[u, i]] if tp[u, i] >= 0 else ()) + (int(code),))
        out.append(paths)
    return out, td, tn


def _lists(data):
    items, lens, n = data
    it, nn = items.cpu().numpy(), n.cpu().numpy()
    ln = lens.cpu().numpy() if lens is not None else np.full(it.shape[:2], it.shape[2])
    return [[tuple(int(c) for c in it[u, k, :ln[u, k]]) for k in range(nn[u])] for u in range(len(nn))]


@pytest.mark.parametrize("reuse", [0, 1])
def test_target_search_small(reuse):
    """atspeed_target_search: the lists equal the strict speculative decode's
    (and so the oracle's beam search, by the decode's own parity tests); every
    level's beams equal those of the host-driven route, bitwise."""
    from paper_2410_05165_amd.binding import Engine
    e = env("small")
    w = e["w"]
    B, K, L = w.batch, w.K, w.L
    eng = Engine(w, e["tw"], e["dw"], e["cat"], reuse_tree_kv=reuse)
    try:
        prefix = torch.from_numpy(e["pre"]).to(DEV)
        items0, n0, _ = _decode(eng, w, prefix)
        items = torch.zeros((B, K, L), dtype=torch.int32, device=DEV)
        scores = torch.zeros((B, K), dtype=torch.float32, device=DEV)
        n = torch.zeros(B, dtype=torch.int32, device=DEV)
        eng.atspeed_target_search(prefix, items, scores, n)
        assert torch.equal(items, items0) and torch.equal(n, n0)
        si, sl, sn = (x.cpu().numpy() for x in _level_beams(eng, w, prefix))
        pi, pl, pn = _py_level_beams(eng, w, prefix)
        assert np.array_equal(sn, pn)
        for u in range(B):
            assert np.array_equal(si[u, :sn[u]], pi[u, :pn[u]]) and np.array_equal(sl[u, :sn[u]], pl[u, :pn[u]]), u
        assert (sl[:, :K] == 1).all() and all((sl[u, sn[u] - n0[u].item():sn[u]] == L).all() for u in range(B))
        # a target-only prefill leaves the draft's caches stale
        with pytest.raises(Exception, match="prefill"):
            eng.atspeed_target_search(prefix, items, scores, n)
            eng.atspeed_draft()
        print(f"[target search, reuse {reuse}] {int(sn.sum())} beams over {L} levels, lists equal the decode's")
    finally:
        eng.close()


@pytest.mark.parametrize("multistep", [False, True], ids=["last_step", "multi_step"])
def test_align_data_small(multistep):
    e, eng, prefix, tr, data, _, _ = _setup("S", multistep)
    try:
        w = e["w"]
        B, T, L, cb, nit = w.batch, eng.max_nodes, w.L, w.codebook, eng.n_item
        Y = _lists(data)
        paths, depth, nn = _contexts(eng, B)
        cw = tr.ctx_weight.view(B, T).cpu().numpy()
        lw = tr.label_weight.view(B, T).cpu().numpy()
        rw = tr.root_weight.cpu().numpy()
        lpk = tr.log_pK.view(B, L).cpu().numpy()
        LPT = tr.lp_target.view(B, T, nit).cpu().numpy()
        RT = tr.root_target.view(B, nit).cpu().numpy()
        from oracle.align import context_weights, label_distributions
        W = context_weights(Y, L)
        for u in range(B):
            want = {y[:t] for y in Y[u] for t in range(1, len(y) + 1)}
            got = paths[u]
            assert len(got) == len(set(got)) == len(want) and set(got) == want, u
            assert all(depth[u, i] <= depth[u, i + 1] for i in range(nn[u] - 1)), u
            pis = label_distributions(Y[u], cb)
            for i, p in enumerate(got):
                assert cw[u, i] == pytest.approx(W[u].get(p, 0.0), rel=1e-6, abs=1e-9), (u, p)
                parent_w = W[u][p[:-1]]
                assert lw[u, i] == pytest.approx(parent_w * pis[p[:-1]][cb * (len(p) - 1) + p[-1]], rel=1e-5), (u, p)
            assert rw[u] == pytest.approx(W[u][()], rel=1e-6), u
            yk = Y[u][-1]
            slot = {p: i for i, p in enumerate(got)}
            for t in range(L):
                row = RT[u] if t == 0 else LPT[u, slot[yk[:t]]]
                assert lpk[u, t] == row[cb * t + yk[t]], (u, t)
        if multistep:
            return
        bar = 2 * LOGIT_TOL[w.dtype]
        for u in (0, 7):
            o = oracle_user("small", u)
            ctx = [()] + [p for p in paths[u] if len(p) == 1][:2] + [p for p in paths[u] if len(p) == 3][:2]
            want = o["lp"](ctx)
            for p, row in zip(ctx, want):
                got = RT[u] if p == () else LPT[u, paths[u].index(p)]
                err = np.abs(got - row).max()
                print(f"[align data] user {u} context {p}: target log-prob max|err| = {err:.3e}")
                assert err <= bar
    finally:
        eng.close()


@pytest.mark.parametrize("name,mode,alpha,multistep", [
    ("small", "S", 1.0, False), ("small", "R", 1.0, False), ("small", "S", 0.5, False), ("small", "S", 0.5, True),
    ("small", "R", 0.5, True), ("tiny", "S", 0.5, True), ("tiny", "R", 0.5, False)])
def test_align_step_matches_oracle(name, mode, alpha, multistep):
    """One step against the oracle: bf16 at the small shape, fp32 at the tiny one
    (the fp32 instantiations of the head-gradient, hidden-row and AdamW kernels;
    an fp32 head is the master copy itself)."""
    hp = dict(alpha=alpha, lr=2e-3, betas=(0.9, 0.99), eps=1e-8, weight_decay=0.01)
    e, eng, prefix, tr, data, _, _ = _setup(mode, multistep, name, **hp)
    try:
        w = e["w"]
        B, T, L, cb, nit, K = w.batch, eng.max_nodes, w.L, w.codebook, eng.n_item, w.K
        d = w.draft.d_model
        head0 = tr.head.float().cpu().numpy().astype(np.float64)
        master0 = tr.master.cpu().numpy().astype(np.float64).reshape(nit, d)
        hidden = torch.full((B * (1 + T), d), float("nan"), dtype=torch.float32, device=DEV)
        loss = tr.step(hidden_out=hidden)
        dl = torch.empty((B, T, nit), dtype=torch.float32, device=DEV)
        dr = torch.empty((B, nit), dtype=torch.float32, device=DEV)
        eng.atspeed_logprobs(1, dl, dr)
        DL, DR = dl.cpu().numpy().astype(np.float64), dr.cpu().numpy().astype(np.float64)
        LPT = tr.lp_target.view(B, T, nit).cpu().numpy().astype(np.float64)
        RT = tr.root_target.view(B, nit).cpu().numpy().astype(np.float64)
        H = hidden.cpu().numpy().astype(np.float64)
        G = tr.grad.view(nit, d).cpu().numpy().astype(np.float64)
        master = tr.master.view(nit, d).cpu().numpy().astype(np.float64)
        head = tr.head.float().cpu().numpy().astype(np.float64)
        paths, _, _ = _contexts(eng, B)
        slot = [{p: i for i, p in enumerate(ps)} for ps in paths]
        Y = _lists(data)

        def lq_of(u, p):
            return DR[u] if p == () else DL[u, slot[u][p]]

        def lp_of(u, p):
            return RT[u] if p == () else LPT[u, slot[u][p]]

        def h_of(u, p):
            return H[u] if p == () else H[B + u * T + slot[u][p]]

        want_loss, grads = aligned_loss(mode, lq_of, lp_of, e["trie"], Y, K, L, cb, alpha)
        tag = f"[align {name} {mode} alpha {alpha}{' multi-step' if multistep else ''}]"
        print(f"{tag} loss GPU {loss:.8f} oracle {want_loss:.8f}; {len(grads)} contexts", flush=True)
        assert abs(loss - want_loss) <= 1e-5 * abs(want_loss) + 1e-7
        hid = {k: h_of(*k) for k in grads}
        want_G = head_gradient(grads, hid)
        scale = np.abs(want_G).max()
        err = np.abs(G - want_G).max()
        print(f"{tag} head gradient max|err| = {err:.3e} (max|dW| {scale:.3e})")
        assert scale > 0 and err <= 1e-4 * scale
        # the hidden rows are the contexts' own: through the head they give the draft's log-probs
        worst = 0.0
        for (u, p), h in list(hid.items())[::7]:
            lq = item_log_softmax(head0 @ h)
            worst = max(worst, np.abs(lq - lq_of(u, p)).max())
        print(f"{tag} log_softmax(head h) vs draft log-probs max|err| = {worst:.3e}")
        assert worst <= 1e-3
        # AdamW on the GPU's gradient, then the bf16 head
        want_w, _, _ = adamw_step(master0, 0.0, 0.0, G, 1, hp["lr"], hp["betas"][0], hp["betas"][1], hp["eps"],
                                  hp["weight_decay"])
        np.testing.assert_allclose(master, want_w, rtol=1e-6, atol=1e-6 * hp["lr"])
        assert np.array_equal(head, round_bf16(master) if w.dtype == "bf16" else master)
        assert not np.array_equal(head, head0)
    finally:
        eng.close()


def _relaxed_decode(eng, w, prefix):
    items, n, acc = _decode(eng, w, prefix)
    return n.float().mean().item(), acc


@pytest.mark.parametrize("mode", ["S", "R"])
def test_align_training_small(mode):
    """200 AdamW steps on the multi-step data (alpha 0.5).  S: the strict decode's
    lists stay the target's and the trained users' accepted levels rise.  R: the
    head is trained on the relaxed engine (its draft), whose sampled decode then
    accepts more levels per step and yields no fewer lists."""
    from paper_2410_05165_amd.align import AlignTrainer, cosine_lr
    from paper_2410_05165_amd.binding import Engine
    steps, peak = 200, 1e-2
    e, eng, prefix, tr, data, acc0, (items0, n0) = _setup(mode, True, alpha=0.5, lr=peak, weight_decay=0.01)
    w = e["w"]
    reng = None
    try:
        if mode == "R":
            reng = Engine(w, e["tw"], e["dw"], e["cat"], mode=2, seed=11)
            lists0, racc0 = _relaxed_decode(reng, w, prefix)
            reng.atspeed_prefill(prefix)
            tr = AlignTrainer(reng, "R", alpha=0.5, lr=peak, weight_decay=0.01)
            items, lens, n = data
            tr.data(items, n, lens)
        losses = [tr.step(lr=cosine_lr(s, steps, peak, 10)) for s in range(1, steps + 1)]
        print(f"[align {mode}] loss {losses[0]:.5f} -> {losses[steps // 2]:.5f} -> {losses[-1]:.5f}")
        assert losses[-1] < losses[0]
        if mode == "S":
            items1, n1, acc1 = _decode(eng, w, prefix)
            assert torch.equal(items0, items1) and torch.equal(n0, n1)   # lossless whatever the draft
            m0, m1 = _mean_accepted(acc0), _mean_accepted(acc1)
            print(f"[align S] strict decode: accepted levels per step {m0:.3f} -> {m1:.3f}; "
                  f"steps {acc0.shape[0]} -> {acc1.shape[0]}")
            assert m1 > m0
        else:
            lists1, racc1 = _relaxed_decode(reng, w, prefix)
            m0, m1 = _mean_accepted(racc0), _mean_accepted(racc1)
            print(f"[align R] relaxed decode: accepted levels per step {m0:.3f} -> {m1:.3f}; "
                  f"lists per user {lists0:.2f} -> {lists1:.2f}")
            assert m1 > m0 and lists1 >= lists0
    finally:
        if reng is not None:
            reng.close()
        eng.close()


def test_align_errors_leave_a_usable_context():
    """Argument and state errors of the alignment calls, each caught by the host
    checks or by the context-tree kernel's own validation before any access it
    could not bound: the call returns its status and a valid batch then works."""
    from paper_2410_05165_amd.align import AlignTrainer
    from paper_2410_05165_amd.binding import AtspeedError, Engine
    e = env("small")
    w = e["w"]
    B, K, L = w.batch, w.K, w.L
    eng = Engine(w, e["tw"], e["dw"], e["cat"])
    inv, state = 1, 5          # ATSPEED_E_INVALID, ATSPEED_E_STATE
    try:
        prefix = torch.from_numpy(e["pre"]).to(DEV)
        items, n, _ = _decode(eng, w, prefix)
        eng.atspeed_prefill(prefix)
        tr = AlignTrainer(eng, "S", alpha=0.5)
        with pytest.raises(AtspeedError) as ex:           # a step before any batch
            tr.step()
        assert ex.value.status == state
        cases = []
        bad = items.clone(); bad[3, 0, 2] = w.codebook + 40           # code out of range
        cases.append(("code out of range", bad, n, None))
        cat = set(map(tuple, e["cat"].tolist()))
        probe = next((a, b, c, d) for a in range(3) for b in range(256) for c in range(3) for d in range(3)
                     if (a, b, c, d) not in cat)
        bad = items.clone(); bad[5, 1] = torch.tensor(probe, dtype=torch.int32)   # not a catalog item
        cases.append(("not in the catalog", bad, n, None))
        bad_n = n.clone(); bad_n[2] = 0
        cases.append(("no sequences", items, bad_n, None))
        bad_n = n.clone(); bad_n[2] = K + 1
        cases.append(("more sequences than S", items, bad_n, None))
        lens = torch.full((B, K), L, dtype=torch.int32, device=DEV); lens[0, n[0] - 1] = 2
        cases.append(("last sequence shorter than L", items, n, lens))
        lens = torch.full((B, K), L, dtype=torch.int32, device=DEV); lens[4, 0] = L + 1
        cases.append(("length above L", items, n, lens))
        for what, it, nn, ll in cases:
            with pytest.raises(AtspeedError) as ex:
                tr.data(it, nn, ll)
            assert ex.value.status == inv, what
            print(f"[align errors] {what}: ATSPEED_E_INVALID")
            with pytest.raises(AtspeedError) as ex:       # the failed batch is not trainable
                tr.step()
            assert ex.value.status == state, what
        tr.data(items, n)
        tr.args.alpha = 1.5
        with pytest.raises(AtspeedError) as ex:
            tr.step()
        assert ex.value.status == inv
        tr.args.alpha = 0.5
        tr.args.step = 0
        assert np.isfinite(tr.step())
    finally:
        eng.close()


def _search(eng, w, prefix, lam=None):
    B, K, L = prefix.shape[0], w.K, w.L
    out = (torch.zeros((B, K, L), dtype=torch.int32, device=DEV), torch.zeros((B, K), device=DEV),
           torch.zeros(B, dtype=torch.int32, device=DEV), torch.zeros((B, K * L, L), dtype=torch.int32, device=DEV),
           torch.zeros((B, K * L), dtype=torch.int32, device=DEV), torch.zeros(B, dtype=torch.int32, device=DEV))
    if lam is None:
        eng.atspeed_target_search(prefix, *out)
    else:
        eng.atspeed_mixed_search(lam, prefix, *out)
    torch.cuda.synchronize()
    return tuple(x.cpu().numpy() for x in out)


def _level_paths(si, sl, sn, u, t):
    return [tuple(int(c) for c in si[u, i, :t]) for i in range(sn[u]) if sl[u, i] == t]


@pytest.mark.parametrize("reuse", [0, 1])
def test_mixed_search_lambda_one_is_the_target_search(reuse):
    from paper_2410_05165_amd.binding import Engine
    e = env("small")
    w = e["w"]
    eng = Engine(w, e["tw"], e["dw"], e["cat"], reuse_tree_kv=reuse)
    try:
        prefix = torch.from_numpy(e["pre"]).to(DEV)
        a = _search(eng, w, prefix)
        b = _search(eng, w, prefix, 1.0)
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
        c = _search(eng, w, prefix, 0.5)
        assert not np.array_equal(a[0], c[0])       # the mixture moves the lists
    finally:
        eng.close()


@pytest.mark.parametrize("lam", [0.5, 0.2])
def test_mixed_search_tiny_matches_oracle(lam):
    """fp32: every level's beams equal the oracle's mixture beam search over its
    own target and draft (fp64), outside a near-tie (the first differing level's
    top-K decision has a margin below 1e-3, and the comparison stops there);
    the final scores within 1e-4."""
    from paper_2410_05165_amd.binding import Engine
    from oracle.align import mixture_beam_search
    e = env("tiny")
    w = e["w"]
    eng = Engine(w, e["tw"], e["dw"], e["cat"])
    try:
        prefix = torch.from_numpy(e["pre"]).to(DEV)
        items, scores, n, si, sl, sn = _search(eng, w, prefix, lam)
        o = oracle_user("tiny", 0)
        log = []
        levels = mixture_beam_search(lambda p: o["lp"]([p])[0], lambda p: o["lq"]([p])[0], e["trie"], w.K, w.L,
                                     w.codebook, lam, log)
        for t, lvl in enumerate(levels, 1):
            got = sorted(_level_paths(si, sl, sn, 0, t))
            want = sorted(p for p, _ in lvl)
            if got != want:
                assert log[t - 1].margin < 1e-3, (t, got, want)
                print(f"[mixed tiny] level {t} differs at a near-tie (margin {log[t - 1].margin:.2e})")
                return
        gs = {tuple(int(c) for c in items[0, k]): float(scores[0, k]) for k in range(n[0])}
        for p, s in levels[-1]:
            assert abs(gs[p] - s) <= 1e-4, (p, gs[p], s)
        print(f"[mixed tiny] lambda {lam}: all {w.L} levels equal the oracle")
    finally:
        eng.close()


def test_mixed_search_small_level1_on_shared_rows():
    """bf16: the first level of the mixture search equals the oracle's TopK of
    the mixture of the GPU's own root rows (target and draft, from a prefill),
    outside near-ties."""
    from paper_2410_05165_amd.binding import Engine
    from oracle.align import mixed_log
    from oracle.search import top_boundary
    e = env("small")
    w = e["w"]
    B, T, nit = w.batch, None, w.n_item_tokens
    eng = Engine(w, e["tw"], e["dw"], e["cat"])
    try:
        prefix = torch.from_numpy(e["pre"]).to(DEV)
        eng.atspeed_prefill(prefix)
        T = eng.max_nodes
        lp = torch.empty((B, T, nit), device=DEV)
        tr = torch.empty((B, nit), device=DEV)
        dr = torch.empty((B, nit), device=DEV)
        eng.atspeed_logprobs(0, lp, tr)
        eng.atspeed_logprobs(1, lp, dr)
        TR, DR = tr.cpu().numpy().astype(np.float64), dr.cpu().numpy().astype(np.float64)
        lam = 0.5
        items, scores, n, si, sl, sn = _search(eng, w, prefix, lam)
        equal = 0
        for u in range(B):
            m = mixed_log(DR[u], TR[u], lam)
            cands = [((c,), float(m[c])) for c in e["trie"].children(())]
            sel, margin, _ = top_boundary(cands, w.K)
            got = sorted(_level_paths(si, sl, sn, u, 1))
            if got != sorted(p for p, _ in sel):
                assert margin < 1e-3, (u, margin)
                continue
            equal += 1
        print(f"[mixed small] level 1: {equal} of {B} users equal, the rest at near-ties")
        assert equal >= B - 2
    finally:
        eng.close()
