"""Relaxed sampling verification (the paper's reading of Algorithm 2) at the full
7B shape the relaxed benchmark line runs: 32 users, K = 20, N = 40, tau = 1.

The oracle cannot decode this batch, and a relaxed decode has no closed-form
output, so the test checks what holds at any size on the same Philox streams:
the decode is deterministic; tree-KV reuse leaves the lists, scores and counts
bitwise unchanged while forwarding no more target rows; and every user gets
between 1 and K distinct catalog items with finite, non-positive cumulative
log-probs.  (Fewer than K is the reading's own outcome: a level that rejects
fills its missing draws without replacement from max(0, pi_p - pi_q), and that
residual can hold fewer candidates than the draws it owes.)  (Small
shapes compare the relaxed path with the oracle element by element, and pin
its laws by chi-square.)
"""
import ctypes as C

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from synth import get_workload, make_catalog, make_prefixes, make_weights  # noqa: E402

DEV = "cuda:0"


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


def test_b7_relaxed_decode_properties():
    from paper_2410_05165_amd.binding import Engine
    w = get_workload("b7_relaxed")
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    print("[b7_relaxed] generating weights", flush=True)
    tw, dw = make_weights(w, "target"), make_weights(w, "draft")
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
