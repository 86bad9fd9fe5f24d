"""Tree-KV reuse (reuse_tree_kv = 1): each verify of atspeed_decode_topk takes
the target K/V and log-probs of the nodes the previous verify forwarded (same
depth and path: Y_t paths, accepted levels) instead of forwarding them again.
A node's K/V depends only on the prefix and its path, and every kernel is
batch-invariant, so the lists, scores, counts and per-step acceptance must be
bitwise those of the decode without reuse, while the target forwards fewer
tree rows whenever a node recurs."""
import ctypes as C

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from synth import get_workload, make_catalog, make_prefixes, make_weights  # noqa: E402

DEV = "cuda:0"


def _case(name):
    if name == "tiny_same_g1":
        # the draft is the target and drafts one level per step: every level is
        # accepted, and each step's Y_t paths were forwarded by the step before
        base = get_workload("tiny")
        w = base.with_(draft=base.target, gamma=1, name=name)
        cat = make_catalog(w)
        tw = make_weights(w, "target")
        return w, cat, make_prefixes(w, cat), tw, tw
    w = get_workload(name)
    cat = make_catalog(w)
    return w, cat, make_prefixes(w, cat), make_weights(w, "target"), make_weights(w, "draft")


def _decode(eng, w, prefix):
    from paper_2410_05165_amd.binding import Stats
    items = torch.zeros((w.batch, w.K, w.L), dtype=torch.int32, device=DEV)
    scores = torch.zeros((w.batch, w.K), dtype=torch.float32, device=DEV)
    n = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
    # the library writes step s's row at s * max_batch: size the array by the context
    acc = np.full((w.L, eng.cfg.max_batch), -9, np.int32)
    st = Stats()
    st.accepted = acc.ctypes.data_as(C.POINTER(C.c_int32))
    eng.atspeed_decode_topk(prefix, items, scores, n, st)
    torch.cuda.synchronize()
    return (items.cpu().numpy(), scores.cpu().numpy(), n.cpu().numpy(), acc[:st.n_steps, :w.batch].copy()), st


@pytest.mark.parametrize("name,mode,start", [
    ("tiny", 0, 0), ("tiny", 0, 1), ("small", 0, 0), ("small", 0, 1), ("tiny_same_g1", 0, 0),
    ("tiny", 1, 0), ("tiny", 2, 0)])
def test_reuse_is_lossless_and_skips_rows(name, mode, start):
    from paper_2410_05165_amd.binding import Engine
    w, cat, pre, tw, dw = _case(name)
    prefix = torch.from_numpy(pre).to(DEV)
    eng0 = Engine(w, tw, dw, cat, mode=mode, seed=3, sd_start_level=start, reuse_tree_kv=0)
    eng1 = Engine(w, tw, dw, cat, mode=mode, seed=3, sd_start_level=start, reuse_tree_kv=1)
    try:
        print(f"[{name} mode {mode} start {start}] decode without and with tree-KV reuse", flush=True)
        ref, st0 = _decode(eng0, w, prefix)
        got, st1 = _decode(eng1, w, prefix)
        # a second call on the same context starts from a fresh prefill (no stale carry)
        again, st2 = _decode(eng1, w, prefix)
        print(f"[{name}] steps {st0.n_steps}, target rows {st0.rows_target} -> {st1.rows_target}")
        for x, y, z in zip(got, ref, again):
            np.testing.assert_array_equal(x, y)
            np.testing.assert_array_equal(z, y)
        assert st1.n_steps == st0.n_steps and st2.rows_target == st1.rows_target
        assert 0 < st1.rows_target <= st0.rows_target
        if name == "tiny_same_g1":
            assert st0.n_steps > 1 and st1.rows_target < st0.rows_target
    finally:
        eng1.close()
        eng0.close()


def test_public_verify_forwards_whole_tree_with_reuse_configured():
    """atspeed_verify never carries: on a reuse context two draft + verify steps
    give the same accepted levels, levels reached and final beams as on a plain
    context, after a decode call on it left carried state behind."""
    from paper_2410_05165_amd.binding import Engine
    w, cat, pre, tw, dw = _case("tiny")
    prefix = torch.from_numpy(pre).to(DEV)
    outs = []
    for reuse in (0, 1):
        eng = Engine(w, tw, dw, cat, reuse_tree_kv=reuse)
        try:
            _decode(eng, w, prefix)
            eng.atspeed_prefill(prefix)
            res = []
            for _ in range(2):
                acc = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
                ta = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
                eng.atspeed_draft()
                eng.atspeed_verify(acc, ta)
                torch.cuda.synchronize()
                res.append((acc.cpu().numpy(), ta.cpu().numpy()))
            res.append(eng.atspeed_get_state(w.batch))
            outs.append(res)
        finally:
            eng.close()
    for a, b in zip(outs[0], outs[1]):
        for x, y in zip(a, b):
            np.testing.assert_array_equal(np.asarray(x), np.asarray(y))


def test_reuse_with_fewer_users_than_max_batch():
    """A context sized for 16 users decodes 5, then all 16, then 3: each call's
    lists equal those of a context without reuse (the carried slots are indexed
    by the call's own users; every prefill drops what an earlier call left)."""
    from paper_2410_05165_amd.binding import Engine
    w, cat, pre, tw, dw = _case("small")
    eng0 = Engine(w, tw, dw, cat, reuse_tree_kv=0)
    eng1 = Engine(w, tw, dw, cat, reuse_tree_kv=1)
    try:
        for b in (5, 16, 3):
            wb = w.with_(batch=b)
            prefix = torch.from_numpy(np.ascontiguousarray(pre[:b])).to(DEV)
            print(f"[small, {b} of {w.batch} users] decode without and with reuse", flush=True)
            ref, st0 = _decode(eng0, wb, prefix)
            got, st1 = _decode(eng1, wb, prefix)
            for x, y in zip(got, ref):
                np.testing.assert_array_equal(x, y)
            assert 0 < st1.rows_target <= st0.rows_target
    finally:
        eng1.close()
        eng0.close()
