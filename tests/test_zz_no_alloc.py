"""The allocation-free accept (atspeed_accept_noalloc): its selection and
acceptance state equals atspeed_accept's, bitwise, on the same logits and tree,
for strict and relaxed verification, on two calls in a row with the second on a
smaller batch (the static scratch keeps the first call's contents); and a batch
whose buffers exceed the static scratch is refused before any launch."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from _gpu_common import env  # noqa: E402

DEV = "cuda:0"


def _step(eng_a, eng_b, w, prefix):
    B = prefix.shape[0]
    roots = []
    for eng in (eng_a, eng_b):
        root = torch.zeros((B, w.n_item_tokens), dtype=torch.float32, device=DEV)
        eng.atspeed_prefill(prefix, root)
        eng.atspeed_draft()
        roots.append(root)
    ta_, tb_ = ([x.cpu().numpy() for x in e.tree_tensors(B)] for e in (eng_a, eng_b))
    np.testing.assert_array_equal(ta_[0], tb_[0])
    for x, y in zip(ta_[1:], tb_[1:]):          # slots past a user's n_nodes are undefined
        for u in range(B):
            np.testing.assert_array_equal(x[u, :ta_[0][u]], y[u, :ta_[0][u]])
    logits = torch.zeros((B, eng_a.max_nodes, w.n_item_tokens), dtype=torch.float32, device=DEV)
    eng_a.atspeed_tree_logits(logits)
    np.testing.assert_array_equal(roots[0].cpu().numpy(), roots[1].cpu().numpy())
    acc = [torch.full((B,), -7, dtype=torch.int32, device=DEV) for _ in range(2)]
    tafter = [torch.full((B,), -7, dtype=torch.int32, device=DEV) for _ in range(2)]
    eng_a.atspeed_accept(logits, roots[0], acc[0], tafter[0])
    eng_b.atspeed_accept_noalloc(logits, roots[0], acc[1], tafter[1])
    np.testing.assert_array_equal(acc[0].cpu().numpy(), acc[1].cpu().numpy())
    np.testing.assert_array_equal(tafter[0].cpu().numpy(), tafter[1].cpu().numpy())
    sa, sb = eng_a.atspeed_get_state(B), eng_b.atspeed_get_state(B)
    for x, y in zip(sa, sb):
        np.testing.assert_array_equal(x, y)
    return sa


@pytest.mark.parametrize("mode", ["strict", "relaxed_paper"])
def test_noalloc_accept_equals_accept(mode):
    from paper_2410_05165_amd.binding import Engine
    e = env("small", mode=mode)
    w = e["w"]
    m = {"strict": 0, "relaxed_paper": 2}[mode]
    eng_a = Engine(w, e["tw"], e["dw"], e["cat"], mode=m, seed=11)
    eng_b = Engine(w, e["tw"], e["dw"], e["cat"], mode=m, seed=11)
    try:
        prefix = torch.from_numpy(e["pre"]).to(DEV)
        for B in (w.batch, 4):                  # the second call on a smaller batch
            print(f"[noalloc {mode}] accept vs accept_noalloc, B = {B}", flush=True)
            t, nb, _, _ = _step(eng_a, eng_b, w, prefix[:B])
            print(f"[noalloc {mode}] B = {B}: equal; levels reached {t.tolist()}", flush=True)
    finally:
        eng_b.close()
        eng_a.close()


def test_noalloc_accept_refuses_a_batch_above_the_scratch():
    from paper_2410_05165_amd.binding import AtspeedError, Engine
    e = env("tiny", K=128, N=128, batch=64)
    w = e["w"]
    eng = Engine(w, e["tw"], e["dw"], e["cat"])
    try:
        prefix = torch.from_numpy(e["pre"]).to(DEV)
        root = torch.zeros((w.batch, w.n_item_tokens), dtype=torch.float32, device=DEV)
        eng.atspeed_prefill(prefix, root)
        logits = torch.zeros((w.batch, eng.max_nodes, w.n_item_tokens), dtype=torch.float32, device=DEV)
        before = eng.atspeed_get_state(w.batch)
        print("[noalloc] 64 users x 896 slots x 1,024 log-probs (235 MB) against the 64 MiB scratch", flush=True)
        with pytest.raises(AtspeedError) as ex:
            eng.atspeed_accept_noalloc(logits, root)
        assert ex.value.status == 3 and "static scratch" in str(ex.value)
        for x, y in zip(before, eng.atspeed_get_state(w.batch)):
            np.testing.assert_array_equal(x, y)
    finally:
        eng.close()
