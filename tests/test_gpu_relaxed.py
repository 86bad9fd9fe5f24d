"""GPU relaxed sampling verification (Sec. 3.2, Algorithm 2) against the oracle.

fp32 "tiny": every speculative step (level reached, accepted levels, beams)
equals the oracle's on the same Philox streams, in both readings.
Law of the output (RELAXED_EXACT, K = 1): the first code of each user's item
follows the target's level distribution pi_p (chi-square over equal-mass bins),
and not the draft's.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from _gpu_common import env, oracle_user  # noqa: E402
from synth import get_workload, make_catalog, make_prefixes, make_weights, philox_key  # noqa: E402
from oracle.model import Decoder, item_log_softmax  # noqa: E402
from oracle.relaxed import sd_decode_relaxed  # noqa: E402
from oracle.trie import Trie  # noqa: E402

MODES = {"relaxed_exact": 1, "relaxed_paper": 2}


def _key_seed(w):
    k = philox_key(w)
    return [int(k[0]), int(k[1])], int(k[0]) | (int(k[1]) << 32)


# (K, N, temperature): the tiny workload's own, and the widest selection (128)
# at a temperature where a rejected level owes more residual draws than one
# wave holds (the oracle redraws 50 and 77 of 128 in the paper reading)
WIDTHS = {"k10": (10, 10, 1.0), "k128": (128, 128, 0.2)}


@pytest.mark.parametrize("width", list(WIDTHS))
@pytest.mark.parametrize("mode", list(MODES))
def test_tiny_relaxed_steps_match_oracle(mode, width):
    from paper_2410_05165_amd.binding import Engine
    K, N, tau = WIDTHS[width]
    e = env("tiny", K=K, N=N, temperature=tau)
    w = e["w"]
    key, seed = _key_seed(w)
    eng = Engine(w, e["tw"], e["dw"], e["cat"], mode=MODES[mode], seed=seed)
    dev = torch.device("cuda:0")
    eng.atspeed_prefill(torch.from_numpy(e["pre"]).to(dev))
    o = oracle_user("tiny", 0)
    log = []
    final, steps = sd_decode_relaxed(mode, o["lp"], o["lq"], e["trie"], w.K, w.N, w.gamma, w.L, w.codebook,
                                     w.temperature, key, 0, log)
    acc = torch.zeros(1, dtype=torch.int32, device=dev)
    ta = torch.zeros(1, dtype=torch.int32, device=dev)
    for i, (t0, D, res) in enumerate(steps):
        t, nb, paths, sc = eng.atspeed_get_state(1)
        assert t[0] == t0
        eng.atspeed_draft()
        eng.atspeed_verify(acc, ta)
        t, nb, paths, sc = eng.atspeed_get_state(1)
        got = [tuple(int(c) for c in paths[0, k, :t[0]]) for k in range(nb[0])]
        want = [p for p, _ in res.beams]
        print(f"[{mode} {width}] step {i}: t {t0}->{t[0]} accepted {int(acc[0])} (oracle {res.t_after}, {res.accepted}), "
              f"{len(got)} beams")
        assert int(ta[0]) == res.t_after and int(acc[0]) == res.accepted
        assert got == want
        np.testing.assert_allclose(sc[0, :nb[0]], [s for _, s in res.beams], rtol=0, atol=1e-4)
    eng.close()


def test_relaxed_exact_output_law():
    from paper_2410_05165_amd.binding import Engine
    base = get_workload("tiny")
    B, runs = 512, 4
    w = base.with_(batch=B, K=1, N=1, name="tiny_law")
    cat = make_catalog(w)
    pre1 = make_prefixes(base, cat)[0]
    pre = np.broadcast_to(pre1, (B, pre1.size)).copy()
    tw, dw = make_weights(w, "target"), make_weights(w, "draft")
    tgt, dft = Decoder(w.target, tw, w.dtype), Decoder(w.draft, dw, w.dtype)
    kids = Trie(cat).children(())
    lp = item_log_softmax(tgt.prefill(pre1).last_logits)[kids]
    lq = item_log_softmax(dft.prefill(pre1).last_logits)[kids]
    p = np.exp(lp - lp.max()); p /= p.sum()
    q = np.exp(lq - lq.max()); q /= q.sum()
    first = []
    dev = torch.device("cuda:0")
    prefix = torch.from_numpy(pre).to(dev)
    for r in range(runs):
        eng = Engine(w, tw, dw, cat, mode=1, seed=1000 + r)
        items = torch.zeros((B, 1, w.L), dtype=torch.int32, device=dev)
        scores = torch.zeros((B, 1), dtype=torch.float32, device=dev)
        n = torch.zeros(B, dtype=torch.int32, device=dev)
        eng.atspeed_decode_topk(prefix, items, scores, n)
        first.extend(items[:, 0, 0].cpu().numpy().tolist())
        eng.close()
    idx = {c: i for i, c in enumerate(kids)}
    counts = np.bincount([idx[c] for c in first], minlength=len(kids)).astype(float)
    # 16 bins of about equal target mass
    order = np.argsort(-p)
    edges = np.searchsorted(np.cumsum(p[order]), np.linspace(0, 1, 17)[1:-1])
    bins = np.split(order, edges)
    obs = np.array([counts[b].sum() for b in bins])
    exp_p = np.array([p[b].sum() for b in bins]) * len(first)
    exp_q = np.array([q[b].sum() for b in bins]) * len(first)
    chi_p = float(((obs - exp_p) ** 2 / exp_p).sum())
    chi_q = float(((obs - exp_q) ** 2 / np.maximum(exp_q, 1e-9)).sum())
    print(f"[law] {len(first)} samples: chi2 vs pi_p = {chi_p:.1f}, vs pi_q = {chi_q:.1f} (15 dof, 1e-3 critical 37.70)")
    assert chi_p < 37.70
    assert chi_q > 37.70


@pytest.mark.parametrize("mode", list(MODES))
def test_identical_draft_accepts_every_level(mode):
    """q = p (the draft is the target): every slot / draft is accepted, one step decodes the items
    (PAPER mode with N = K, so that both distributions share their candidate sets)."""
    from paper_2410_05165_amd.binding import Engine
    base = get_workload("tiny")
    w = base.with_(draft=base.target, N=base.K, name="tiny_same")
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    tw = make_weights(w, "target")
    eng = Engine(w, tw, tw, cat, mode=MODES[mode], seed=7)
    dev = torch.device("cuda:0")
    eng.atspeed_prefill(torch.from_numpy(pre).to(dev))
    acc = torch.zeros(1, dtype=torch.int32, device=dev)
    ta = torch.zeros(1, dtype=torch.int32, device=dev)
    eng.atspeed_draft()
    eng.atspeed_verify(acc, ta)
    print(f"[{mode} q=p] accepted {int(acc[0])}, t_after {int(ta[0])}")
    assert int(acc[0]) == w.L and int(ta[0]) == w.L
    eng.close()
