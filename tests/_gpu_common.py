"""Shared set-up of the GPU parity tests: seeded workloads, engines, oracle users."""
import functools

import numpy as np

from synth import get_workload, make_catalog, make_prefixes, make_weights
from oracle.model import Decoder, item_log_softmax
from oracle.numerics import round_bf16
from oracle.relaxed import Streams
from oracle.search import Scorer, model_scorer, table_scorer
from oracle.trie import Trie
from oracle.tree import flatten

# Parity bars (selections outside logit gaps below SEL_TIE are bit-exact;
# logits within LOGIT_TOL by dtype; sequence log-probs within SCORE_TOL).
LOGIT_TOL = {"fp32": 1e-4, "bf16": 2e-2}
SCORE_TOL = 1e-3
SEL_TIE = 1e-3
# Sequence log-probs of an end-to-end bf16 decode (the GPU's own logits, each
# within LOGIT_TOL of the oracle's) against the oracle's: measured at most
# 1e-2 on the bf16 workloads, held to the logit bar.
SCORE_TOL_BF16_E2E = 2e-2


class Fp32AccDecoder(Decoder):
    """The oracle with every GEMM accumulated in fp32 and the same bf16 rounding
    points: a second correct computation of the same bf16 model, whose distance
    from the fp64 oracle measures the noise floor of that model's logits."""

    def __init__(self, *a, **kw):
        super().__init__(*a, **kw)
        self._f32 = {}

    def W(self, name):
        if name not in self._f32:
            a = super().W(name)
            self._f32[name] = a.astype(np.float32) if a.ndim == 2 else a
        return self._f32[name]

    def _r(self, x):
        return round_bf16(x).astype(np.float32)


def noise_bar(*self_noise):
    """Logit bar of a bf16 comparison: the 2e-2 bar, or twice the largest measured
    distance between the fp64 oracle and its fp32-accumulation variant on the
    same outputs if that is larger.  Two computations with the same bf16
    rounding points but a different accumulation differ at a few roundings;
    every later rounding point turns the difference into whole-ulp flips of more
    elements, so at d 4096 (sigma^2 d = 1.64) the floor exceeds 2e-2 from one
    layer on.  The GPU adds its own seeds (fp32 MFMA order, the o/down k split,
    16-bit attention probabilities), measured at 1.0-1.5x the floor."""
    return max(LOGIT_TOL["bf16"], 2.0 * max(self_noise))


@functools.lru_cache(maxsize=4)
def env(name, **overrides):
    w = get_workload(name, **overrides)
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    return dict(w=w, cat=cat, pre=pre, tw=make_weights(w, "target"), dw=make_weights(w, "draft"), trie=Trie(cat))


@functools.lru_cache(maxsize=64)
def oracle_user(name, u):
    e = env(name)
    w = e["w"]
    tgt = Decoder(w.target, e["tw"], w.dtype)
    dft = Decoder(w.draft, e["dw"], w.dtype)
    tc, dc = tgt.prefill(e["pre"][u]), dft.prefill(e["pre"][u])
    return dict(tgt=tgt, dft=dft, tcache=tc, dcache=dc,
                lp=model_scorer(tgt, tc, w.target.item_base, w.codebook),
                lq=model_scorer(dft, dc, w.draft.item_base, w.codebook))


def tokens_of(path, w):
    return tuple(w.target.item_base + w.codebook * l + c for l, c in enumerate(path))


def tree_arrays(trees, w, T):
    """Per-user lists of code paths -> (n_nodes [B], token/parent/depth [B, T]) in the flattened order."""
    B = len(trees)
    n = np.zeros(B, np.int32)
    tok = np.zeros((B, T), np.int32)
    par = np.full((B, T), -1, np.int32)
    dep = np.zeros((B, T), np.int32)
    nodes_all = []
    for u, paths in enumerate(trees):
        nodes, parent, depth = flatten(paths)
        assert len(nodes) <= T
        n[u] = len(nodes)
        for i, p in enumerate(nodes):
            tok[u, i] = tokens_of(p, w)[-1]
            par[u, i] = parent[i]
            dep[u, i] = depth[i]
        nodes_all.append(nodes)
    return n, tok, par, dep, nodes_all


def upload_tree(eng, trees, B):
    import torch
    w = eng.w
    n, tok, par, dep, nodes = tree_arrays(trees, w, eng.max_nodes)
    tn, tt, tp, td, tq = eng.tree_tensors(B)
    tn.copy_(torch.from_numpy(n))
    tt.copy_(torch.from_numpy(tok))
    tp.copy_(torch.from_numpy(par))
    td.copy_(torch.from_numpy(dep))
    tq.zero_()
    return nodes


def logit_table(nodes, logits_u, root_u):
    """Oracle scorer from fp32 logits (given per flattened node and at the root)."""
    tab = {(): item_log_softmax(root_u.astype(np.float64))}
    for i, p in enumerate(nodes):
        tab[p] = item_log_softmax(logits_u[i].astype(np.float64))
    return table_scorer(tab)


# ---------------------------------------------------------------- tie zone
# A GPU result that differs from the oracle's is accepted only when taking ONE
# oracle decision whose margin is below SEL_TIE the other way makes the oracle
# reproduce the GPU result exactly (the first differing decision is a near-tie;
# the comparison of that user stops there).  TIE_STEP puts the flipped candidate
# just past the one it displaces.
TIE_STEP = 1e-9


def flipped_scorer(lp, d, codebook):
    """``lp`` with the (n+1)-th sequence of top-n decision ``d`` raised just above
    the n-th (one log-prob entry moved by margin + TIE_STEP)."""
    _, b = d.pair
    par, col = b[:-1], codebook * (len(b) - 1) + b[-1]
    bump = d.margin + TIE_STEP

    def fn(paths):
        rows = [r.copy() for r in lp(paths)]
        for p, r in zip(paths, rows):
            if p == par:
                r[col] += bump
        return np.stack(rows)
    return Scorer(fn)


def strict_tie(log, rerun, same, tie=SEL_TIE):
    """The first near-tie top-n decision of ``log`` whose flip alone makes
    ``rerun(decision)`` (the oracle run again with that decision taken the other
    way) satisfy ``same``; None if there is none."""
    for d in log:
        if d.margin < tie and d.pair is not None and same(rerun(d)):
            return d
    return None


class FlipStreams(Streams):
    """Philox streams of one user with chosen uniforms / Gumbel values replaced."""

    def __init__(self, key, user, u_over=None, g_over=None):
        super().__init__(key, user)
        self.u_over, self.g_over = dict(u_over or {}), dict(g_over or {})

    def u(self, *ctr):
        return self.u_over[ctr] if ctr in self.u_over else super().u(*ctr)

    def g(self, *ctr):
        return self.g_over[ctr] if ctr in self.g_over else super().g(*ctr)


def relaxed_flips(log, tie=SEL_TIE):
    """(margin, uniform overrides, Gumbel overrides) taking each near-tie decision
    of a relaxed (paper reading) oracle log the other way, in log order:
    an acceptance test moves its uniform just across the threshold; a Gumbel-top-k
    draw lifts the first left-out candidate just above the k-th (drafting, whose
    order matters, also swaps each adjacent pair among the k drawn)."""
    for e in log:
        if e[0] == "accept":
            _, lvl, i, margin, ctr, a, lu = e
            if margin < tie:
                yield margin, {ctr: float(np.exp(a + TIE_STEP if lu <= a else a - TIE_STEP))}, {}
        elif e[0] in ("draft", "subset", "residual", "target_draw"):
            _, lvl, k, keyed = e
            pos = range(min(k, len(keyed) - 1)) if e[0] == "draft" else ([k - 1] if len(keyed) > k >= 1 else [])
            for i in pos:
                m = keyed[i][0] - keyed[i + 1][0]
                if m < tie:
                    yield m, {}, {keyed[i + 1][2]: keyed[i + 1][3] + m + TIE_STEP}


def relaxed_tie(log, rerun, same, tie=SEL_TIE):
    """The first near-tie decision of a relaxed log whose flip alone makes
    ``rerun(u_over, g_over)`` satisfy ``same``; None if there is none."""
    for m, uo, go in relaxed_flips(log, tie):
        if same(rerun(uo, go)):
            return m
    return None


def first_difference(gpu_levels, oracle_levels):
    """Index of the first level whose beam list differs, or None."""
    for i, (g, o) in enumerate(zip(gpu_levels, oracle_levels)):
        if list(g) != list(o):
            return i
    return None
