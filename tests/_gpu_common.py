"""Shared set-up of the GPU parity tests: seeded workloads, engines, oracle users."""
import functools

import numpy as np

from synth import get_workload, make_catalog, make_prefixes, make_weights
from oracle.model import Decoder, item_log_softmax
from oracle.search import model_scorer, table_scorer
from oracle.trie import Trie
from oracle.tree import flatten

# Parity bars (selections outside logit gaps below SEL_TIE are bit-exact;
# logits within LOGIT_TOL by dtype; sequence log-probs within SCORE_TOL).
LOGIT_TOL = {"fp32": 1e-4, "bf16": 2e-2}
SCORE_TOL = 1e-3
SEL_TIE = 1e-3


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


def first_difference(gpu_levels, oracle_levels):
    """Index of the first level whose beam list differs, or None."""
    for i, (g, o) in enumerate(zip(gpu_levels, oracle_levels)):
        if list(g) != list(o):
            return i
    return None
