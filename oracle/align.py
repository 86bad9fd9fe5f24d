"""Draft alignment objectives of AtSpeed (Sec. 3.1 and 3.2), fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Per training context c = (x, y_<t) -- a user's prefix followed by the first t-1
codes of a sequence y -- the draft's token distribution q(.|c) and the target's
p(.|c) are softmaxes over the item-token columns (the normaliser of the pinned
reading), and V_c = ConstrainedTopK(q) is the set of the K trie-valid codes of
level t with the largest q (ties: smaller code first).

AtSpeed-S, per context (the bracket of the Align-S loss of Sec. 3.1): the
reverse KL over V_c minus the density regulariser,
    sum_{v in V_c} q(v) log(q(v)/p(v)) - sum_{v in V_c} q(v) log(q(v)/p_K),
where p_K = p(y_{K,t} | y_{K,<t}) is the target's probability of the t-th code
of the K-th sequence of the context's user given that sequence's own prefix.
The q log q terms cancel, leaving sum_{v in V_c} q(v) (log p_K - log p(v)).

AtSpeed-R, per context (Sec. 3.2): TVD(p', q') = 1/2 sum_{v in V_c} |p'(v) - q'(v)|
with p', q' the distributions p, q truncated to V_c and renormalised.  The
paper's "top-K valid tokens" is read as the same V_c as AtSpeed-S.

Aggregation: L = (1 / |D'|) sum_{(x, Y) in D'} sum_{y in Y} (1/|y|) sum_t l(c_t).
A context shared by several sequences of Y (a common prefix) counts once per
sequence through it.  D' holds, per user, the target's top-K sequences
(AtSpeed-R) or the top-K of beam search under the mixture (1-lambda) q + lambda p
of the two models' token distributions (AtSpeed-S; lambda = 1 gives the target's
top-K): the last beam-search step's sequences by default, or those of every step
(the multi-step data the paper compares against; sequences of length 1..L, the
K-th full-length sequence last, which fixes p_K).

Overall objective (Eq. 5 and its AtSpeed-R counterpart): alpha L_Align +
(1 - alpha) L_Rec.  L_Rec, the recommender's own loss (the NLL of the next
item's tokens), may be substituted by the recommender's loss of choice; the
synthetic histories have no ground-truth next item, so its labels are the
training sequences themselves:
    L_Rec = (1 / |D'|) sum sum_{y in Y} (1/|y|) sum_t -log q(y_t | c_t),
i.e. per context c with weight w_c and label distribution pi_c (the sequences'
next codes, each counted with 1/|y|, normalised): -sum_v pi_c(v) log q(v), with
gradient q - pi_c.

Gradients with respect to the draft's item logits z (q = softmax(z)), V_c held
fixed (the selection is piecewise constant in z):
    S: dl/dz_j = q_j (a_j [j in V_c] - sum_{v in V_c} q_v a_v),  a_v = log p_K - log p(v)
    R: dl/dz_j = [j in V_c] q'_j (s_j - sum_{v in V_c} s_v q'_v) / 2,  s_v = sign(q'_v - p'_v)
Training the draft's item-head rows W (z = W h for the normed final hidden h of
the context) then has dL/dW = sum_c w_c (dl/dz)(c) h(c)^T.

D' for AtSpeed-S with lambda < 1 (Sec. 3.1): the top-K sequences of constrained
beam search (width K, every level's beams kept for multi-step data) under the
token-level mixture m(c | s) = (1 - lambda) q(c | s) + lambda p(c | s) of the two
models' item distributions, a sequence scored by sum_t log m(y_t | y_<t); ties
by the lexicographically smaller sequence, as in every other search here.

The optimizer is AdamW (the paper's implementation details) with decoupled
weight decay: w <- w - lr wd w - lr m_hat / (sqrt(v_hat) + eps), m_hat and v_hat
the bias-corrected first and second moments.

Parity: pinned in tests/test_oracle_align.py -- the mixture search against
the target's and the draft's own beam search at lambda = 1 and 0, against
brute-force enumeration of a small catalog and against a hand-worked table
(tests/golden/mixture_example.json); the gradients against central
finite differences of the losses, a hand-worked context for each loss
(tests/golden/align_example.json), the regulariser's sign (negative when every
code of V_c is more probable under the target than the K-th sequence's code,
positive when every one is less), TVD's range and its Eq. 6 identity
(1 - TVD = sum of minima), the dataset weights and label distributions against
hand counts, the recommendation loss against torch's cross-entropy with class
probabilities and the aggregate at alpha = 0 against the per-sequence NLL summed
token by token, and AdamW
against torch.optim.AdamW (fp64, CPU) over several steps and against its
first-step closed form (a step of lr times the gradient's sign without decay).
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .search import Decision, top_boundary

Path = Tuple[int, ...]


def softmax(z: np.ndarray) -> np.ndarray:
    e = np.exp(z - np.max(z))
    return e / e.sum()


def constrained_topk(lq: np.ndarray, cols: Sequence[int], K: int) -> List[int]:
    """The K columns of ``cols`` with the largest draft log-prob (ties: smaller column)."""
    return sorted(cols, key=lambda c: (-lq[c], c))[:K]


def align_s(lq: np.ndarray, lp: np.ndarray, cols: Sequence[int], K: int, log_pK: float):
    """AtSpeed-S loss of one context and its gradient with respect to the draft's logits.

    lq, lp: log-probabilities over the item columns (draft, target); cols: the
    trie-valid columns of the level; log_pK: log p(y_{K,t} | y_{K,<t}).
    """
    q = np.exp(lq)
    vc = constrained_topk(lq, cols, K)
    a = {v: log_pK - lp[v] for v in vc}
    loss = sum(q[v] * a[v] for v in vc)
    grad = -q * loss
    for v in vc:
        grad[v] += q[v] * a[v]
    return float(loss), grad, vc


def align_r(lq: np.ndarray, lp: np.ndarray, cols: Sequence[int], K: int):
    """AtSpeed-R loss (TVD over V_c) of one context and its gradient."""
    vc = constrained_topk(lq, cols, K)
    qv = np.exp(np.array([lq[v] for v in vc]))
    pv = np.exp(np.array([lp[v] for v in vc]))
    qn, pn = qv / qv.sum(), pv / pv.sum()
    loss = 0.5 * float(np.abs(pn - qn).sum())
    s = np.sign(qn - pn)
    g = 0.5 * qn * (s - float((s * qn).sum()))
    grad = np.zeros_like(lq)
    for i, v in enumerate(vc):
        grad[v] = g[i]
    return loss, grad, vc


def rec_loss(lq: np.ndarray, pi: Dict[int, float]):
    """Recommendation (NLL) loss of one context with label distribution ``pi``
    (column -> probability) and its gradient with respect to the draft's logits."""
    q = np.exp(lq)
    loss = -sum(w * lq[c] for c, w in pi.items())
    grad = q * sum(pi.values())
    for c, w in pi.items():
        grad[c] -= w
    return float(loss), grad


def label_distributions(Y: Sequence[Path], codebook: int) -> Dict[Path, Dict[int, float]]:
    """Per context of one user: the next codes of the sequences through it, each
    counted with 1/|y|, as a distribution over item columns."""
    acc: Dict[Path, Dict[int, float]] = {}
    for y in Y:
        for t in range(len(y)):
            d = acc.setdefault(tuple(y[:t]), {})
            col = codebook * t + y[t]
            d[col] = d.get(col, 0.0) + 1.0 / len(y)
    return {c: {k: v / sum(d.values()) for k, v in d.items()} for c, d in acc.items()}


def context_weights(Y: Sequence[Sequence[Path]], L: int) -> List[Dict[Path, float]]:
    """Per user, the weight of every context (a prefix of length 0..L-1) in the
    aggregated loss: (sequences of Y through it) / (|y| x number of users)."""
    B = len(Y)
    out = []
    for seqs in Y:
        w: Dict[Path, float] = {}
        for y in seqs:
            for t in range(len(y)):
                w[tuple(y[:t])] = w.get(tuple(y[:t]), 0.0) + 1.0 / (len(y) * B)
        out.append(w)
    return out


def log_pK_of(Y: Sequence[Path], lp_of, codebook: int) -> List[float]:
    """log p(y_{K,t} | y_{K,<t}) for t = 1..L of the K-th (last) sequence of one user's Y."""
    yk = Y[-1]
    return [float(lp_of(tuple(yk[:t]))[codebook * t + yk[t]]) for t in range(len(yk))]


def aligned_loss(mode: str, lq_of, lp_of, trie, Y: Sequence[Sequence[Path]], K: int, L: int, codebook: int,
                 alpha: float = 1.0):
    """Aggregated loss alpha L_Align + (1 - alpha) L_Rec over all users and the
    gradient of every context.

    lq_of / lp_of(u, path) -> item log-probs of the draft / target at that
    context of user u.  Returns (loss, {(u, path): (weight, grad)}), grad the
    per-context gradient alpha dl/dz + (1 - alpha)(q - pi).
    """
    W = context_weights(Y, L)
    total, grads = 0.0, {}
    for u, wu in enumerate(W):
        if len(Y[u][-1]) != L:
            raise ValueError("the K-th (last) sequence of a user must be a whole item")
        lpk = log_pK_of(Y[u], lambda p: lp_of(u, p), codebook)
        pis = label_distributions(Y[u], codebook)
        for path, w in wu.items():
            t = len(path)
            cols = [codebook * t + c for c in trie.children(path)]
            lq, lp = lq_of(u, path), lp_of(u, path)
            if mode == "S":
                l, g, _ = align_s(lq, lp, cols, K, lpk[t])
            else:
                l, g, _ = align_r(lq, lp, cols, K)
            lr, gr = rec_loss(lq, pis[path])
            total += w * (alpha * l + (1.0 - alpha) * lr)
            grads[(u, path)] = (w, alpha * g + (1.0 - alpha) * gr)
    return total, grads


def head_gradient(grads: Dict, hidden: Dict) -> np.ndarray:
    """dL/dW for the item head: sum over contexts of w * grad ⊗ h (hidden: (u, path) -> h)."""
    keys = list(grads)
    G = np.stack([grads[k][0] * grads[k][1] for k in keys])      # [C, n_item]
    Hm = np.stack([np.asarray(hidden[k], dtype=np.float64) for k in keys])   # [C, d]
    return G.T @ Hm


def adamw_step(w: np.ndarray, m: np.ndarray, v: np.ndarray, g: np.ndarray, step: int, lr: float,
               beta1: float, beta2: float, eps: float, weight_decay: float):
    """One AdamW step (1-based ``step``); returns the new (w, m, v)."""
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** step)
    v_hat = v / (1.0 - beta2 ** step)
    w = w - lr * weight_decay * w
    w = w - lr * m_hat / (np.sqrt(v_hat) + eps)
    return w, m, v


def mixed_log(lq: np.ndarray, lp: np.ndarray, lam: float) -> np.ndarray:
    """log((1 - lam) q + lam p) of two log-probability rows (lam 0 and 1 return a row unchanged)."""
    if lam == 1.0:
        return np.asarray(lp, dtype=np.float64)
    if lam == 0.0:
        return np.asarray(lq, dtype=np.float64)
    mx = np.maximum(lq, lp)
    return mx + np.log((1.0 - lam) * np.exp(lq - mx) + lam * np.exp(lp - mx))


def mixture_beam_search(lp_of, lq_of, trie, K: int, L: int, codebook: int, lam: float,
                        log: Optional[List[Decision]] = None):
    """Constrained beam search of width K under the mixture (1 - lam) q + lam p;
    lp_of / lq_of(path) -> item log-probs of the target / draft at that context.
    Returns the beams (path, mixed score) of every level 1..L."""
    beams = [((), 0.0)]
    levels = []
    for lvl in range(1, L + 1):
        cands = []
        for path, score in beams:
            row = mixed_log(lq_of(path), lp_of(path), lam)
            for c in trie.children(path):
                cands.append((path + (c,), score + float(row[codebook * (lvl - 1) + c])))
        beams, margin, pair = top_boundary(cands, K)
        if log is not None:
            log.append(Decision("mixture_topk", lvl, margin, pair))
        levels.append(beams)
    return levels
