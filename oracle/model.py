"""LLaMA-style causal decoder, fp64 (the oracle's forward pass).

The paper's target and draft are LLaMA-7B and LLaMA-68M (Sec. 4.1,
implementation details); it does not restate the architecture, so the block is
pinned as:

  x = E[token]
  per layer:  h = x + W_o · Attn(RoPE(W_q n(x)), RoPE(W_k n(x)), W_v n(x))
              x = h + W_down · (SiLU(W_gate n(h)) ⊙ W_up n(h))
  logits   = W_item · n(x)                         (item-token rows only)

with n(v) = g ⊙ v / sqrt(mean(v²) + 1e-6), multi-head attention without
biases and scale 1/sqrt(d_head), and rotary embeddings in the rotate-half
pairing (i, i + d_head/2), angle pos · 10000^(-2i/d_head).

Tree semantics (tree-based attention, Sec. 3.3 and its implementation
appendix): the logits at a drafted node equal the causal-LM logits at the last
position of ``prefix ‖ path(node)``, with the path token at depth d placed at
position ``len(prefix) + d - 1``.  The oracle computes them literally, one
causal forward per path (``Decoder.path_logits``); ``Decoder.forward`` also
accepts an explicit attention mask so that the flattened-tree form can be
checked against the per-path form.

Precision (bf16 workloads): weights are bf16; GEMM inputs (normed activations,
attention output, SiLU(g)·u), q/k/v after RoPE and the KV cache are rounded to
bf16 (ties to even); everything else, including the residual stream, softmax
and logits, is fp64.  The fp32 workload rounds nothing.

Parity: pinned by the tests in tests/test_oracle_model.py (closed forms for
zero-weight and zero-query cases, a two-token attention case whose weights
(1/4, 3/4) follow from the 1/sqrt(d_head) scale, through the plain forward and
the prefix-cache branch, rotary embedding as complex rotation, causality and
prefix-cache invariants, hand-computed SwiGLU value).  ``item_log_softmax`` is
pinned in tests/test_oracle_search.py: it sums to one over every item column,
and a hand-worked two-level search (tests/golden/normaliser_example.json) gives
other beams or scores under a per-level normaliser or none.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

from .numerics import round_bf16, to_f64

RMS_EPS = 1e-6
ROPE_BASE = 10000.0


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float = RMS_EPS) -> np.ndarray:
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def rope(x: np.ndarray, pos: np.ndarray, base: float = ROPE_BASE) -> np.ndarray:
    """Rotary embedding on the last axis of ``x`` (d_head), rotate-half pairing.

    ``x``: [..., T, d_head]; ``pos``: [T] absolute positions.
    """
    dh = x.shape[-1]
    half = dh // 2
    inv = base ** (-2.0 * np.arange(half, dtype=np.float64) / dh)
    ang = pos.astype(np.float64)[:, None] * inv[None, :]          # [T, half]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, mask: np.ndarray,
           pk: Optional[np.ndarray] = None, pv: Optional[np.ndarray] = None) -> np.ndarray:
    """Multi-head attention with scale 1/sqrt(d_head): queries ``q`` [S, H, T, dh]
    attend to the prefix keys/values ``pk``/``pv`` [H, P, dh] (if given) and to
    their own sequence's keys ``k``/``v`` [S, H, T, dh] where ``mask`` [T, T]
    allows.  Returns [S, H, T, dh]."""
    dh = q.shape[-1]
    sc = (q @ k.transpose(0, 1, 3, 2)) / np.sqrt(dh)                 # [S, H, T, T]
    sc = np.where(mask[None, None], sc, -np.inf)
    if pk is not None:
        sp = np.einsum("shtd,hpd->shtp", q, pk) / np.sqrt(dh)
        sc = np.concatenate([sp, sc], axis=-1)
    m = np.max(sc, axis=-1, keepdims=True)
    e = np.exp(sc - m)
    pr = e / np.sum(e, axis=-1, keepdims=True)
    if pk is not None:
        P = pk.shape[1]
        return np.einsum("shtp,hpd->shtd", pr[..., :P], pv) + pr[..., P:] @ v
    return pr @ v


class PrefixCache:
    """Per-layer K/V of a user's prefix (after RoPE and rounding), [H, P, dh]."""

    def __init__(self, k: List[np.ndarray], v: List[np.ndarray], last_logits: np.ndarray):
        self.k = k
        self.v = v
        self.last_logits = last_logits   # item logits at the last prefix position (the root)

    @property
    def length(self) -> int:
        return self.k[0].shape[1]


class Decoder:
    """fp64 decoder over weights from ``synth.make_weights``."""

    def __init__(self, dims, weights: Dict[str, np.ndarray], dtype: str, cache_f64: Optional[bool] = None):
        self.dims = dims
        self.w = weights
        self.bf16 = dtype == "bf16"
        nparams = sum(a.size for a in weights.values())
        self._keep = (nparams < 400_000_000) if cache_f64 is None else cache_f64
        self._cache: Dict[str, np.ndarray] = {}

    # -- weights
    def W(self, name: str) -> np.ndarray:
        if name in self._cache:
            return self._cache[name]
        a = to_f64(self.w[name])
        if self._keep:
            self._cache[name] = a
        return a

    def _r(self, x: np.ndarray) -> np.ndarray:
        return round_bf16(x) if self.bf16 else x

    def embed(self, tokens: np.ndarray) -> np.ndarray:
        E = self.w["tok_emb"]
        return to_f64(E[tokens])

    # -- one forward
    def forward(self, tokens: np.ndarray, pos: np.ndarray, prefix: Optional[PrefixCache] = None,
                mask: Optional[np.ndarray] = None, keep_kv: bool = False):
        """Run the decoder on ``tokens`` [S, T] at positions ``pos`` [T].

        Every sequence attends to all keys of ``prefix`` (if given) and, within
        itself, to the keys allowed by ``mask`` [T, T] (default: causal).
        Returns (item logits [S, T, n_item], per-layer (k, v) if keep_kv).
        """
        T = tokens.shape[1]
        if mask is None:
            mask = np.tril(np.ones((T, T), dtype=bool))
        x = self.embed(tokens)                                          # [S, T, d]
        kvs = []
        for l in range(self.dims.n_layers):
            _, x, k, v = self.block(l, x, pos, prefix.k[l] if prefix is not None else None,
                                    prefix.v[l] if prefix is not None else None, mask)
            if keep_kv:
                kvs.append((k, v))
        return self.head(x), kvs

    def head(self, x: np.ndarray) -> np.ndarray:
        """Item logits of residual-stream rows: final RMSNorm, then the item rows of the output head."""
        return self._r(self.norm(-1, "", x)) @ self.W("lm_head_item").T

    def block(self, l: int, x: np.ndarray, pos: np.ndarray, pk: Optional[np.ndarray] = None,
              pv: Optional[np.ndarray] = None, mask: Optional[np.ndarray] = None):
        """Decoder block ``l`` on the residual stream ``x`` [S, T, d] at positions
        ``pos`` [T]: every sequence attends to the prefix keys ``pk``/``pv``
        [H, P, dh] (if given) and, within itself, to the keys ``mask`` [T, T]
        allows (default: causal).  Returns (h, x_out, k, v): the residual after
        the attention sublayer, after the FFN sublayer, and this block's k, v
        [S, H, T, dh] after RoPE and rounding."""
        S, T = x.shape[0], x.shape[1]
        if mask is None:
            mask = np.tril(np.ones((T, T), dtype=bool))
        p = f"l{l}."
        hn = self._r(self.norm(l, "attn_norm", x))
        q, k, v = (self._r(a) for a in self.qkv(l, hn, pos))
        o = self._r(self.merge_heads(attend(q, k, v, mask, pk, pv)))
        h = x + o @ self.W(p + "wo").T
        h2 = self._r(self.norm(l, "ffn_norm", h))
        a = self._r(self.swiglu(l, h2))
        return h, h + a @ self.W(p + "w_down").T, k, v

    # -- the steps of a block (unrounded results; the block rounds them where
    #    the bf16 model does)
    def norm(self, l: int, which: str, x: np.ndarray) -> np.ndarray:
        """RMSNorm of layer ``l`` (``which``: attn_norm or ffn_norm; l < 0: the final norm)."""
        return rmsnorm(x, self.W("final_norm" if l < 0 else f"l{l}.{which}"))

    def qkv(self, l: int, hn: np.ndarray, pos: np.ndarray):
        """q, k (after RoPE) and v [S, H, T, dh] of the normalised rows ``hn`` [S, T, d]."""
        d = self.dims
        S, T = hn.shape[0], hn.shape[1]
        H, dh = d.n_heads, d.d_head
        p = f"l{l}."
        q = (hn @ self.W(p + "wq").T).reshape(S, T, H, dh).transpose(0, 2, 1, 3)
        k = (hn @ self.W(p + "wk").T).reshape(S, T, H, dh).transpose(0, 2, 1, 3)
        v = (hn @ self.W(p + "wv").T).reshape(S, T, H, dh).transpose(0, 2, 1, 3)
        return rope(q, pos), rope(k, pos), v

    def merge_heads(self, o: np.ndarray) -> np.ndarray:
        """[S, H, T, dh] -> [S, T, d]."""
        S, H, T, dh = o.shape
        return o.transpose(0, 2, 1, 3).reshape(S, T, H * dh)

    def swiglu(self, l: int, h2: np.ndarray) -> np.ndarray:
        """SiLU(W_gate h2) * (W_up h2) of layer ``l``."""
        p = f"l{l}."
        return silu(h2 @ self.W(p + "w_gate").T) * (h2 @ self.W(p + "w_up").T)

    # -- prefix and paths
    def prefill(self, prefix_tokens: np.ndarray) -> PrefixCache:
        """Causal forward over one user's prefix; keeps its K/V and the root logits."""
        P = prefix_tokens.shape[0]
        logits, kvs = self.forward(prefix_tokens[None, :], np.arange(P), keep_kv=True)
        return PrefixCache([k[0] for k, _ in kvs], [v[0] for _, v in kvs], logits[0, -1])

    def path_logits(self, cache: PrefixCache, paths: Sequence[Sequence[int]]) -> np.ndarray:
        """Item logits at the last token of ``prefix ‖ path`` for each path (token ids).

        Paths of equal length are evaluated together; each is its own causal
        sequence after the shared prefix.  The empty path returns the root logits.
        """
        out = np.empty((len(paths), self.w["lm_head_item"].shape[0]), dtype=np.float64)
        by_len: Dict[int, List[int]] = {}
        for i, pth in enumerate(paths):
            by_len.setdefault(len(pth), []).append(i)
        P = cache.length
        for T, idx in by_len.items():
            if T == 0:
                out[idx] = cache.last_logits
                continue
            toks = np.asarray([list(paths[i]) for i in idx], dtype=np.int64)
            for s in range(0, len(idx), 256):
                lg, _ = self.forward(toks[s:s + 256], P + np.arange(T), prefix=cache)
                out[idx[s:s + 256]] = lg[:, -1]
        return out


def item_log_softmax(logits: np.ndarray) -> np.ndarray:
    """Log-softmax over the item-token columns (the normaliser of the pinned reading)."""
    m = np.max(logits, axis=-1, keepdims=True)
    return logits - (m + np.log(np.sum(np.exp(logits - m), axis=-1, keepdims=True)))
