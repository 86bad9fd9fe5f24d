"""Seeded input generators (catalog, histories, prompt, weights).

The paper's datasets (Amazon Beauty/Games, MovieLens-1M, Goodreads; Sec. 4.1
and the dataset-statistics table) and its trained LC-Rec / LLaMA weights are
not available, so every input here is synthetic and seeded:

* items are fixed-length identifiers of L = 4 codebook tokens (task formulation,
  footnote on codebook identifiers; L = 4 in the implementation details);
  a catalog is a set of distinct random L-tuples of codes;
* a user history is a list of catalog items, drawn uniformly or from a
  truncated Zipf(1.1) law over a random popularity ranking; the prefix is an
  optional shared text prompt followed by the item tokens of the history;
* all weight matrices are N(0, 0.02) draws (rounded to bf16 with
  round-to-nearest-even for the bf16 workloads); norm gains are 1.

Token ids: an item code ``c`` at item level ``l`` (0-based) is token
``item_base + codebook * l + c``.  Text tokens are ``[0, item_base)``.

Nothing in this module computes any part of the method.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os
from typing import Dict, List, Optional

import numpy as np

# Order in which independent streams are spawned from the workload seed.
STREAMS = ("catalog", "popularity", "histories", "prompt", "target_w", "draft_w", "philox")


@dataclasses.dataclass(frozen=True)
class ModelDims:
    n_layers: int
    d_model: int
    n_heads: int
    d_ffn: int
    vocab: int        # full vocabulary (text + item tokens)
    item_base: int    # first item-token id

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_heads


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    dtype: str                 # "fp32" or "bf16"
    target: ModelDims
    draft: ModelDims
    n_items: int
    batch: int
    hist_items: int
    prompt_len: int
    hist_dist: str             # "uniform" or "zipf"
    K: int
    N: int
    gamma: int
    mode: str = "strict"       # "strict", "relaxed_exact", "relaxed_paper"
    temperature: float = 1.0
    L: int = 4
    codebook: int = 256
    zipf_s: float = 1.1
    seed: int = 0

    @property
    def prefix_len(self) -> int:
        return self.prompt_len + self.L * self.hist_items

    @property
    def n_item_tokens(self) -> int:
        return self.L * self.codebook

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _dims(n_layers, d_model, n_heads, d_ffn, vocab, item_base):
    return ModelDims(n_layers, d_model, n_heads, d_ffn, vocab, item_base)


_T7B = _dims(32, 4096, 32, 11008, 33024, 32000)
_D7B = _dims(4, 768, 12, 3072, 33024, 32000)

WORKLOADS: Dict[str, Workload] = {
    # 2-layer fp32 target, 1-layer draft, 2,000 items, one user, 20 uniform items.
    "tiny": Workload("tiny", "fp32", _dims(2, 128, 4, 512, 1024, 0), _dims(1, 64, 2, 256, 1024, 0),
                     n_items=2000, batch=1, hist_items=20, prompt_len=0, hist_dist="uniform",
                     K=10, N=10, gamma=4),
    # 8-layer bf16 target, 2-layer draft, 20,000 items, 16 users with 30 Zipf items.
    "small": Workload("small", "bf16", _dims(8, 1024, 16, 2816, 1024, 0), _dims(2, 256, 4, 1024, 1024, 0),
                      n_items=20000, batch=16, hist_items=30, prompt_len=0, hist_dist="zipf",
                      K=20, N=40, gamma=4),
    # LLaMA-7B-shaped target, 4-layer draft, 100,000 items, 32 users, 64-token prompt + 20 Zipf items.
    "b7": Workload("b7", "bf16", _T7B, _D7B, n_items=100_000, batch=32, hist_items=20, prompt_len=64,
                   hist_dist="zipf", K=10, N=20, gamma=4),
    # Same model and batch, relaxed sampling verification, K=20, N=40.
    "b7_relaxed": Workload("b7_relaxed", "bf16", _T7B, _D7B, n_items=100_000, batch=32, hist_items=20,
                           prompt_len=64, hist_dist="zipf", K=20, N=40, gamma=4, mode="relaxed_paper"),
    # Stress: 1M items, 128 users with 1,024-token prefixes, K=50, N=100.
    "stress": Workload("stress", "bf16", _T7B, _D7B, n_items=1_000_000, batch=128, hist_items=240,
                       prompt_len=64, hist_dist="zipf", K=50, N=100, gamma=4),
}


def get_workload(name: str, **overrides) -> Workload:
    w = WORKLOADS[name]
    return w.with_(**overrides) if overrides else w


def seed_streams(seed: int) -> Dict[str, np.random.SeedSequence]:
    ss = np.random.SeedSequence(seed).spawn(len(STREAMS))
    return dict(zip(STREAMS, ss))


def item_token(item_base: int, codebook: int, level: int, code):
    """Token id of ``code`` at item level ``level`` (0-based)."""
    return item_base + codebook * level + code


def make_catalog(w: Workload) -> np.ndarray:
    """``[n_items, L]`` int32 distinct random code tuples, in draw order."""
    rng = np.random.default_rng(seed_streams(w.seed)["catalog"])
    space = w.codebook ** w.L
    if w.n_items > space:
        raise ValueError("catalog larger than the code space")
    keys: List[np.ndarray] = []
    seen = np.empty(0, dtype=np.int64)
    need = w.n_items
    while need > 0:
        draw = rng.integers(0, space, size=max(2 * need, 64), dtype=np.int64)
        # keep first occurrences, in draw order, that are not already taken
        _, first = np.unique(draw, return_index=True)
        draw = draw[np.sort(first)]
        draw = draw[~np.isin(draw, seen)]
        draw = draw[:need]
        keys.append(draw)
        seen = np.concatenate([seen, draw])
        need -= draw.size
    key = np.concatenate(keys)
    codes = np.empty((w.n_items, w.L), dtype=np.int32)
    for l in range(w.L - 1, -1, -1):
        codes[:, l] = key % w.codebook
        key = key // w.codebook
    return codes


def make_histories(w: Workload, n_catalog: int) -> np.ndarray:
    """``[batch, hist_items]`` catalog indices of each user's history."""
    st = seed_streams(w.seed)
    rng_h = np.random.default_rng(st["histories"])
    if w.hist_dist == "uniform":
        return rng_h.integers(0, n_catalog, size=(w.batch, w.hist_items)).astype(np.int64)
    if w.hist_dist != "zipf":
        raise ValueError(w.hist_dist)
    ranking = np.random.default_rng(st["popularity"]).permutation(n_catalog)
    ranks = np.arange(1, n_catalog + 1, dtype=np.float64)
    pmf = ranks ** (-w.zipf_s)
    cdf = np.cumsum(pmf)
    cdf /= cdf[-1]
    u = rng_h.random(size=(w.batch, w.hist_items))
    r = np.minimum(np.searchsorted(cdf, u, side="right"), n_catalog - 1)
    return ranking[r].astype(np.int64)


def make_prompt(w: Workload) -> np.ndarray:
    rng = np.random.default_rng(seed_streams(w.seed)["prompt"])
    if w.prompt_len == 0:
        return np.zeros(0, dtype=np.int32)
    return rng.integers(0, w.target.item_base, size=w.prompt_len).astype(np.int32)


def make_prefixes(w: Workload, catalog: Optional[np.ndarray] = None) -> np.ndarray:
    """``[batch, prefix_len]`` int32 token ids: shared prompt, then history item tokens."""
    if catalog is None:
        catalog = make_catalog(w)
    hist = make_histories(w, catalog.shape[0])
    prompt = make_prompt(w)
    lvl = np.arange(w.L, dtype=np.int32)
    toks = item_token(w.target.item_base, w.codebook, lvl[None, None, :], catalog[hist])  # [B, H, L]
    toks = toks.reshape(w.batch, w.hist_items * w.L).astype(np.int32)
    out = np.concatenate([np.broadcast_to(prompt, (w.batch, prompt.size)), toks], axis=1)
    return np.ascontiguousarray(out, dtype=np.int32)


def philox_key(w: Workload) -> np.ndarray:
    """Two 32-bit words keying the counter-based generator of the relaxed modes."""
    return seed_streams(w.seed)["philox"].generate_state(2, dtype=np.uint32)


# ---------------------------------------------------------------- weights

def _bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit pattern (uint16), round to nearest even (storage format of the draws)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    t = (u >> np.uint32(16)) & np.uint32(1)
    t += u
    t += np.uint32(0x7FFF)
    t >>= np.uint32(16)
    return t.astype(np.uint16)


LAYER_MATS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def weight_shapes(m: ModelDims, n_item_tokens: int) -> Dict[str, tuple]:
    d, f = m.d_model, m.d_ffn
    s = {"tok_emb": (m.vocab, d)}
    for l in range(m.n_layers):
        s.update({f"l{l}.wq": (d, d), f"l{l}.wk": (d, d), f"l{l}.wv": (d, d), f"l{l}.wo": (d, d),
                  f"l{l}.w_gate": (f, d), f"l{l}.w_up": (f, d), f"l{l}.w_down": (d, f)})
    s["lm_head_item"] = (n_item_tokens, d)
    return s


def make_weights(w: Workload, which: str = "target", threads: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Random-init weights of the target or the draft.

    Matrices are ``[out, in]`` (row ``o`` holds the weights of output ``o``).
    ``lm_head_item`` holds only the rows of the item tokens (the text-token rows
    of the output head are never read on this path).  Norm gains are ones
    (``l{i}.attn_norm``, ``l{i}.ffn_norm``, ``final_norm``).  For bf16 workloads
    the matrices are uint16 bf16 bit patterns, else float32.
    """
    m = w.target if which == "target" else w.draft
    shapes = weight_shapes(m, w.n_item_tokens)
    names = list(shapes)
    root = seed_streams(w.seed)["target_w" if which == "target" else "draft_w"]
    child = dict(zip(names, root.spawn(len(names))))

    def draw(name):
        x = np.random.default_rng(child[name]).standard_normal(shapes[name], dtype=np.float32)
        x *= np.float32(0.02)
        return name, (_bf16_bits(x) if w.dtype == "bf16" else x)

    nthreads = threads or min(16, os.cpu_count() or 1)
    out: Dict[str, np.ndarray] = {}
    with _cf.ThreadPoolExecutor(nthreads) as ex:
        for name, arr in ex.map(draw, names):
            out[name] = arr
    ones = np.ones(m.d_model, dtype=np.float32)
    for l in range(m.n_layers):
        out[f"l{l}.attn_norm"] = ones
        out[f"l{l}.ffn_norm"] = ones
    out["final_norm"] = ones
    return out
