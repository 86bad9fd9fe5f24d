"""Pins for the oracle decoder (CPU): closed forms, invariants, the tree example."""
import json
import math
import os

import numpy as np
import pytest

from synth import ModelDims, Workload, make_weights
from oracle.model import Decoder, rope, RMS_EPS
from oracle.tree import ancestor_mask, flatten

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _tiny_workload(**kw):
    base = dict(name="t", dtype="fp32",
                target=ModelDims(2, 32, 4, 64, 4 * 6 + 10, 10),
                draft=ModelDims(1, 16, 2, 32, 4 * 6 + 10, 10),
                n_items=200, batch=1, hist_items=3, prompt_len=2, hist_dist="uniform",
                K=3, N=4, gamma=4, codebook=6)
    base.update(kw)
    return Workload(**base)


def _zeros_like_weights(w):
    return {k: (np.zeros_like(v) if k.startswith("l") and not k.endswith("norm") else v.copy())
            for k, v in w.items()}


def _rms(x):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + RMS_EPS)


def test_zero_blocks_reduce_to_embedding_readout():
    w = _tiny_workload()
    W = _zeros_like_weights(make_weights(w, "target"))
    dec = Decoder(w.target, W, "fp32")
    toks = np.array([[3, 17, 25, 11]])
    logits, _ = dec.forward(toks, np.arange(4))
    E = W["tok_emb"].astype(np.float64)
    want = _rms(E[toks[0]]) @ W["lm_head_item"].astype(np.float64).T
    np.testing.assert_allclose(logits[0], want, rtol=0, atol=1e-12)


def test_zero_query_gives_uniform_causal_average():
    # Wq = 0 -> every visible key scores 0 -> attention output is the mean of the
    # visible values; with Wv = Wo = I and no FFN: x_i + mean_{j<=i} n(x_j).
    w = _tiny_workload(target=ModelDims(1, 32, 4, 64, 34, 10))
    W = _zeros_like_weights(make_weights(w, "target"))
    W["l0.wv"] = np.eye(32, dtype=np.float32)
    W["l0.wo"] = np.eye(32, dtype=np.float32)
    W["l0.wk"] = np.random.default_rng(3).standard_normal((32, 32)).astype(np.float32)
    dec = Decoder(w.target, W, "fp32")
    toks = np.array([[1, 5, 9, 13, 2]])
    logits, _ = dec.forward(toks, np.arange(5))
    x = W["tok_emb"].astype(np.float64)[toks[0]]
    n = _rms(x)
    h = x + np.cumsum(n, axis=0) / np.arange(1, 6)[:, None]
    want = _rms(h) @ W["lm_head_item"].astype(np.float64).T
    np.testing.assert_allclose(logits[0], want, rtol=0, atol=1e-12)


def test_rope_is_complex_rotation_of_half_pairs():
    rng = np.random.default_rng(0)
    dh = 16
    x = rng.standard_normal((3, dh))
    pos = np.array([0, 7, 1000])
    z = x[:, :8] + 1j * x[:, 8:]
    theta = np.array([10000.0 ** (-(2.0 * i) / dh) for i in range(8)])
    zr = z * np.exp(1j * pos[:, None] * theta[None, :])
    want = np.concatenate([zr.real, zr.imag], axis=1)
    np.testing.assert_allclose(rope(x, pos), want, rtol=0, atol=1e-12)
    # q.k after rotation depends only on the position difference
    q, k = rng.standard_normal(dh), rng.standard_normal(dh)
    a = rope(q[None], np.array([5])) @ rope(k[None], np.array([2])).T
    b = rope(q[None], np.array([105])) @ rope(k[None], np.array([102])).T
    assert abs(a - b).max() < 1e-12


def test_swiglu_hand_value():
    # d=2, one head, f=1, attention off; gate weight 2, up weight 3, down 0.5 on
    # the first coordinate: x1' = 1 + 0.5 * silu(2) * 3 with silu(2) = 2/(1+e^-2).
    dims = ModelDims(1, 2, 1, 1, 2, 0)
    W = {"tok_emb": np.array([[1.0, 1.0], [0.0, 0.0]], np.float32),
         "l0.wq": np.zeros((2, 2), np.float32), "l0.wk": np.zeros((2, 2), np.float32),
         "l0.wv": np.zeros((2, 2), np.float32), "l0.wo": np.zeros((2, 2), np.float32),
         "l0.w_gate": np.array([[2.0, 0.0]], np.float32), "l0.w_up": np.array([[3.0, 0.0]], np.float32),
         "l0.w_down": np.array([[0.5], [0.0]], np.float32),
         "l0.attn_norm": np.ones(2, np.float32), "l0.ffn_norm": np.ones(2, np.float32),
         "final_norm": np.ones(2, np.float32), "lm_head_item": np.eye(2, dtype=np.float32)}
    dec = Decoder(dims, W, "fp32")
    logits, _ = dec.forward(np.array([[0]]), np.arange(1))
    s = 1.0 / math.sqrt(1.0 + RMS_EPS)          # n([1, 1])
    x1 = 1.0 + 0.5 * (2 * s / (1 + math.exp(-2 * s))) * (3 * s)
    want = np.array([x1, 1.0]) / math.sqrt((x1 * x1 + 1.0) / 2 + RMS_EPS)
    np.testing.assert_allclose(logits[0, 0], want, rtol=0, atol=1e-12)
    # hand value of the FFN output at eps -> 0: 0.5 * 3 * 2 / (1 + e^-2)
    assert abs(0.5 * 3 * 2 / (1 + math.exp(-2)) - 2.642391233933647) < 1e-12


def _one_head_d2(a, b):
    # d = 2, one head (d_head 2), FFN off, W_q = a I, W_k = b I, W_v = W_o = I,
    # identity item head; token 0 embeds to sqrt(2) e1, token 1 to sqrt(2) e2.
    dims = ModelDims(1, 2, 1, 1, 2, 0)
    W = {"tok_emb": np.array([[math.sqrt(2.0), 0.0], [0.0, math.sqrt(2.0)]], np.float64),
         "l0.wq": (a * np.eye(2)).astype(np.float64), "l0.wk": (b * np.eye(2)).astype(np.float64),
         "l0.wv": np.eye(2, dtype=np.float32), "l0.wo": np.eye(2, dtype=np.float32),
         "l0.w_gate": np.zeros((1, 2), np.float32), "l0.w_up": np.zeros((1, 2), np.float32),
         "l0.w_down": np.zeros((2, 1), np.float32),
         "l0.attn_norm": np.ones(2, np.float32), "l0.ffn_norm": np.ones(2, np.float32),
         "final_norm": np.ones(2, np.float32), "lm_head_item": np.eye(2, dtype=np.float32)}
    return Decoder(dims, W, "fp32")


def test_attention_scale_closed_form():
    # Sequence (token 0 at position 0, token 1 at position 1).  After the norm the
    # inputs are h0 = sqrt(2) r e1 and h1 = sqrt(2) r e2 with r = 1/sqrt(1 + eps).
    # With d_head = 2 the rotary angle of pair 0 at position p is p radians, so
    # q1 = a sqrt(2) r (-sin 1, cos 1), k0 = b sqrt(2) r e1, k1 = b sqrt(2) r (-sin 1, cos 1):
    #   q1.k0 = -2 a b r^2 sin 1,   q1.k1 = 2 a b r^2.
    # Scaled by 1/sqrt(d_head) = 1/sqrt(2), the score gap s11 - s10 is
    # sqrt(2) a b r^2 (1 + sin 1); a b is chosen to make it ln 3, so token 1's
    # attention weights are (1/4, 3/4).  Its output is x1 + h0/4 + 3 h1/4 =
    # sqrt(2) (r/4, 1 + 3r/4), and the identity head reads the ratio r / (4 + 3r).
    r = 1.0 / math.sqrt(1.0 + RMS_EPS)
    ab = math.log(3.0) / (math.sqrt(2.0) * r * r * (1.0 + math.sin(1.0)))
    dec = _one_head_d2(1.5, ab / 1.5)
    want = r / (4.0 + 3.0 * r)
    logits, _ = dec.forward(np.array([[0, 1]]), np.arange(2))
    assert abs(logits[0, 1, 0] / logits[0, 1, 1] - want) < 1e-12
    # the same value through the prefix-cache branch (prefix = token 0, path = token 1)
    got = dec.path_logits(dec.prefill(np.array([0])), [(1,)])[0]
    assert abs(got[0] / got[1] - want) < 1e-12
    # token 0 sees only itself: its output stays on e1
    assert abs(logits[0, 0, 1]) < 1e-15 and logits[0, 0, 0] > 0


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_causality_and_prefix_cache(dtype):
    w = _tiny_workload(dtype=dtype)
    dec = Decoder(w.target, make_weights(w, "target"), dtype)
    rng = np.random.default_rng(5)
    seq = rng.integers(0, w.target.vocab, size=9)
    full, _ = dec.forward(seq[None], np.arange(9))
    for i in (0, 3, 8):
        part, _ = dec.forward(seq[None, : i + 1], np.arange(i + 1))
        np.testing.assert_allclose(part[0, -1], full[0, i], rtol=0, atol=1e-12)
    cache = dec.prefill(seq[:6])
    got = dec.path_logits(cache, [tuple(seq[6:])])
    np.testing.assert_allclose(got[0], full[0, 8], rtol=0, atol=1e-12)
    np.testing.assert_allclose(dec.path_logits(cache, [()])[0], full[0, 5], rtol=0, atol=1e-12)


def test_tree_example_flattening():
    with open(os.path.join(GOLDEN, "tree_example.json")) as f:
        g = json.load(f)
    beams = [b for step in g["beams_by_step"] for b in step]
    nodes, parent, depth = flatten(beams)
    assert [n[-1] for n in nodes] == g["flattened"]
    m = ancestor_mask(parent)
    for i, n in enumerate(nodes):
        want = set(g["rows"][" ".join(n)])
        got = {nodes[j][-1] for j in range(len(nodes)) if m[i, j]}
        assert got == want


def test_tree_forward_equals_per_path_forward():
    # Flattened tree with the ancestor mask and depth positions (P + depth - 1)
    # gives the same logits as one causal forward per path.
    w = _tiny_workload()
    dec = Decoder(w.target, make_weights(w, "target"), "fp32")
    rng = np.random.default_rng(2)
    prefix = rng.integers(0, w.target.vocab, size=7)
    cache = dec.prefill(prefix)
    paths = [(11,), (12,), (11, 20), (12, 21), (11, 20, 30), (11, 20, 31), (13,), (13, 22)]
    nodes, parent, depth = flatten(paths)
    toks = np.array([[n[-1] for n in nodes]])
    pos = len(prefix) + np.array(depth) - 1
    tree, _ = dec.forward(toks, pos, prefix=cache, mask=ancestor_mask(parent).astype(bool))
    per = dec.path_logits(cache, nodes)
    np.testing.assert_allclose(tree[0], per, rtol=0, atol=1e-12)
    # flattened positions 0..Lf-1 would be a different (wrong) model
    bad, _ = dec.forward(toks, len(prefix) + np.arange(len(nodes)), prefix=cache,
                         mask=ancestor_mask(parent).astype(bool))
    assert np.abs(bad[0] - per).max() > 1e-6


def test_rmsnorm_epsilon_closed_form():
    # The norm's epsilon is 1e-6 (reading of the model details; LLaMA-7B's value).
    # A row whose mean square is itself 1e-6 makes it visible: [1e-3, -1e-3]
    # normalises to [1, -1] / sqrt(2) with epsilon 1e-6 (1/sqrt(11) with 1e-5).
    w = _tiny_workload(target=ModelDims(1, 2, 1, 1, 2, 0))
    W = {"tok_emb": np.array([[1e-3, -1e-3]], np.float64),
         "l0.wq": np.zeros((2, 2)), "l0.wk": np.zeros((2, 2)), "l0.wv": np.zeros((2, 2)), "l0.wo": np.zeros((2, 2)),
         "l0.w_gate": np.zeros((1, 2)), "l0.w_up": np.zeros((1, 2)), "l0.w_down": np.zeros((2, 1)),
         "l0.attn_norm": np.ones(2), "l0.ffn_norm": np.ones(2), "final_norm": np.ones(2),
         "lm_head_item": np.eye(2)}
    dec = Decoder(w.target, W, "fp32")
    logits, _ = dec.forward(np.array([[0]]), np.arange(1))
    np.testing.assert_allclose(logits[0, 0], [1 / math.sqrt(2.0), -1 / math.sqrt(2.0)], rtol=0, atol=1e-12)


def _bf16_block_d2(wv, wo, wg, wu, wd, wq=None):
    dims = ModelDims(1, 2, 1, 1, 2, 0)
    W = {"tok_emb": np.zeros((1, 2)), "l0.wq": np.zeros((2, 2)) if wq is None else wq, "l0.wk": np.eye(2),
         "l0.wv": wv, "l0.wo": wo, "l0.w_gate": wg, "l0.w_up": wu, "l0.w_down": wd,
         "l0.attn_norm": np.ones(2), "l0.ffn_norm": np.ones(2), "final_norm": np.ones(2),
         "lm_head_item": np.eye(2)}
    return Decoder(dims, W, "bf16")


def test_bf16_rounding_of_the_attention_output():
    # Precision contract: the attention output is rounded to bf16 before the o
    # projection.  W_q = 0 makes token 1 average the values of tokens 0 and 1;
    # W_v = W_o = I, FFN off.  Token 0's normed row [1, 1] (1/sqrt(1 + 1e-6) ->
    # 1 in bf16) and token 1's [1, 1 + 2^-6] / 1.00778 -> [0.9921875, 1.0078125]
    # average to [1 - 2^-8, 1 + 2^-8]; the second is a bf16 tie and rounds to 1,
    # so h_1 = x_1 + [1 - 2^-8, 1] (unrounded: 1 + 2^-8 in the second slot).
    dec = _bf16_block_d2(np.eye(2), np.eye(2), np.zeros((1, 2)), np.zeros((1, 2)), np.zeros((2, 1)))
    x = np.array([[[1.0, 1.0], [1.0, 1.0 + 2.0 ** -6]]])
    h, xo, k, v = dec.block(0, x, np.arange(2))
    assert h[0, 1, 0] == 1.0 + (1.0 - 2.0 ** -8) and h[0, 1, 1] == (1.0 + 2.0 ** -6) + 1.0
    assert (xo == h).all()                       # FFN off
    # k and v are bf16 values
    from oracle.numerics import round_bf16
    assert (round_bf16(k) == k).all() and (round_bf16(v) == v).all()


def test_bf16_rounding_of_the_swiglu_product():
    # Precision contract: SiLU(gate) * up is rounded to bf16 before the down
    # projection.  Attention off (W_v = 0), x = [1, 1] normalises to [1, 1] in
    # bf16; gate = up = the first coordinate, so the product is
    # SiLU(1) = 1 / (1 + e^-1) = 0.7310585786..., whose bf16 rounding is
    # 187 / 256 = 0.73046875; W_down puts it on the first coordinate.
    dec = _bf16_block_d2(np.zeros((2, 2)), np.eye(2), np.array([[1.0, 0.0]]), np.array([[1.0, 0.0]]),
                         np.array([[1.0], [0.0]]))
    x = np.array([[[1.0, 1.0]]])
    h, xo, _, _ = dec.block(0, x, np.arange(1))
    assert (h == x).all()
    assert xo[0, 0, 0] == 1.0 + 187.0 / 256.0 and xo[0, 0, 1] == 1.0
    assert abs(1.0 / (1.0 + math.exp(-1.0)) - 0.7310585786300049) < 1e-15


def test_bf16_rounding_of_the_final_norm():
    # The final norm's output is rounded to bf16 before the item head: with an
    # identity head the logits are bf16 values ([1, 3] normalises to
    # [0.4472..., 1.3416...] -> [229/512, 172/128]).
    dec = _bf16_block_d2(np.zeros((2, 2)), np.eye(2), np.zeros((1, 2)), np.zeros((1, 2)), np.zeros((2, 1)))
    lg = dec.head(np.array([[1.0, 3.0]]))
    assert lg[0, 0] == 229.0 / 512.0 and lg[0, 1] == 172.0 / 128.0


def test_bf16_rounding_of_the_normalised_inputs():
    # Precision contract: the normed rows entering q/k/v and gate/up are rounded
    # to bf16.  Both cases use x = [1, 1 + k/64], whose norm is x / sqrt((1 +
    # x_1^2) / 2 + 1e-6).
    # (1) Attention input: x = [1, 1.109375] normalises to [0.946876, 1.050440]
    # -> bf16 [242/256, 134/128]; W_v = [[1, 1], [0, 0]] sums them to 255/128
    # exactly (unrounded inputs: 1.997316, whose rounding is 2); one token
    # attends to itself, W_o = I, FFN off: h = x + [255/128, 0].
    dec = _bf16_block_d2(np.array([[1.0, 1.0], [0.0, 0.0]]), np.eye(2), np.zeros((1, 2)), np.zeros((1, 2)),
                         np.zeros((2, 1)))
    h, _, _, _ = dec.block(0, np.array([[[1.0, 1.109375]]]), np.arange(1))
    assert h[0, 0, 0] == 1.0 + 255.0 / 128.0 and h[0, 0, 1] == 1.109375
    # (2) FFN input: attention off, x = [1, 1.078125] normalises to [0.961726,
    # 1.036861] -> bf16 [246/256, 133/128]; gate = 64 x_0 (SiLU of 61.5 is 61.5 to
    # 1e-26), up = x_1 / 64, so SiLU(gate) * up = (246/256)(133/128) = 0.998474,
    # whose bf16 rounding is 1 (unrounded inputs: 0.997176, whose rounding is
    # 255/256); W_down puts it on the first coordinate.
    dec = _bf16_block_d2(np.zeros((2, 2)), np.eye(2), np.array([[64.0, 0.0]]), np.array([[0.0, 1.0 / 64.0]]),
                         np.array([[1.0], [0.0]]))
    h, xo, _, _ = dec.block(0, np.array([[[1.0, 1.078125]]]), np.arange(1))
    assert xo[0, 0, 0] == 1.0 + 1.0 and xo[0, 0, 1] == 1.078125
