"""Kernel-by-kernel parity at the full 7B shape (32 layers, d 4096, 32 heads,
FFN 11008, 32 users, 144-token prefixes with the shared 64-token prompt, the
t = 0 draft tree of 1,920 rows), at the relaxed workload's tree (3,840 rows),
at the stress shape (128 users with 1,024-token prefixes, 38,400 tree rows)
and at the small workload (d 1024): every step of the decoder blocks of
the GPU's prefill and tree forward (the LLaMA block of the implementation
details, Sec. 4.1, with tree-based attention, Sec. 3.3), recomputed by the
oracle's step function from the GPU's own inputs to that step, for a user who
forwards its whole prefix and one who takes the shared prompt's K/V from it;
and the 7B shape's draft model (4 layers, d 768, 12 heads, FFN 3072) in its
prefill and its forward of the first drafted level.

End to end, two correct bf16 computations of a 32-layer model at d 4096 drift
apart by more than the 2e-2 logit bar: each bf16 rounding point turns a small
difference into whole-ulp flips, and every layer adds more.  Fed its own
inputs, each step leaves only its own arithmetic to compare:
  * steps with bf16 results (the two RMSNorms, q/k/v with RoPE, attention,
    SiLU(gate) * up, the final norm): bit-exact, except elements whose GPU value
    is the rounding of a value within the GPU's own arithmetic error of the
    exact one (near-ties, and values near zero, where cancellation makes that
    error span several ulps);
  * steps with fp32 results (the o and down projections with their residual
    adds, the item head): within the GPU's own arithmetic error, and within the
    1e-4 fp32 bar.
The error bound of an element is derived from fp32 arithmetic (unit roundoff
u = 2^-24): a dot product of length K accumulated in fp32 is within
8 sqrt(K) u sum_k |x_k w_k| (a random walk of roundings, each at most u times
the partial sum, which sum_k |x_k w_k| bounds, with a wide margin), RMSNorm
within 64 u |y| (its fp32 sum of 4,096 squares), attention within 2^-14
sum_j p_j |v_j| (probabilities carried as two bf16 halves, about 16 bits, and
fp32 online softmax), SiLU(g) * u by propagating the bounds of g and u; a
residual add adds 8 u |y|.  A wrong weight, index or formula moves values by
far more.  At most 1% of a step's elements may be off the exact rounding.
Measured: 0.001-0.11% of a step's elements off the exact rounding, each within
0.07 of its bound; fp32 results within 1.4e-5 (0.007 of their bounds); the item
logits from the GPU's last residual within 6e-6.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from synth import get_workload, make_catalog, make_prefixes, make_weights  # noqa: E402
from oracle.model import Decoder, attend  # noqa: E402
from oracle.numerics import round_bf16  # noqa: E402

U = 2.0 ** -24
FLIP_FRACTION = 0.01  # at most this share of a step's elements off the exact rounding
FP32_BAR = 1e-4       # the fp32 logit bar, also held by every fp32 result here


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def dot_bound(xa: np.ndarray, W: np.ndarray) -> np.ndarray:
    """fp32 accumulation error bound of xa @ W.T (xa, W as fp64)."""
    return 8.0 * np.sqrt(W.shape[1]) * U * (np.abs(xa) @ np.abs(W).T)


def check_bf16(name, got_bits, exact, bound, stats):
    """got_bits: the GPU's bf16 results; exact: the oracle's unrounded values
    from the same inputs; bound: the GPU's arithmetic error bound per element.
    Equal after rounding, or the GPU's value is the rounding of some value
    within the bound of the exact one (a near-tie, or a value near zero whose
    bound spans several ulps)."""
    want = round_bf16(exact)
    got = bf16_to_f64(got_bits)
    diff = got != want
    n = int(diff.sum())
    worst = 0.0
    if n:
        g, y, b = got[diff], exact[diff], np.broadcast_to(bound, exact.shape)[diff]
        with np.errstate(divide="ignore"):
            ulp = np.where(g != 0, 2.0 ** (np.floor(np.log2(np.abs(np.where(g != 0, g, 1.0)))) - 7), 0.0)
        # the rounding interval of g reaches the bound around the exact value
        excess = np.maximum(np.abs(g - y) - 0.5 * ulp, 0.0)
        worst = float((excess / b).max())
        assert worst <= 1.0, (name, worst)
        assert n <= FLIP_FRACTION * got.size, (name, n, got.size)
    old = stats.get(name, (0, 0, 0.0))
    stats[name] = (old[0] + n, old[1] + got.size, max(old[2], worst))


def check_f32(name, got, exact, bound, stats):
    r = float((np.abs(got - exact) / bound).max())
    assert r <= 1.0, (name, r, float(np.abs(got - exact).max()))
    assert np.abs(got - exact).max() <= FP32_BAR, (name, float(np.abs(got - exact).max()))
    old = stats.get(name, (0.0, 0.0))
    stats[name] = (max(old[0], float(np.abs(got - exact).max())), max(old[1], r))


class Capture:
    """The residual and activation capture of one forward of ``model`` (0
    target, 1 draft; the one after ``skip`` others of it), on the device; the
    first ``rows`` rows of the forward are kept."""

    def __init__(self, eng, dims, rows, fn, model=0, skip=0):
        self.nl, self.d, self.f, self.R = dims.n_layers, dims.d_model, dims.d_ffn, rows
        self.x = torch.zeros((2 * self.nl + 1, rows, self.d), dtype=torch.float32, device="cuda")
        self.layer = rows * (6 * self.d + self.f)
        self.act = torch.zeros((self.nl * self.layer + rows * self.d,), dtype=torch.int16, device="cuda")
        plan = torch.full((3 * rows + 1,), -2, dtype=torch.int32, device="cuda")
        eng.atspeed_capture_hidden(self.x, plan, rows, act=self.act, model=model, skip=skip)
        fn()
        torch.cuda.synchronize()
        p = plan.cpu().numpy()
        self.M = int(p[3 * rows])                 # rows of the forward; the first min(M, R) are captured
        assert self.M > 0, self.M
        self.user, self.pos, self.slot = p[:3 * rows].reshape(3, rows)[:, :min(self.M, rows)]

    def take(self, idx):
        """Host copies of the captured values of rows ``idx``: x [2 nl + 1, n, d]
        (fp64) and per layer the seven bf16 arrays (uint16)."""
        ix = torch.from_numpy(np.asarray(idx)).cuda()
        x = self.x[:, ix].cpu().numpy().astype(np.float64)
        acts = []
        for l in range(self.nl + 1):
            base = l * self.layer
            parts = []
            for k in range(6 if l < self.nl else 1):
                a = self.act[base + k * self.R * self.d: base + (k + 1) * self.R * self.d].view(self.R, self.d)
                parts.append(a[ix].cpu().numpy().view(np.uint16))
            if l < self.nl:
                a = self.act[base + 6 * self.R * self.d: base + self.layer].view(self.R, self.f)
                parts.append(a[ix].cpu().numpy().view(np.uint16))
            acts.append(parts)
        return x, acts


def prefix_rows(cp, users, P):
    """Per user: (S, captured values of its P prefix rows), the shared prompt
    positions [0, S) being user 0's rows (same tokens; the prefill copies their
    K/V), the rest the user's own."""
    rows0 = np.nonzero(cp.user == 0)[0]
    assert (cp.pos[rows0] == np.arange(P)).all(), "user 0 forwards every prefix position"
    out = {}
    for u in users:
        ru = np.nonzero(cp.user == u)[0]
        S = int(cp.pos[ru][0])
        assert (cp.pos[ru] == np.arange(S, P)).all()
        out[u] = (S, cp.take(np.concatenate([rows0[:S], ru])))
    return out


def tree_rows(cp, users, T, parent, depth, P, L):
    """Per user: (nodes, ancestor-or-self mask among the user's forwarded
    nodes, captured values of those rows)."""
    out = {}
    for u in users:
        r = np.nonzero(cp.user == u)[0]
        nodes = cp.slot[r] - u * T
        assert len(r) > 0 and (nodes >= 0).all() and (depth[u, nodes] < L).all()
        assert (cp.pos[r] == P + depth[u, nodes] - 1).all()
        where = {int(n): i for i, n in enumerate(nodes)}
        mask = np.zeros((len(r), len(r)), dtype=bool)
        for i, n in enumerate(nodes):
            a = int(n)
            while a >= 0:
                mask[i, where[a]] = True
                a = int(parent[u, a])
        out[u] = (nodes, mask, cp.take(r))
    return out


def check_layers(dec, dims, layers, pre_cap, tree_cap, depth, P, stride, stats_b, stats_f, tag):
    """Every step of blocks ``layers`` on the captured prefix rows (every
    ``stride``-th a user computed itself, its last included) and tree rows."""
    nl, d, H, dh = dims.n_layers, dims.d_model, dims.n_heads, dims.d_head

    def heads(bits, n):   # [n, d] bf16 bits -> [1, H, n, dh] fp64
        return bf16_to_f64(bits).reshape(1, n, H, dh).transpose(0, 2, 1, 3)

    def rot_pairs(b):     # a rotated column's bound: its own and its rotate-half partner's
        bb = b.reshape(b.shape[0], H, 2, dh // 2)
        return (bb + bb[:, :, ::-1]).reshape(b.shape)

    for l in layers:
        dec._cache.clear()                       # one layer's fp64 weights at a time
        p_ = f"l{l}."
        Wq, Wk, Wv, Wo = (dec.W(p_ + n_) for n_ in ("wq", "wk", "wv", "wo"))
        Wg, Wu, Wd = (dec.W(p_ + n_) for n_ in ("w_gate", "w_up", "w_down"))
        for u in tree_cap:
            S, (xp, ap) = pre_cap[u]
            nodes, mask, (xt, at) = tree_cap[u]
            pk_ = heads(ap[l][2], P)[0]          # the user's prefix K/V of this layer [H, P, dh]
            pv_ = heads(ap[l][3], P)[0]
            own = np.arange(S, P)[::-1][::stride][::-1]
            for kind, x, a, pos, n, sel in (("prefix", xp, ap, np.arange(P), P, own),
                                            ("tree", xt, at, P + depth[u, nodes] - 1, len(nodes),
                                             np.arange(len(nodes)))):
                xn1, q, k, v, ao, xn2, act = a[l]
                y = dec.norm(l, "attn_norm", x[2 * l][sel])
                check_bf16("attn_norm", xn1[sel], y, 64 * U * np.abs(y), stats_b)
                h1 = bf16_to_f64(xn1[sel])
                yq, yk, yv = (t[0].transpose(1, 0, 2).reshape(len(sel), d) for t in dec.qkv(l, h1[None], pos[sel]))
                check_bf16("q", q[sel], yq, rot_pairs(dot_bound(h1, Wq)), stats_b)
                check_bf16("k", k[sel], yk, rot_pairs(dot_bound(h1, Wk)), stats_b)
                check_bf16("v", v[sel], yv, dot_bound(h1, Wv), stats_b)
                # the checked queries against every key of the forward (the GPU's k/v)
                if kind == "prefix":
                    msk = np.arange(n)[None, :] <= pos[sel][:, None]
                    kw, kwa = {}, {}
                else:
                    msk = mask
                    kw, kwa = dict(pk=pk_, pv=pv_), dict(pk=pk_, pv=np.abs(pv_))
                qh, kh, vh = heads(q[sel], len(sel)), heads(k, n), heads(v, n)
                yo = dec.merge_heads(attend(qh, kh, vh, msk, **kw))[0]
                yav = dec.merge_heads(attend(qh, kh, np.abs(vh), msk, **kwa))[0]   # sum_j p_j |v_j|
                check_bf16("attention", ao[sel], yo, 2.0 ** -14 * yav, stats_b)
                a1 = bf16_to_f64(ao[sel])
                y = x[2 * l][sel] + a1 @ Wo.T
                check_f32("o + residual", x[2 * l + 1][sel], y, dot_bound(a1, Wo) + 8 * U * np.abs(y), stats_f)
                y = dec.norm(l, "ffn_norm", x[2 * l + 1][sel])
                check_bf16("ffn_norm", xn2[sel], y, 64 * U * np.abs(y), stats_b)
                h2 = bf16_to_f64(xn2[sel])
                g_, u_ = h2 @ Wg.T, h2 @ Wu.T            # for the bound only
                bg, bu = dot_bound(h2, Wg), dot_bound(h2, Wu)
                sg = 1.0 / (1.0 + np.exp(-g_))
                sil = g_ * sg
                dsil = np.abs(sg * (1.0 + g_ * (1.0 - sg)))
                ya = dec.swiglu(l, h2)
                ba = np.abs(u_) * (dsil * bg + 4 * U * np.abs(sil)) + np.abs(sil) * bu + 4 * U * np.abs(ya)
                check_bf16("silu(gate)*up", act[sel], ya, ba, stats_b)
                if kind == "tree" or l + 1 < nl:   # a prefill captures no residual after the last layer
                    a2 = bf16_to_f64(act[sel])
                    y = x[2 * l + 1][sel] + a2 @ Wd.T
                    check_f32("down + residual", x[2 * l + 2][sel], y, dot_bound(a2, Wd) + 8 * U * np.abs(y),
                              stats_f)
        print(f"[{tag}] layer {l:2d} checked; elements off the exact rounding so far: "
              + ", ".join(f"{k_} {v_[0]}" for k_, v_ in stats_b.items()), flush=True)


def report(tag, stats_b, stats_f):
    print(f"[{tag}] bf16 steps (elements off the exact rounding / elements, largest distance over its bound): "
          + ", ".join(f"{k_} {v_[0]}/{v_[1]} ({v_[2]:.3f})" for k_, v_ in stats_b.items()), flush=True)
    print(f"[{tag}] fp32 steps (max |err|, largest error over its bound): "
          + ", ".join(f"{k_} {v_[0]:.2e} ({v_[1]:.3f})" for k_, v_ in stats_f.items()), flush=True)


# b7: every layer, every prefix row the two users forward; stress (1,024-token
# prefixes, 38,400 tree rows: the long-context attention and the large-batch
# tile shapes): three layers and every 8th prefix row (the last included) of
# the first two users, whose rows lead the forward
CASES = {
    "b7": dict(users=(0, 31), layers=None, stride=1, rows=None),
    # the relaxed workload's t = 0 tree: 3N = 120 nodes per user, 3,840 rows
    # (other tile shapes than at 1,920 rows)
    "b7_relaxed": dict(users=(0, 31), layers=(0, 15, 31), stride=4, rows=None),
    "stress": dict(users=(0, 1), layers=(0, 15, 31), stride=8, rows=2048),
    # d 1024, 16 heads, FFN 2816, 16 users with their own 120-token prefixes
    "small": dict(users=(0, 15), layers=None, stride=1, rows=None),
}


@pytest.mark.parametrize("case", list(CASES))
def test_every_kernel_against_the_oracle_step(case):
    from paper_2410_05165_amd.binding import Engine
    cfg = CASES[case]
    w = get_workload(case)
    m = w.target
    nl, P, L, B = m.n_layers, w.prefix_len, w.L, w.batch
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    print(f"[{case} kernels] generating weights", flush=True)
    tw, dw = make_weights(w, "target"), make_weights(w, "draft")
    eng = Engine(w, tw, dw, cat)
    prefix = torch.from_numpy(pre).cuda()

    print(f"[{case} kernels] prefill with the capture armed", flush=True)
    cp = Capture(eng, m, cfg["rows"] or B * P, lambda: eng.atspeed_prefill(prefix))
    pre_cap = prefix_rows(cp, cfg["users"], P)
    del cp
    torch.cuda.empty_cache()

    print(f"[{case} kernels] draft, then the tree forward with the capture armed", flush=True)
    eng.atspeed_draft()
    T = eng.max_nodes
    logits = torch.full((B, T, w.n_item_tokens), float("nan"), dtype=torch.float32, device="cuda")
    ct = Capture(eng, m, cfg["rows"] or B * T, lambda: eng.atspeed_tree_logits(logits))
    assert ct.M == B * 3 * w.N, ct.M         # the t = 0 tree: drafted depths 1..3
    tn, tt, tp, td, _ = (a.cpu().numpy() for a in eng.tree_tensors(B))
    tree_cap = tree_rows(ct, cfg["users"], T, tp, td, P, L)
    assert all(len(v_[0]) == 3 * w.N for v_ in tree_cap.values())
    lg = logits.cpu().numpy()
    del ct
    eng.close()

    dec = Decoder(m, tw, w.dtype, cache_f64=True)
    stats_b, stats_f = {}, {}
    check_layers(dec, m, cfg["layers"] or range(nl), pre_cap, tree_cap, td, P, cfg["stride"], stats_b, stats_f,
                 f"{case} kernels")
    dec._cache.clear()
    Wh = dec.W("lm_head_item")
    for u, (nodes, mask, (xt, at)) in tree_cap.items():
        y = dec.norm(-1, "", xt[2 * nl])
        check_bf16("final_norm", at[nl][0], y, 64 * U * np.abs(y), stats_b)
        hf = bf16_to_f64(at[nl][0])
        y = hf @ Wh.T
        check_f32("item head", lg[u, nodes], y, dot_bound(hf, Wh) + 8 * U * np.abs(y), stats_f)
    report(f"{case} kernels", stats_b, stats_f)


def test_b7_draft_kernels_against_the_oracle_step():
    """The 7B shape's draft (4 layers, d 768, 12 heads of 64, FFN 3072): its
    prefill and its forward of the first drafted level (N = 20 nodes per user at
    depth 1, attending to the draft's prefix cache and themselves; the draft's
    first forward at t = 0, over the paths of the empty beams, has no rows)."""
    from paper_2410_05165_amd.binding import Engine
    w = get_workload("b7")
    m = w.draft
    P, L, B, users = w.prefix_len, w.L, w.batch, (0, 31)
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    tw, dw = make_weights(w, "target"), make_weights(w, "draft")
    eng = Engine(w, tw, dw, cat)
    prefix = torch.from_numpy(pre).cuda()
    print("[b7 draft kernels] prefill with the draft's capture armed", flush=True)
    cp = Capture(eng, m, B * P, lambda: eng.atspeed_prefill(prefix), model=1)
    pre_cap = prefix_rows(cp, users, P)
    del cp
    print("[b7 draft kernels] draft with the capture of its second forward armed", flush=True)
    T = eng.max_nodes
    ct = Capture(eng, m, B * w.N, lambda: eng.atspeed_draft(), model=1, skip=1)
    assert ct.M == B * w.N, ct.M
    tn, tt, tp, td, _ = (a.cpu().numpy() for a in eng.tree_tensors(B))
    tree_cap = tree_rows(ct, users, T, tp, td, P, L)
    assert all(len(v_[0]) == w.N and (td[u, v_[0]] == 1).all() for u, v_ in tree_cap.items())
    del ct
    eng.close()
    dec = Decoder(m, dw, w.dtype, cache_f64=True)
    stats_b, stats_f = {}, {}
    check_layers(dec, m, range(m.n_layers), pre_cap, tree_cap, td, P, 1, stats_b, stats_f, "b7 draft kernels")
    dec._cache.clear()
    for u, (nodes, mask, (xt, at)) in tree_cap.items():
        y = dec.norm(-1, "", xt[2 * m.n_layers])
        check_bf16("final_norm", at[m.n_layers][0], y, 64 * U * np.abs(y), stats_b)
    report("b7 draft kernels", stats_b, stats_f)


def test_capture_error_paths_and_a_small_capture():
    """The capture call's argument checks, and a capture of the tiny fp32
    workload's prefill (residual only: activations are captured for bf16 models)
    against the oracle's blocks on the same inputs within the fp32 bar."""
    from paper_2410_05165_amd.binding import AtspeedError, Engine
    w = get_workload("tiny")
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    tw, dw = make_weights(w, "target"), make_weights(w, "draft")
    eng = Engine(w, tw, dw, cat)
    m = w.target
    x = torch.zeros((2 * m.n_layers + 1, w.prefix_len, m.d_model), dtype=torch.float32, device="cuda")
    plan = torch.zeros(3 * w.prefix_len + 1, dtype=torch.int32, device="cuda")
    act = torch.zeros(16, dtype=torch.int16, device="cuda")
    for what, kw in (("model 2", dict(model=2)), ("skip -1", dict(skip=-1)), ("max_rows 0", dict(max_rows=0)),
                     ("no plan", dict(plan=None)), ("activations of an fp32 model", dict(act=act))):
        args = dict(x=x, plan=plan, max_rows=w.prefix_len)
        args.update(kw)
        with pytest.raises(AtspeedError) as ex:
            eng.atspeed_capture_hidden(**args)
        assert ex.value.status == 1, what          # ATSPEED_E_INVALID
    eng.atspeed_capture_hidden()                    # all null: disarmed
    eng.atspeed_capture_hidden(x=x, plan=plan, max_rows=w.prefix_len)
    eng.atspeed_prefill(torch.from_numpy(pre).cuda())
    torch.cuda.synchronize()
    p = plan.cpu().numpy()
    assert p[3 * w.prefix_len] == w.prefix_len
    assert (p[w.prefix_len:2 * w.prefix_len] == np.arange(w.prefix_len)).all()
    assert (p[2 * w.prefix_len:3 * w.prefix_len] == -1).all()
    xs = x.cpu().numpy().astype(np.float64)
    eng.close()
    dec = Decoder(m, tw, w.dtype)
    P = w.prefix_len
    assert np.abs(xs[0] - dec.embed(pre[0][None])[0]).max() == 0.0
    for l in range(m.n_layers):
        h, xo, _, _ = dec.block(l, xs[2 * l][None], np.arange(P))
        assert np.abs(h[0] - xs[2 * l + 1]).max() <= FP32_BAR
        if l + 1 < m.n_layers:
            assert np.abs(xo[0] - xs[2 * l + 2]).max() <= FP32_BAR
