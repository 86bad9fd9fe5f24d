#!/usr/bin/env python3
"""Throughput of the AtSpeed top-K decode on one MI355X.

Workload (default): the LLaMA-7B-shaped target (32 layers, d 4096, 32 heads,
FFN 11008, vocabulary 33,024 with 1,024 item tokens), 4-layer draft, 100,000
random 4-token items, 32 users with 144-token prefixes, K = 10, N = 20,
gamma = 4, strict verification; random-init bf16 weights N(0, 0.02).

A step is one ``atspeed_decode_topk`` over the batch: prefill of target and
draft, then speculative steps (device drafting, one target forward over the
tree, item log-softmax, cumulative log-probs, trie-constrained TopK, strict
acceptance) until every user's top-K list is complete, with the library's own
drafts (natural acceptance; random weights accept about nothing).  value =
users x steps / time.  Beside it: the same decode with the level-1 start and
tree-KV reuse, under the replay-paper-AS and replay-all-accept profiles, the
t = 0 verify step alone, the decode-bound probe, the relaxed (config-4)
decode, the strict and relaxed decodes after draft alignment (AtSpeed-S /
AtSpeed-R training of the draft's item head on the benchmark users, measured on
them and on held-out users), and the target-only beam search that the paper's
walltime speedup WS is measured against (with the speedup of each decode, and
WS at batch sizes 1, 4 and 32 with the random and the aligned draft), and the
stress decode (config 5: 1M items, 128 users x 1,024 tokens, K 50); the
roofline kernel is the target's gate/up GEMM over the timed decodes.

Prints ONE JSON line.  Progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA, published figure
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E, published figure


def gemm_code_sha(path=None):
    """sha256 of the GEMM source with comments and whitespace removed: the
    counter record stays valid across comment-only edits, not across code ones."""
    import hashlib
    import re
    path = path or os.path.join(ROOT, "paper_2410_05165_amd", "csrc", "gemm.hip")
    text = open(path, encoding="utf-8").read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return hashlib.sha256("".join(text.split()).encode()).hexdigest()


def gemm_traffic(kernel_key, workload):
    """HBM bytes per launch of a kernel from the committed rocprofv3 counter record
    (taken on the b7 verify step), or None for another workload or if the kernel
    code changed since the counters were taken."""
    if workload != "b7":
        return None
    path = os.path.join(ROOT, "profiles", "traffic_b7.json")
    try:
        rec = json.load(open(path))
        ent = rec["kernels"][kernel_key]
        return ent["bytes_per_launch"] if rec["gemm_code_sha256"] == gemm_code_sha() else None
    except (OSError, KeyError, ValueError):
        return None


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def catalog_children(cat):
    """prefix (tuple of codes) -> sorted codes that extend it within the catalog."""
    kids = {}
    for row in cat.tolist():
        for l in range(len(row)):
            kids.setdefault(tuple(row[:l]), set()).add(row[l])
    return {k: sorted(v) for k, v in kids.items()}


def tree_arrays(eng, trees, B):
    """Per-user path lists as the context's tree arrays (level-ordered, deduplicated):
    n_nodes [B], token, parent, depth [B, T] int32."""
    import numpy as np
    w = eng.w
    T = eng.max_nodes
    n = np.zeros(B, np.int32)
    tok = np.zeros((B, T), np.int32)
    par = np.full((B, T), -1, np.int32)
    dep = np.zeros((B, T), np.int32)
    for u, paths in enumerate(trees):
        order = {}
        for p in paths:
            for d in range(1, len(p) + 1):
                order.setdefault(tuple(p[:d]), len(order))
        nodes = sorted(order, key=lambda q: (len(q), order[q]))
        index = {q: i for i, q in enumerate(nodes)}
        n[u] = len(nodes)
        for i, q in enumerate(nodes):
            tok[u, i] = w.target.item_base + w.codebook * (len(q) - 1) + q[-1]
            par[u, i] = index[q[:-1]] if len(q) > 1 else -1
            dep[u, i] = len(q)
    return n, tok, par, dep


def upload_tree(eng, trees, B):
    """Write per-user path lists into the context's tree (level-ordered, deduplicated)."""
    import torch
    n, tok, par, dep = tree_arrays(eng, trees, B)
    tn, tt, tp, td, tq = eng.tree_tensors(B)
    tn.copy_(torch.from_numpy(n))
    tt.copy_(torch.from_numpy(tok))
    tp.copy_(torch.from_numpy(par))
    td.copy_(torch.from_numpy(dep))
    tq.zero_()


def replay_all_accept_tree(eng, kids, w, levels):
    """Per user: drafted level j = the target's TopK of level j, padded to N with
    other valid extensions of the drafted level j-1 (in slot and code order)."""
    B = w.batch
    trees = []
    for u in range(B):
        nodes = []
        prev = [()]
        for j, (t, nb, paths, _) in enumerate(levels):
            top = [tuple(int(c) for c in paths[u, k, :j + 1]) for k in range(nb[u])]
            lvl = list(top)
            seen = set(top)
            for p in prev:
                if len(lvl) >= w.N:
                    break
                for c in kids.get(p, []):
                    q = p + (c,)
                    if q not in seen:
                        lvl.append(q)
                        seen.add(q)
                        if len(lvl) >= w.N:
                            break
            nodes.extend(lvl)
            prev = lvl
        trees.append(nodes)
    return trees


# Continuation probability of the forced-acceptance profile: accepted levels per
# step a ~ P(a >= j) = ALPHA^j truncated at the L - t levels left, so that at
# t = 0 (four levels) E[a] = 0.675 + 0.675^2 + 0.675^3 + 0.675^4 = 1.64, the
# acceptance steps AtSpeed-S reaches at K = 10 on Amazon Beauty (Table 1).
AS_ALPHA = 0.675


def replay_as_steps(kids, w, levels, seed):
    """Trees of one decode under forced acceptance.  At state t a user draws a
    accepted levels; drafted levels t+1..t+a hold the target's TopK of that level
    (padded to N as in the replay-all-accept tree), level t+a+1 holds N other
    valid extensions (none of the target's TopK, so strict verification rejects
    there and takes the target's level as the bonus), and t moves to t+a+1.
    Returns [(trees, accepted, t_after)] per step; finished users get []."""
    import numpy as np
    rng = np.random.default_rng(seed)
    B, L, N = w.batch, w.L, w.N
    t = [0] * B
    steps = []

    def top(u, depth):
        _, nb, paths, _ = levels[depth - 1]
        return [tuple(int(c) for c in paths[u, k, :depth]) for k in range(nb[u])]

    while any(tu < L for tu in t):
        trees, acc, after = [], [], []
        for u in range(B):
            if t[u] >= L:
                trees.append([]); acc.append(-1); after.append(L)
                continue
            a = 0
            while a < L - t[u] and rng.random() < AS_ALPHA:
                a += 1
            prev = top(u, t[u]) if t[u] > 0 else [()]
            nodes = [p for p in prev if p]
            for depth in range(t[u] + 1, min(t[u] + a + 1, L) + 1):
                tp = top(u, depth)
                seen = set(tp)
                if depth <= t[u] + a:           # accepted level: the target's TopK, padded
                    lvl = list(tp)
                else:                           # the rejected level: other extensions only
                    lvl = []
                for p in prev:
                    if len(lvl) >= N:
                        break
                    for c in kids.get(p, []):
                        q = p + (c,)
                        if q not in seen:
                            lvl.append(q)
                            seen.add(q)
                            if len(lvl) >= N:
                                break
                nodes.extend(lvl)
                prev = lvl
            trees.append(nodes)
            acc.append(a)
            t[u] = min(L, t[u] + a + 1)
            after.append(t[u])
        steps.append((trees, acc, after))
    return steps


def decode_replay_as(eng, w, prefix, levels, kids, reps, seed=1):
    """Whole decode (prefill, then per step the device draft and a verify of the
    forced-acceptance tree, copied device-to-device over the drafted one) under
    the replay-paper-AS profile.  Returns the profile's figures."""
    import numpy as np
    import torch
    B = w.batch
    steps = replay_as_steps(kids, w, levels, seed)
    dev_trees = [tuple(torch.from_numpy(a).to(prefix.device) for a in tree_arrays(eng, tr, B)) for tr, _, _ in steps]
    tn, tt, tp, td, tq = eng.tree_tensors(B)
    acc = torch.zeros(B, dtype=torch.int32, device=prefix.device)
    ta = torch.zeros(B, dtype=torch.int32, device=prefix.device)

    def decode(check):
        eng.atspeed_prefill(prefix)
        for s, (n, tok, par, dep) in enumerate(dev_trees):
            eng.atspeed_draft()
            tn.copy_(n); tt.copy_(tok); tp.copy_(par); td.copy_(dep); tq.zero_()
            eng.atspeed_verify(acc, ta)
            if check:
                a_exp, t_exp = steps[s][1], steps[s][2]
                got_a, got_t = acc.cpu().numpy(), ta.cpu().numpy()
                for u in range(B):
                    if a_exp[u] >= 0:
                        assert got_a[u] == a_exp[u] and got_t[u] == t_exp[u], (s, u, got_a[u], a_exp[u])

    decode(True)                                # the library accepts exactly the forced levels
    final = eng.atspeed_get_state(B)
    assert (final[2] == levels[-1][2]).all(), "replayed decode differs from target beam search"
    for _ in range(2):                          # with the checked decode: 3 warm-ups
        decode(False)
    torch.cuda.synchronize()
    tt_ = []
    for _ in range(reps):
        a = time.perf_counter()
        decode(False)
        torch.cuda.synchronize()
        tt_.append(time.perf_counter() - a)
    ms = 1e3 * float(np.median(tt_))
    first = [a for a in steps[0][1] if a >= 0]
    return dict(lists_per_s=B / (ms * 1e-3), ms_per_decode=ms, steps=len(steps),
                accepted_first_step_mean=float(np.mean(first)),
                accepted_mean=float(np.mean([a for _, acc_, _ in steps for a in acc_ if a >= 0])),
                profile="replay-paper-AS (first rejection forced; AS@10 = 1.64 at t = 0)")


def gpu_target_beam_search(eng, w, prefix, upload_tree):
    """GPU target-only beam search: verify on trees holding only the Y_t paths."""
    eng.atspeed_prefill(prefix)
    levels = []
    for _ in range(w.L):
        t, nb, paths, sc = eng.atspeed_get_state(w.batch)
        trees = [[tuple(int(c) for c in paths[u, k, :t[u]]) for k in range(nb[u])] if t[u] > 0 else []
                 for u in range(w.batch)]
        upload_tree(eng, trees, w.batch)
        eng.atspeed_verify()
        levels.append(eng.atspeed_get_state(w.batch))
    return levels


def cpu_baseline(w, tw, dw, pre, cat, gpu_items):
    """The oracle's whole decode of user 0 under the natural profile (fp64): the
    target's and the draft's prefill, then speculative steps -- draft beam search
    (Eq. 1), per-path target forwards of the levels Algorithm 1 examines,
    strict verification -- until the top-K list is complete."""
    from oracle.model import Decoder
    from oracle.search import model_scorer, sd_decode_strict
    from oracle.trie import Trie
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    trie = Trie(cat)
    tgt = Decoder(w.target, tw, w.dtype, cache_f64=False)
    dft = Decoder(w.draft, dw, w.dtype)
    log("cpu baseline: oracle decode of user 0 (timed: prefill of both models + speculative steps)")
    t0 = time.perf_counter()
    lp = model_scorer(tgt, tgt.prefill(pre[0]), w.target.item_base, w.codebook)
    lq = model_scorer(dft, dft.prefill(pre[0]), w.draft.item_base, w.codebook)
    final, steps = sd_decode_strict(lp, lq, trie, w.K, w.N, w.gamma, w.L, w.codebook)
    dt = time.perf_counter() - t0
    got = [tuple(int(c) for c in row) for row in gpu_items]
    same = sum(1 for p, _ in final if p in set(got))
    return dict(value=1.0 / dt, unit="lists/s", cores=int(threads), kind="oracle",
                sample=f"whole decode of user 0 of {w.batch} (natural drafts: fp64 prefill of target and draft, "
                       f"{len(steps)} speculative steps of draft beam search + per-path target forwards + "
                       f"Algorithm 1), {dt:.1f} s; its top-{w.K} list shares {same} of {w.K} items with the GPU's "
                       f"(bf16 vs fp64 logits); host cpus={os.cpu_count()}")


def decode_bound_probe(eng, w, prefix, levels, steps, users=None):
    """Target-only beam step at t = 1 (the K beams of each of the first ``users``
    users forwarded, K rows per user): the weights and the prefix KV cache stream
    once per step with little arithmetic per byte, so it is HBM-bound at few
    users; reports its algorithmic bytes/s."""
    import torch
    K, L = w.K, w.L
    B = w.batch if users is None else users
    eng.atspeed_prefill(prefix[:B].contiguous())
    t1, nb1, p1, s1 = (x[:B] for x in levels[0])
    upload_tree(eng, [[tuple(int(c) for c in p1[u, k, :1]) for k in range(nb1[u])] for u in range(B)], B)
    rows = int(nb1.sum())

    def step():
        eng.atspeed_set_state(t1, nb1, p1, s1)
        eng.atspeed_verify()
    for _ in range(2):
        step()
    torch.cuda.synchronize()
    a = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms = 1e3 * (time.perf_counter() - a) / steps
    m = w.target
    weights = m.n_layers * (4 * m.d_model ** 2 + 3 * m.d_model * m.d_ffn) * 2 + w.n_item_tokens * m.d_model * 2
    kv = m.n_layers * 2 * B * w.prefix_len * m.d_model * 2
    gbs = (weights + kv) / (ms * 1e-3) / 1e9
    log(f"decode-bound probe: {B} users, {rows} rows, {ms:.2f} ms/step, {gbs:.0f} GB/s "
        f"({gbs / PEAK_HBM_GBS:.1%} of HBM)")
    return dict(users=B, rows=rows, ms_per_step=round(ms, 3), bytes=weights + kv, gbs=round(gbs, 1),
                hbm_frac=round(gbs / PEAK_HBM_GBS, 4),
                what="target-only beam step at t=1: target weights + prefix KV read once per step")


def timed_decodes(eng, w, prefix, steps, warmup, roofline=True):
    """``warmup`` untimed decodes, then exactly ``steps`` timed ones (host clock,
    bracketed by device synchronisation).  With ``roofline`` the target's gate/up
    GEMM launches inside the timed region are bracketed by HIP events on the
    library's stream, with their algorithmic flops (2 x rows x 2f x d per launch)."""
    import ctypes as C
    import numpy as np
    import torch
    from paper_2410_05165_amd.binding import Stats
    B, K, L = w.batch, w.K, w.L
    items = torch.zeros((B, K, L), dtype=torch.int32, device=prefix.device)
    scores = torch.zeros((B, K), dtype=torch.float32, device=prefix.device)
    n = torch.zeros(B, dtype=torch.int32, device=prefix.device)
    for _ in range(warmup):
        eng.atspeed_decode_topk(prefix, items, scores, n, None)
    torch.cuda.synchronize()
    if roofline:
        eng.atspeed_set_timing(["gu"], target_only=True)
    per = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        a = time.perf_counter()
        eng.atspeed_decode_topk(prefix, items, scores, n, None)  # returns after its last step's synchronisation
        per.append(time.perf_counter() - a)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gu = None
    if roofline:
        ms, nl, gf = eng.atspeed_get_timing()["gu"]
        eng.atspeed_set_timing(False)
        gu = dict(ms=ms, launches=int(nl), gflop=gf)
    out = (items.cpu().numpy(), scores.cpu().numpy(), n.cpu().numpy())
    # stage times, steps and accepted levels from one more decode outside the
    # timed region (the per-stage timing synchronises between the stages)
    acc = np.zeros((L, eng.cfg.max_batch), np.int32)
    st = Stats()
    st.accepted = acc.ctypes.data_as(C.POINTER(C.c_int32))
    eng.atspeed_decode_topk(prefix, items, scores, n, st)
    torch.cuda.synchronize()
    r = dict(lists_per_s=B * steps / elapsed, ms_per_decode=1e3 * elapsed / steps,
             ms_per_decode_median=1e3 * float(np.median(per)), steps=int(st.n_steps),
             ms_prefill=round(st.ms_prefill, 3), ms_draft=round(st.ms_draft, 3), ms_verify=round(st.ms_verify, 3),
             lists_per_s_decode_only=B / ((st.ms_draft + st.ms_verify) / 1e3),
             target_tree_rows=int(st.rows_target), accepted_levels=acc[:st.n_steps, :B].tolist())
    return r, out, gu, elapsed


def relaxed_line(w, tw, dw, cat, pre, dev, steps, warmup):
    """Config-4 style decode: relaxed sampling verification (paper reading of
    Algorithm 2) at the workload's K, N and temperature, with and without tree-KV
    reuse (same lists)."""
    import numpy as np
    import torch
    from paper_2410_05165_amd.binding import Engine
    key = [int(x) for x in __import__("synth").philox_key(w)]
    prefix = torch.from_numpy(pre).to(dev)
    res = {}
    outs = []
    for reuse in (0, 1):
        eng = Engine(w, tw, dw, cat, mode={"relaxed_exact": 1, "relaxed_paper": 2}[w.mode],
                     seed=key[0] | (key[1] << 32), reuse_tree_kv=reuse)
        r, out, gu, _ = timed_decodes(eng, w, prefix, steps, warmup, roofline=not reuse)
        eng.close()
        outs.append(out)
        if gu:
            r["gate_up_tflops"] = round(gu["gflop"] / gu["ms"], 1)
        r["lists_mean"] = float(out[2].mean())
        res["reuse" if reuse else "plain"] = r
        log(f"relaxed decode ({w.name}, reuse {reuse}): {r['ms_per_decode']:.1f} ms "
            f"({r['lists_per_s']:.0f} user lists/s), {r['steps']} steps, mean lists per user {r['lists_mean']:.1f}")
    for x, y in zip(*outs):
        assert (x == y).all(), "tree-KV reuse changed the relaxed lists"
    res["workload"] = (f"{w.name}: whole decode with {w.mode} at tau={w.temperature}, B={w.batch}, "
                       f"P={w.prefix_len}, K={w.K}, N={w.N}, gamma={w.gamma}")
    return res


def target_search_line(w, tw, cat, pre, dev, steps, warmup):
    """The paper's walltime-speedup baseline: target-only constrained beam search
    (atspeed_target_search: target prefill, then one target forward and TopK per
    level; with tree-KV reuse each level forwards only its new nodes, as a
    KV-cached beam search does).  Returns its figures and lists."""
    import numpy as np
    import torch
    from paper_2410_05165_amd.binding import Engine
    B, K, L = w.batch, w.K, w.L
    prefix = torch.from_numpy(pre).to(dev)
    res, outs = {}, []
    for reuse in (1, 0):
        eng = Engine(w.with_(mode="strict"), tw, None, cat, reuse_tree_kv=reuse)
        items = torch.zeros((B, K, L), dtype=torch.int32, device=dev)
        scores = torch.zeros((B, K), dtype=torch.float32, device=dev)
        n = torch.zeros(B, dtype=torch.int32, device=dev)
        for _ in range(warmup):
            eng.atspeed_target_search(prefix, items, scores, n)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            eng.atspeed_target_search(prefix, items, scores, n)
        torch.cuda.synchronize()
        ms = 1e3 * (time.perf_counter() - t0) / steps
        eng.close()
        outs.append(items.cpu().numpy())
        res["kv_cached" if reuse else "recompute_paths"] = dict(ms_per_decode=ms, lists_per_s=B / (ms * 1e-3))
        log(f"target-only beam search ({w.name}, {'earlier levels carried' if reuse else 'paths recomputed'}): "
            f"{ms:.1f} ms per {B} lists ({B / (ms * 1e-3):.0f} lists/s)")
    assert (outs[0] == outs[1]).all()
    return res, outs[0]


def ws_by_batch(w, tw, dw, cat, pre, dev, steps, warmup, batches=(1, 4, 32), train_steps=300):
    """Walltime speedup WS (Sec. 4.1: the target-only beam search's time over the
    speculative decode's) at several batch sizes, first users of the workload:
    the KV-cached target-only search (atspeed_target_search with tree-KV reuse),
    the speculative decode with the random-init draft, and with the draft
    aligned on those users (AtSpeed-S or -R, multi-step data, alpha 0.5)."""
    import numpy as np
    import torch
    from paper_2410_05165_amd.align import AlignTrainer, cosine_lr
    from paper_2410_05165_amd.binding import Engine
    from synth import philox_key
    K, L = w.K, w.L
    strict = w.mode == "strict"
    key = [int(x) for x in philox_key(w)]
    mode = {"strict": 0, "relaxed_exact": 1, "relaxed_paper": 2}[w.mode]
    search_eng = Engine(w.with_(mode="strict"), tw, dw, cat, reuse_tree_kv=1)
    sd_eng = Engine(w, tw, dw, cat, mode=mode, seed=key[0] | (key[1] << 32))
    head0 = sd_eng.draft_dev["lm_head_item"].clone()

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            fn()
        torch.cuda.synchronize()
        return 1e3 * (time.perf_counter() - t0) / steps

    rows = []
    for B in batches:
        prefix = torch.from_numpy(np.ascontiguousarray(pre[:B])).to(dev)
        items = torch.zeros((B, K, L), dtype=torch.int32, device=dev)
        scores = torch.zeros((B, K), dtype=torch.float32, device=dev)
        n = torch.zeros(B, dtype=torch.int32, device=dev)
        si = torch.zeros((B, K * L, L), dtype=torch.int32, device=dev)
        sl = torch.zeros((B, K * L), dtype=torch.int32, device=dev)
        sn = torch.zeros(B, dtype=torch.int32, device=dev)
        ms_search = timed(lambda: search_eng.atspeed_target_search(prefix, items, scores, n))
        search_eng.atspeed_target_search(prefix, items, scores, n, si, sl, sn)
        ref = items.clone()
        sd_eng.draft_dev["lm_head_item"].copy_(head0)
        ms_sd = timed(lambda: sd_eng.atspeed_decode_topk(prefix, items, scores, n))
        if strict:
            assert torch.equal(items, ref), "speculative decode differs from the target-only search"
        sd_eng.atspeed_prefill(prefix)
        tr = AlignTrainer(sd_eng, "S" if strict else "R", alpha=0.5, lr=1e-2, weight_decay=0.01)
        tr.data(si, sn, sl)
        for s_ in range(1, train_steps + 1):
            tr.step(lr=cosine_lr(s_, train_steps, 1e-2, 20))
        ms_al = timed(lambda: sd_eng.atspeed_decode_topk(prefix, items, scores, n))
        if strict:
            assert torch.equal(items, ref), "aligned speculative decode differs from the target-only search"
        r = dict(batch=B, target_search_ms=round(ms_search, 3), sd_random_draft_ms=round(ms_sd, 3),
                 sd_aligned_in_sample_ms=round(ms_al, 3), ws_random_draft=round(ms_search / ms_sd, 3),
                 ws_aligned_in_sample=round(ms_search / ms_al, 3))
        rows.append(r)
        log(f"WS at B={B} ({w.name}): target search {ms_search:.1f} ms, SD random draft {ms_sd:.1f} ms "
            f"(WS {ms_search / ms_sd:.2f}), SD aligned in-sample {ms_al:.1f} ms (WS {ms_search / ms_al:.2f})")
    sd_eng.close()
    search_eng.close()
    return dict(rows=rows, what="WS = target-only beam search time / speculative decode time (prefill included "
                                "in both), first B users; the aligned draft is trained on those users")


def stress_line(tw, dw, dev, steps, warmup):
    """Config 5 (stress): 1M items, 128 users with 1,024-token prefixes, K 50,
    N 100, the same 7B-shaped target and draft (the same seeded weights as the
    benchmark's, passed in).  Whole decodes (natural drafts) and the target-only
    search on the same context (paths recomputed: the tree-KV reuse buffers would
    need 74 GB more at this shape)."""
    import numpy as np
    import torch
    from paper_2410_05165_amd.binding import Engine
    from synth import get_workload, make_catalog, make_prefixes
    w = get_workload("stress")
    t0 = time.time()
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    eng = Engine(w, tw, dw, cat)
    log(f"stress: {len(cat)} items, prefixes {pre.shape}, workspace {eng.ws.numel() / 2**30:.1f} GiB "
        f"({time.time() - t0:.1f}s)")
    prefix = torch.from_numpy(pre).to(dev)
    r, out, _, _ = timed_decodes(eng, w, prefix, steps, warmup, roofline=False)
    B, K, L = w.batch, w.K, w.L
    items = torch.zeros((B, K, L), dtype=torch.int32, device=dev)
    scores = torch.zeros((B, K), dtype=torch.float32, device=dev)
    n = torch.zeros(B, dtype=torch.int32, device=dev)
    eng.atspeed_target_search(prefix, items, scores, n)
    torch.cuda.synchronize()
    assert (items.cpu().numpy() == out[0]).all(), "stress: decode differs from the target-only search"
    t1 = time.perf_counter()
    for _ in range(steps):
        eng.atspeed_target_search(prefix, items, scores, n)
    torch.cuda.synchronize()
    ms_search = 1e3 * (time.perf_counter() - t1) / steps
    eng.close()
    res = {k: r[k] for k in ("lists_per_s", "ms_per_decode", "steps", "ms_prefill", "ms_draft", "ms_verify",
                             "lists_per_s_decode_only", "target_tree_rows")}
    res.update(target_search_ms=ms_search, ws=round(ms_search / r["ms_per_decode"], 3),
               workload=f"stress: B={B}, P={w.prefix_len}, K={K}, N={w.N}, {w.n_items} items, strict, natural drafts",
               lists_mean=float(out[2].mean()))
    log(f"stress decode: {r['ms_per_decode']:.0f} ms per {B} users ({r['lists_per_s']:.0f} lists/s; prefill "
        f"{r['ms_prefill']:.0f} ms, verify {r['ms_verify']:.0f} ms, {r['steps']} steps); target-only search "
        f"{ms_search:.0f} ms")
    return res


def aligned_line(w, tw, dw, cat, pre, dev, steps, warmup, ref_lists=None, train_steps=300, alpha=0.5, peak_lr=1e-2):
    """Draft alignment, then natural decodes: AtSpeed-S for strict verification,
    AtSpeed-R for relaxed, on the multi-step data of the benchmark users (the
    target's K beams of every step), alpha 0.5, AdamW with a cosine schedule.
    The decodes run the aligned draft on the same users (in-sample) and on as
    many held-out users (same catalog and prompt, their own histories)."""
    import numpy as np
    import torch
    from paper_2410_05165_amd.align import AlignTrainer, cosine_lr
    from paper_2410_05165_amd.binding import Engine
    from synth import make_prefixes, philox_key
    B, K, L = w.batch, w.K, w.L
    strict = w.mode == "strict"
    ws = w if strict else w.with_(mode="strict")
    prefix = torch.from_numpy(pre).to(dev)
    seng = Engine(ws, tw, dw, cat)
    lists = (torch.zeros((B, K, L), dtype=torch.int32, device=dev), torch.zeros((B, K), device=dev),
             torch.zeros(B, dtype=torch.int32, device=dev))
    items = torch.zeros((B, K * L, L), dtype=torch.int32, device=dev)
    lens = torch.zeros((B, K * L), dtype=torch.int32, device=dev)
    n = torch.zeros(B, dtype=torch.int32, device=dev)
    seng.atspeed_target_search(prefix, *lists, items, lens, n)
    if strict:
        eng = seng
    else:
        seng.close()
        key = [int(x) for x in philox_key(w)]
        eng = Engine(w, tw, dw, cat, mode={"relaxed_exact": 1, "relaxed_paper": 2}[w.mode],
                     seed=key[0] | (key[1] << 32))
    held = torch.from_numpy(np.ascontiguousarray(make_prefixes(w.with_(batch=2 * B), cat)[B:])).to(dev)
    before_held, _, _, _ = timed_decodes(eng, w, held, 1, 0, roofline=False)
    eng.atspeed_prefill(prefix)
    tr = AlignTrainer(eng, "S" if strict else "R", alpha=alpha, lr=peak_lr, weight_decay=0.01)
    tr.data(items, n, lens)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    losses = [tr.step(lr=cosine_lr(s, train_steps, peak_lr, 20)) for s in range(1, train_steps + 1)]
    torch.cuda.synchronize()
    ms_train = 1e3 * (time.perf_counter() - t0) / train_steps
    r_in, out_in, _, _ = timed_decodes(eng, w, prefix, steps, warmup, roofline=False)
    r_held, out_held, _, _ = timed_decodes(eng, w, held, steps, warmup, roofline=False)
    eng.close()
    if ref_lists is not None:
        assert (out_in[0] == ref_lists).all(), "the aligned draft changed the strict lists"

    def accept(r):
        a = np.array(r["accepted_levels"])
        return float(a[a >= 0].mean())
    res = dict(
        objective=f"AtSpeed-{'S' if strict else 'R'}: {alpha} L_Align + {1 - alpha} L_Rec (NLL of the training "
                  f"sequences), multi-step data ({int(n.sum().item())} sequences of the {B} users), draft item head "
                  f"trained, AdamW lr {peak_lr} cosine, {train_steps} steps",
        train=dict(ms_per_step=round(ms_train, 3), loss_first=round(losses[0], 4), loss_last=round(losses[-1], 4)),
        trained_users=dict(lists_per_s=r_in["lists_per_s"], ms_per_decode=r_in["ms_per_decode"], steps=r_in["steps"],
                           accepted_per_step=accept(r_in), lists_mean=float(out_in[2].mean())),
        held_out_users=dict(lists_per_s=r_held["lists_per_s"], ms_per_decode=r_held["ms_per_decode"],
                            steps=r_held["steps"], accepted_per_step=accept(r_held),
                            accepted_per_step_before=accept(before_held), lists_mean=float(out_held[2].mean())),
        workload=f"{w.name}: {w.mode} verification, B={B}, K={K}, N={w.N}")
    log(f"aligned draft ({w.name}, {res['objective'].split(':')[0]}): training {ms_train:.2f} ms/step; trained users "
        f"{r_in['ms_per_decode']:.1f} ms ({r_in['lists_per_s']:.0f} lists/s, {r_in['steps']} steps, accepted/step "
        f"{accept(r_in):.2f}); held-out users {r_held['ms_per_decode']:.1f} ms (accepted/step "
        f"{accept(before_held):.2f} -> {accept(r_held):.2f})")
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="b7")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="only the headline decode (profiling runs): no other profiles, verify step, probe or relaxed line")
    ap.add_argument("--only", default="",
                    help="comma list of extra sections to run: "
                         "schedule,paper_as,all_accept,verify,probe,relaxed,aligned,search,ws,stress")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one plain device copy of this size (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the verify path has no multi-GPU mode "
              f"(users shard across GPUs with no exchange); got --gpus {args.gpus}", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from synth import get_workload, make_catalog, make_prefixes, make_weights
    from paper_2410_05165_amd.binding import Engine

    sections = {"schedule", "paper_as", "all_accept", "verify", "probe", "relaxed", "aligned", "search", "ws",
                "stress"}
    if args.no_extras:
        sections = set()
    elif args.only:
        sections = set(args.only.split(","))
    w = get_workload(args.workload)
    dev = torch.device("cuda:0")
    t0 = time.time()
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    log(f"catalog {cat.shape}, prefixes {pre.shape} ({time.time() - t0:.1f}s)")
    tw = make_weights(w, "target")
    log(f"target weights {sum(a.nbytes for a in tw.values()) / 2**30:.1f} GiB ({time.time() - t0:.1f}s)")
    dw = make_weights(w, "draft")
    mode = {"strict": 0, "relaxed_exact": 1, "relaxed_paper": 2}[w.mode]
    key = [int(x) for x in __import__("synth").philox_key(w)]
    seed = key[0] | (key[1] << 32)
    eng = Engine(w, tw, dw, cat, mode=mode, seed=seed)
    log(f"engine ready, workspace {eng.ws.numel() / 2**30:.2f} GiB ({time.time() - t0:.1f}s)")
    prefix = torch.from_numpy(pre).to(dev)
    B, K, L = w.batch, w.K, w.L
    m = w.target

    # ---- headline: whole decode (prefill + draft/verify steps until every list is complete)
    head, out0, gu, elapsed = timed_decodes(eng, w, prefix, args.steps, args.warmup)
    value = head["lists_per_s"]
    log(f"decode ({w.mode}, natural drafts): {head['ms_per_decode']:.1f} ms per decode (median "
        f"{head['ms_per_decode_median']:.1f}) -> {value:.1f} lists/s; {head['steps']} steps")
    gu_avg_ms = gu["ms"] / gu["launches"]
    gu_flop = gu["gflop"] * 1e9 / gu["launches"]
    gu_tflops = gu["gflop"] / gu["ms"]
    log(f"roofline: target gate/up GEMM, {gu['launches']} launches in the timed region, {1e3 * gu_avg_ms:.1f} us and "
        f"{gu_flop / 1e9:.1f} GFLOP per launch on average -> {gu_tflops:.0f} TFLOP/s")
    roofline = dict(bound="mfma", kernel="target gate/up GEMM (SiLU*up epilogue), every launch of the timed decodes "
                                         "(prefill and each verify step)",
                    achieved=round(gu_tflops, 2), peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                    frac=round(gu_tflops / PEAK_BF16_TFLOPS, 4),
                    traffic=gemm_traffic("gate/up GEMM, natural decode", w.name),
                    per_launch_flops=round(gu_flop), avg_launch_ms=round(gu_avg_ms, 5),
                    launches_timed=gu["launches"])

    extras = {}
    levels = kids = None
    if mode == 0 and sections & {"paper_as", "all_accept", "verify", "probe"}:
        kids = catalog_children(cat)
        levels = gpu_target_beam_search(eng, w, prefix, upload_tree)
        assert (levels[-1][2] == out0[0]).all(), "speculative decode differs from the GPU's target beam search"

    if mode == 0 and "schedule" in sections:
        for start, reuse, name in ((1, 0, "decode_level1_start"), (0, 1, "decode_reuse"),
                                   (1, 1, "decode_level1_start_reuse")):
            e2 = Engine(w, tw, dw, cat, mode=mode, seed=seed, sd_start_level=start, reuse_tree_kv=reuse)
            r, out, _, _ = timed_decodes(e2, w, prefix, args.steps, args.warmup, roofline=False)
            e2.close()
            for x, y in zip(out0, out):
                assert (x == y).all(), f"{name} changed the lists"
            extras[name] = r
            log(f"{name}: {r['ms_per_decode']:.1f} ms ({r['lists_per_s']:.0f} lists/s), target rows "
                f"{r['target_tree_rows']}")

    if mode == 0 and "paper_as" in sections:
        r = decode_replay_as(eng, w, prefix, levels, kids, reps=args.steps)
        extras["decode_paper_as"] = r
        log(f"decode, replay-paper-AS: {r['ms_per_decode']:.1f} ms ({r['lists_per_s']:.0f} lists/s), "
            f"{r['steps']} steps, accepted levels per step {r['accepted_mean']:.2f}")

    trees = replay_all_accept_tree(eng, kids, w, levels) if levels is not None else None
    if mode == 0 and "all_accept" in sections:
        # whole decode under replay-all-accept: prefill, the device draft, then its
        # tree replaced by the replay tree -- one verify completes every list
        n_, tok_, par_, dep_ = (torch.from_numpy(a).to(dev) for a in tree_arrays(eng, trees, B))
        tn, tt, tp, td, tq = eng.tree_tensors(B)
        acc = torch.zeros(B, dtype=torch.int32, device=dev)

        def decode_all():
            eng.atspeed_prefill(prefix)
            eng.atspeed_draft()
            tn.copy_(n_); tt.copy_(tok_); tp.copy_(par_); td.copy_(dep_); tq.zero_()
            eng.atspeed_verify(acc)
        decode_all()
        assert (acc.cpu().numpy() == L).all() and (eng.atspeed_get_state(B)[2] == levels[-1][2]).all()
        for _ in range(args.warmup):
            decode_all()
        torch.cuda.synchronize()
        a = time.perf_counter()
        for _ in range(args.steps):
            decode_all()
        torch.cuda.synchronize()
        ms = 1e3 * (time.perf_counter() - a) / args.steps
        extras["decode_all_accept"] = dict(lists_per_s=B / (ms * 1e-3), ms_per_decode=ms, steps=1,
                                           profile="replay-all-accept (the drafted tree holds the target's TopK at "
                                                   "every level; one verify completes the lists)")
        log(f"decode, replay-all-accept: {ms:.1f} ms ({B / (ms * 1e-3):.0f} lists/s)")

    if mode == 0 and "verify" in sections:
        # the t = 0 verify step alone over the replay-all-accept tree (fixed shape)
        eng.atspeed_prefill(prefix)
        upload_tree(eng, trees, B)
        M = sum(sum(1 for p in t if len(p) < L) for t in trees)
        root_state = (np.zeros(B, np.int32), np.ones(B, np.int32), np.zeros((B, K, L), np.int32),
                      np.zeros((B, K), np.float32))
        acc = torch.zeros(B, dtype=torch.int32, device=dev)

        def vstep():
            eng.atspeed_set_state(*root_state)
            eng.atspeed_verify(acc)
        vstep()
        assert (acc.cpu().numpy() == L).all() and (eng.atspeed_get_state(B)[2] == levels[-1][2]).all()
        for _ in range(args.warmup):
            vstep()
        eng.atspeed_set_timing(["gu"])
        torch.cuda.synchronize()
        a = time.perf_counter()
        for _ in range(args.steps):
            vstep()
        torch.cuda.synchronize()
        ms_step = 1e3 * (time.perf_counter() - a) / args.steps
        vgu = eng.atspeed_get_timing()["gu"]
        steps_kt = max(3, args.steps // 2)
        eng.atspeed_set_timing(True)                 # breakdown: every launch bracketed (a separate pass)
        for _ in range(steps_kt):
            vstep()
        kt = eng.atspeed_get_timing()
        eng.atspeed_set_timing(False)
        d, f, P, nl = m.d_model, m.d_ffn, w.prefix_len, m.n_layers
        classes = {}
        for k_, (ms_, nlaunch, gf) in kt.items():
            if nlaunch == 0:
                continue
            avg = ms_ / nlaunch
            ent = dict(ms_per_step=ms_ / steps_kt, launches_per_step=nlaunch / steps_kt, avg_launch_ms=avg)
            if gf:
                ent["tflops"] = gf / ms_
                ent["mfma_frac"] = ent["tflops"] / PEAK_BF16_TFLOPS
            if k_ == "attention":
                kv = B * P * 2 * d * 2                  # prefix K and V of every user, read once
                tree = M * d * 2 * 4                    # q, tree k/v and output rows (bf16)
                ent["gbs"] = (kv + tree) / (avg * 1e-3) / 1e9
                ent["hbm_frac"] = ent["gbs"] / PEAK_HBM_GBS
            classes[k_] = ent
        gemm_ms = sum(kt[k_][0] for k_ in ("qkv", "o", "gu", "down", "lm_head")) / steps_kt
        gemm_gf = sum(kt[k_][2] for k_ in ("qkv", "o", "gu", "down", "lm_head")) / steps_kt
        extras["verify_step"] = dict(
            what=f"one atspeed_verify at t=0 over the replay-all-accept tree ({M} target rows), "
                 f"completing all {B} lists", ms_per_step=round(ms_step, 3), lists_per_s=B / (ms_step * 1e-3),
            gate_up=dict(tflops=round(vgu[2] / vgu[0], 1), mfma_frac=round(vgu[2] / vgu[0] / PEAK_BF16_TFLOPS, 4),
                         avg_launch_ms=round(vgu[0] / vgu[1], 5), traffic=gemm_traffic("gate/up GEMM", w.name)),
            gemm=dict(tflops=gemm_gf / gemm_ms, mfma_frac=gemm_gf / gemm_ms / PEAK_BF16_TFLOPS, ms_per_step=gemm_ms),
            kernels=classes)
        log(f"verify step (t=0, all-accept tree, {M} rows): {ms_step:.2f} ms; GEMMs "
            f"{gemm_gf / gemm_ms:.0f} TFLOP/s; gate/up {vgu[2] / vgu[0]:.0f} TFLOP/s")

    if mode == 0 and "probe" in sections:
        extras["decode_bound"] = decode_bound_probe(eng, w, prefix, levels, max(3, args.steps // 2))
        extras["decode_bound_one_user"] = decode_bound_probe(eng, w, prefix, levels, max(3, args.steps // 2), users=1)

    eng.close()

    def ws(search, ms):
        # walltime speedup over the KV-cached target-only beam search
        return round(search["kv_cached"]["ms_per_decode"] / ms, 3)
    search = None
    if "search" in sections:
        search, search_lists = target_search_line(w, tw, cat, pre, dev, args.steps, args.warmup)
        if mode == 0:
            assert (search_lists == out0[0]).all(), "target-only beam search differs from the speculative decode"
        search["ws_headline_decode"] = ws(search, head["ms_per_decode"])
        for k_ in ("decode_level1_start", "decode_reuse", "decode_level1_start_reuse", "decode_paper_as",
                   "decode_all_accept"):
            if k_ in extras:
                search[f"ws_{k_}"] = ws(search, extras[k_]["ms_per_decode"])
        extras["target_search"] = search
    if "aligned" in sections:
        al = aligned_line(w, tw, dw, cat, pre, dev, args.steps, args.warmup, ref_lists=out0[0] if mode == 0 else None)
        if search is not None:
            for k_ in ("trained_users", "held_out_users"):
                al[k_]["ws"] = ws(search, al[k_]["ms_per_decode"])
        extras["decode_aligned"] = al
    if "ws" in sections:
        extras["ws_by_batch"] = ws_by_batch(w, tw, dw, cat, pre, dev, args.steps, args.warmup)
    if "relaxed" in sections and w.name == "b7":
        wr = get_workload("b7_relaxed")
        extras["relaxed_decode"] = rl = relaxed_line(wr, tw, dw, cat, pre, dev, args.steps, args.warmup)
        rsearch = None
        if "search" in sections:
            rsearch, _ = target_search_line(wr, tw, cat, pre, dev, args.steps, args.warmup)
            for k_ in ("plain", "reuse"):
                rsearch[f"ws_relaxed_{k_}"] = ws(rsearch, rl[k_]["ms_per_decode"])
            extras["target_search_k20"] = rsearch
        if "aligned" in sections:
            al = aligned_line(wr, tw, dw, cat, pre, dev, args.steps, args.warmup)
            if rsearch is not None:
                for k_ in ("trained_users", "held_out_users"):
                    al[k_]["ws"] = ws(rsearch, al[k_]["ms_per_decode"])
            extras["relaxed_decode_aligned"] = al
    elif mode != 0 and "relaxed" in sections:
        extras["relaxed_decode"] = relaxed_line(w, tw, dw, cat, pre, dev, args.steps, args.warmup)

    if "stress" in sections and w.name == "b7":
        extras["stress_decode"] = stress_line(tw, dw, dev, max(2, min(args.steps, 3)), 1)

    cpu = None
    if not args.no_cpu_baseline and mode == 0:
        cpu = cpu_baseline(w, tw, dw, pre, cat, out0[0][0, :out0[2][0]])
        log(f"cpu baseline: {cpu['value']:.4f} lists/s ({cpu['sample']})")

    if args.copy_calibration_mib:
        x = torch.empty(args.copy_calibration_mib * 2**20 // 4, dtype=torch.float32, device=dev).fill_(1.0)
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        y.copy_(x)
        torch.cuda.synchronize()
        log(f"copy calibration: {args.copy_calibration_mib} MiB read + write")

    prof = {0: "natural drafts (random-init draft: the library's own draft and verify, no forced trees)"}
    out = {
        "metric": "top-K lists/sec/GPU at 7B shape K=10; verify-step MFMA util + HBM GB/s",
        "value": round(value, 2), "unit": "lists/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(1e3 * elapsed / args.steps, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded catalog, Zipf histories, random-init N(0,0.02) weights)",
        "config": {"workload": f"{w.name}: whole atspeed_decode_topk including prefill, {w.mode} verification, "
                               f"acceptance profile {prof.get(mode, 'sampled drafts')}; target {m.n_layers}L/"
                               f"{m.d_model}/{m.n_heads}h/FFN {m.d_ffn}, V {m.vocab} ({w.n_item_tokens} item tokens), "
                               f"4L/768 draft, {w.n_items} items, B={B} users, P={w.prefix_len}, K={K}, N={w.N}, "
                               f"gamma={w.gamma}",
                   "global_batch": B, "seq_len": w.prefix_len, "parallelism": "none (1 GPU)"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "decode": head,
    }
    out.update(extras)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
