#!/usr/bin/env python3
"""Throughput of the AtSpeed verify step on one MI355X.

Workload (default): the LLaMA-7B-shaped target (32 layers, d 4096, 32 heads,
FFN 11008, vocabulary 33,024 with 1,024 item tokens), 4-layer draft, 100,000
random 4-token items, 32 users with 144-token prefixes, K = 10, N = 20,
gamma = 4, strict verification; random-init bf16 weights N(0, 0.02).

A step is one ``atspeed_verify`` over the batch: tree planning, one target
forward over the t = 0 tree (drafted depths 1..3 forwarded, 60 nodes per user),
item log-softmax, cumulative log-probs, trie-constrained TopK and strict
acceptance.  The tree is the replay-all-accept tree (every drafted level holds
the target's TopK, padded to N with other valid extensions), so each step
completes the top-K lists of all users: value = users x steps / time.  Random
weights make natural acceptance ~0, so the end-to-end decode (prefill + draft +
verify until complete, natural acceptance) is reported beside it.

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


def cpu_baseline(w, tw, pre, cat, tree_paths):
    """The oracle's verify step for one user of the same workload (fp64, per-path forwards)."""
    import numpy as np
    from oracle.model import Decoder
    from oracle.search import model_scorer, verify_strict
    from oracle.trie import Trie
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    trie = Trie(cat)
    dec = Decoder(w.target, tw, w.dtype, cache_f64=False)
    log("cpu baseline: oracle prefill of user 0 (untimed set-up)")
    cache = dec.prefill(pre[0])
    lp = model_scorer(dec, cache, w.target.item_base, w.codebook)
    D = [[p for p in tree_paths if len(p) == d] for d in range(1, w.L + 1)]
    fwd = [p for lvl in D[:-1] for p in lvl]
    log("cpu baseline: oracle verify of user 0 (timed)")
    t0 = time.perf_counter()
    lp(fwd)                        # logits of every forwarded tree node (one causal forward per path)
    res = verify_strict(lp, trie, [((), 0.0)], D, w.K, w.L, w.codebook)
    dt = time.perf_counter() - t0
    return dict(value=1.0 / dt, unit="lists/s", cores=int(threads), kind="oracle",
                sample=f"verify step of 1 of {w.batch} users (t=0 replay tree, {len(fwd)} forwarded nodes: "
                       f"per-path fp64 forwards of all of them + Algorithm 1), {dt:.1f} s; "
                       f"accepted={res.accepted}, host cpus={os.cpu_count()}"), res


def decode_bound_probe(eng, w, prefix, levels, steps):
    """Target-only beam step at t = 1 (the K beams of every user forwarded, K*B
    rows): the weights and the prefix KV cache stream once per step with little
    arithmetic per byte, so it is HBM-bound; reports its algorithmic bytes/s."""
    import torch
    B, K, L = w.batch, w.K, w.L
    eng.atspeed_prefill(prefix)
    t1, nb1, p1, s1 = levels[0]
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
    log(f"decode-bound probe: {rows} rows, {ms:.2f} ms/step, {gbs:.0f} GB/s ({gbs / PEAK_HBM_GBS:.1%} of HBM)")
    return dict(rows=rows, ms_per_step=round(ms, 3), bytes=weights + kv, gbs=round(gbs, 1),
                hbm_frac=round(gbs / PEAK_HBM_GBS, 4),
                what="target-only beam step at t=1: target weights + prefix KV read once per step")


def bench_decode(args, w, eng, pre, dev, make_engine=None):
    """Relaxed workloads: a step is one whole decode (prefill, sampled drafting and
    relaxed verification until every user holds L-token items); the replay-tree
    step of the strict workload does not apply (relaxed verification consumes
    the context's own sampled draft)."""
    import numpy as np
    import torch
    from paper_2410_05165_amd.binding import Stats
    B, K, L = w.batch, w.K, w.L
    prefix = torch.from_numpy(pre).to(dev)
    items = torch.zeros((B, K, L), dtype=torch.int32, device=dev)
    scores = torch.zeros((B, K), dtype=torch.float32, device=dev)
    n = torch.zeros(B, dtype=torch.int32, device=dev)
    for _ in range(args.warmup):
        eng.atspeed_decode_topk(prefix, items, scores, n, None)
    torch.cuda.synchronize()
    acc = np.zeros((L, B), np.int32)
    st = Stats()
    import ctypes as C
    st.accepted = acc.ctypes.data_as(C.POINTER(C.c_int32))
    a = time.perf_counter()
    for _ in range(args.steps):
        eng.atspeed_decode_topk(prefix, items, scores, n, st)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - a
    # breakdown by kernel class: a separate pass with every launch bracketed
    steps_kt = max(1, args.steps // 2)
    eng.atspeed_set_timing(True)
    for _ in range(steps_kt):
        eng.atspeed_decode_topk(prefix, items, scores, n, None)
    kt = eng.atspeed_get_timing()
    eng.atspeed_set_timing(False)
    value = B * args.steps / elapsed
    log(f"decode {1e3 * elapsed / args.steps:.1f} ms -> {value:.0f} lists/s; last decode steps {st.n_steps}")
    # the same decode with tree-KV reuse across its verify steps (same lists)
    reuse = None
    if make_engine is not None:
        out0 = (items.cpu().numpy(), scores.cpu().numpy(), n.cpu().numpy())
        eng_r = make_engine(reuse_tree_kv=1)
        st_r = Stats()
        for _ in range(args.warmup):
            eng_r.atspeed_decode_topk(prefix, items, scores, n, None)
        torch.cuda.synchronize()
        a = time.perf_counter()
        for _ in range(args.steps):
            eng_r.atspeed_decode_topk(prefix, items, scores, n, st_r)
        torch.cuda.synchronize()
        el_r = time.perf_counter() - a
        eng_r.close()
        for x, y in zip(out0, (items.cpu().numpy(), scores.cpu().numpy(), n.cpu().numpy())):
            assert (x == y).all(), "tree-KV reuse changed the relaxed lists"
        reuse = dict(ms_per_decode=1e3 * el_r / args.steps, lists_per_s=B * args.steps / el_r,
                     target_tree_rows=int(st_r.rows_target), target_tree_rows_without_reuse=int(st.rows_target))
        log(f"decode with tree-KV reuse {reuse['ms_per_decode']:.1f} ms, target rows "
            f"{st.rows_target} -> {st_r.rows_target}")
    # Roofline of the dominant kernel at one fixed shape: the t = 0 verify step
    # (the context's own sampled draft), gate/up launches bracketed by events.
    gu_ms, gu_n, rows = 0.0, 0, 0
    for _ in range(max(3, args.steps)):
        eng.atspeed_prefill(prefix)
        eng.atspeed_draft()
        tn, _, _, td, _ = eng.tree_tensors(B)
        nn, dd = tn.cpu().numpy(), td.cpu().numpy()
        rows = int(sum(int((dd[u, :nn[u]] < L).sum()) for u in range(B)))   # forwarded: depth < L
        eng.atspeed_set_timing(["gu"])
        eng.atspeed_verify()
        g = eng.atspeed_get_timing()["gu"]
        eng.atspeed_set_timing(False)
        gu_ms += g[0]
        gu_n += g[1]
    m = w.target
    gu_flops = 2.0 * rows * m.d_model * 2 * m.d_ffn
    gu_avg = gu_ms / gu_n
    gu_tflops = gu_flops / (gu_avg * 1e-3) / 1e12
    log(f"t=0 verify: {rows} rows, gate/up {1e3 * gu_avg:.1f} us per launch, {gu_tflops:.0f} TFLOP/s")
    out = {"metric": "top-K lists/sec/GPU (relaxed sampling verification, whole decode)", "value": round(value, 2),
           "unit": "lists/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(1e3 * elapsed / args.steps, 3), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": f"{w.name}: whole decode with {w.mode}, B={B}, P={w.prefix_len}, K={K}, N={w.N}, "
                                  f"gamma={w.gamma}, tau={w.temperature}", "global_batch": B, "seq_len": w.prefix_len,
                      "parallelism": "none (1 GPU)"},
           "roofline": dict(bound="mfma", kernel=f"gemm_bf16 gate/up at the t=0 verify step ({rows} rows)",
                            achieved=round(gu_tflops, 2), peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                            frac=round(gu_tflops / PEAK_BF16_TFLOPS, 4), traffic=None,
                            per_launch_flops=gu_flops, avg_launch_ms=round(gu_avg, 4), launches_timed=int(gu_n)),
           "cpu_baseline": None,
           "kernels": {k: dict(ms_per_step=v[0] / steps_kt, launches_per_step=v[1] / steps_kt)
                       for k, v in kt.items() if v[1]},
           "accepted_levels_last_decode": acc[:st.n_steps].tolist(),
           "decode_reuse": reuse}
    print(json.dumps(out), flush=True)
    eng.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="b7")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-e2e", action="store_true")
    ap.add_argument("--no-probe", action="store_true", help="skip the decode-bound probe (profiling runs)")
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
    from paper_2410_05165_amd.binding import Engine, Stats

    w = get_workload(args.workload)
    dev = torch.device("cuda:0")
    t0 = time.time()
    cat = make_catalog(w)
    pre = make_prefixes(w, cat)
    log(f"catalog {cat.shape}, prefixes {pre.shape} ({time.time() - t0:.1f}s)")
    tw = make_weights(w, "target")
    log(f"target weights {sum(a.nbytes for a in tw.values()) / 2**30:.1f} GiB ({time.time() - t0:.1f}s)")
    dw = make_weights(w, "draft")
    relaxed = w.mode != "strict"
    mode = {"strict": 0, "relaxed_exact": 1, "relaxed_paper": 2}[w.mode]
    key = [int(x) for x in __import__("synth").philox_key(w)]
    eng = Engine(w, tw, dw, cat, mode=mode, seed=key[0] | (key[1] << 32))
    log(f"engine ready, workspace {eng.ws.numel() / 2**30:.2f} GiB ({time.time() - t0:.1f}s)")
    if relaxed:
        return bench_decode(args, w, eng, pre, dev,
                            make_engine=lambda **kw: Engine(w, tw, dw, cat, mode=mode, seed=key[0] | (key[1] << 32),
                                                            **kw))
    kids = catalog_children(cat)
    prefix = torch.from_numpy(pre).to(dev)
    B, K, L = w.batch, w.K, w.L

    # ---- end-to-end decode (natural acceptance)
    def e2e_natural(engine, label):
        items = torch.zeros((B, K, L), dtype=torch.int32, device=dev)
        scores = torch.zeros((B, K), dtype=torch.float32, device=dev)
        n = torch.zeros(B, dtype=torch.int32, device=dev)
        st = Stats()
        for _ in range(3):                      # warm-up decodes
            engine.atspeed_decode_topk(prefix, items, scores, n, None)
        torch.cuda.synchronize()
        reps, tt = 20, []                       # median of 20 timed decodes
        for _ in range(reps):
            torch.cuda.synchronize()
            a = time.perf_counter()
            engine.atspeed_decode_topk(prefix, items, scores, n, st)
            torch.cuda.synchronize()
            tt.append(time.perf_counter() - a)
        r = dict(lists_per_s=B / float(np.median(tt)), ms_per_decode=1e3 * float(np.median(tt)),
                 steps=int(st.n_steps), ms_prefill=st.ms_prefill, ms_draft=st.ms_draft, ms_verify=st.ms_verify,
                 lists_per_s_decode_only=B / ((st.ms_draft + st.ms_verify) / 1e3),
                 target_tree_rows=int(st.rows_target), profile=label)
        log(f"e2e decode ({label}): {r['ms_per_decode']:.1f} ms ({r['lists_per_s']:.0f} lists/s), steps {st.n_steps}")
        return r, (items.cpu().numpy(), scores.cpu().numpy(), n.cpu().numpy())

    e2e = e2e_l1 = e2e_reuse = e2e_l1_reuse = None
    if not args.no_e2e:
        e2e, out0 = e2e_natural(eng, "natural")
        # the level-1 start: level 1 from the prefill, speculation from t = 1
        eng1 = Engine(w, tw, dw, cat, mode=mode, seed=key[0] | (key[1] << 32), sd_start_level=1)
        e2e_l1, out1 = e2e_natural(eng1, "natural, level-1 start")
        eng1.close()
        for x, y in zip(out0, out1):
            assert (x == y).all(), "level-1 start changed the lists"
        # tree-KV reuse across the verify steps, from t = 0 and from level 1
        for start in (0, 1):
            eng2 = Engine(w, tw, dw, cat, mode=mode, seed=key[0] | (key[1] << 32), sd_start_level=start,
                          reuse_tree_kv=1)
            r2, out2 = e2e_natural(eng2, "natural, tree-KV reuse" + (", level-1 start" if start else ""))
            eng2.close()
            for x, y in zip(out0, out2):
                assert (x == y).all(), "tree-KV reuse changed the lists"
            if start:
                e2e_l1_reuse = r2
            else:
                e2e_reuse = r2

    # ---- replay-all-accept tree from the GPU's own target beam search
    levels = gpu_target_beam_search(eng, w, prefix, upload_tree)
    e2e_as = None
    if not args.no_e2e:
        e2e_as = decode_replay_as(eng, w, prefix, levels, kids, reps=20)
        log(f"e2e decode, replay-paper-AS: {e2e_as['ms_per_decode']:.1f} ms ({e2e_as['lists_per_s']:.0f} lists/s), "
            f"{e2e_as['steps']} steps, accepted levels per step {e2e_as['accepted_mean']:.2f} "
            f"(first step {e2e_as['accepted_first_step_mean']:.2f})")
    trees = replay_all_accept_tree(eng, kids, w, levels)
    final = levels[-1]
    eng.atspeed_prefill(prefix)
    upload_tree(eng, trees, B)
    n_fwd = sum(sum(1 for p in t if len(p) < L) for t in trees)
    root_state = (np.zeros(B, np.int32), np.ones(B, np.int32), np.zeros((B, K, L), np.int32),
                  np.zeros((B, K), np.float32))
    acc = torch.zeros(B, dtype=torch.int32, device=dev)
    tafter = torch.zeros(B, dtype=torch.int32, device=dev)

    def step():
        eng.atspeed_set_state(*root_state)
        eng.atspeed_verify(acc, tafter)

    step()
    t_, nb_, paths_, sc_ = eng.atspeed_get_state(B)
    assert (acc.cpu().numpy() == L).all() and (t_ == L).all(), "replay tree is not all-accept"
    assert (paths_ == final[2]).all() and (sc_ == final[3]).all(), "verify differs from target beam search"
    log(f"replay tree: {n_fwd} forwarded nodes ({n_fwd // B}/user), all levels accepted")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Timed region: HIP events bracket only the gate/up launches (the roofline
    # kernel), since every event adds stream time.
    eng.atspeed_set_timing(["gu"])
    torch.cuda.synchronize()
    a = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - a
    kt_gu = eng.atspeed_get_timing()["gu"]
    eng.atspeed_set_timing(False)
    ms_step = 1e3 * elapsed / args.steps
    value = B * args.steps / elapsed
    log(f"verify step {ms_step:.2f} ms -> {value:.0f} lists/s")
    # Breakdown by kernel class: a separate pass with every launch bracketed.
    steps_kt = max(3, args.steps // 2)
    eng.atspeed_set_timing(True)
    for _ in range(steps_kt):
        step()
    kt = eng.atspeed_get_timing()
    eng.atspeed_set_timing(False)

    # ---- roofline of the dominant kernel (gate/up GEMM) and of the other classes
    M, d, f, H = n_fwd, w.target.d_model, w.target.d_ffn, w.target.n_heads
    P, nl = w.prefix_len, w.target.n_layers
    flops = {"qkv": 2 * M * d * 3 * d, "o": 2 * M * d * d, "gu": 2 * M * d * 2 * f, "down": 2 * M * f * d,
             "lm_head": 2 * M * d * w.n_item_tokens}
    classes = {}
    for k, (ms, nlaunch) in kt.items():
        if nlaunch == 0:
            continue
        avg = ms / nlaunch
        ent = dict(ms_per_step=ms / steps_kt, launches_per_step=nlaunch / steps_kt, avg_launch_ms=avg)
        if k in flops:
            ent["tflops"] = flops[k] / (avg * 1e-3) / 1e12
            ent["mfma_frac"] = ent["tflops"] / PEAK_BF16_TFLOPS
        if k == "attention":
            kv = B * P * 2 * d * 2                      # prefix K and V of every user, read once
            tree = M * d * 2 * 4                        # q, tree k/v and output rows (bf16)
            ent["gbs"] = (kv + tree) / (avg * 1e-3) / 1e9
            ent["hbm_frac"] = ent["gbs"] / PEAK_HBM_GBS
        classes[k] = ent
    gemm_ms = sum(kt[k][0] for k in flops) / steps_kt
    gemm_flops = nl * sum(flops[k] for k in ("qkv", "o", "gu", "down")) + flops["lm_head"]
    gu_avg = kt_gu[0] / kt_gu[1]                        # ms per gate/up launch in the timed region
    gu_tflops = flops["gu"] / (gu_avg * 1e-3) / 1e12
    roofline = dict(bound="mfma", kernel="gemm_bf16 gate/up (SiLU*up epilogue)",
                    achieved=round(gu_tflops, 2), peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                    frac=round(gu_tflops / PEAK_BF16_TFLOPS, 4), traffic=gemm_traffic("gate/up GEMM", w.name),
                    per_launch_flops=flops["gu"], avg_launch_ms=round(gu_avg, 4),
                    launches_timed=int(kt_gu[1]))

    probe = None if args.no_probe else decode_bound_probe(eng, w, prefix, levels, max(3, args.steps // 2))

    cpu = None
    if not args.no_cpu_baseline:
        cpu, _ = cpu_baseline(w, tw, pre, cat, trees[0])
        log(f"cpu baseline: {cpu['value']:.4f} lists/s ({cpu['sample']})")

    if args.copy_calibration_mib:
        x = torch.empty(args.copy_calibration_mib * 2**20 // 4, dtype=torch.float32, device=dev).fill_(1.0)
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        y.copy_(x)
        torch.cuda.synchronize()
        log(f"copy calibration: {args.copy_calibration_mib} MiB read + write")

    out = {
        "metric": "top-K lists/sec/GPU at 7B shape K=10; verify-step MFMA util + HBM GB/s",
        "value": round(value, 2), "unit": "lists/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded catalog, Zipf histories, random-init N(0,0.02) weights)",
        "config": {"workload": f"{w.name}: verify step at t=0 over the replay-all-accept tree; target 32L/4096/32h/"
                               f"FFN 11008, V 33024 (1024 item tokens), B={B} users, P={P}, K={K}, N={w.N}, "
                               f"gamma={w.gamma}, strict; {M} tree rows; prefill and drafting excluded",
                   "global_batch": B, "seq_len": P, "parallelism": "none (1 GPU)"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels": classes,            # separate pass, every launch bracketed by events
        "verify_gemm": dict(tflops=gemm_flops / (gemm_ms * 1e-3) / 1e12,
                            mfma_frac=gemm_flops / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                            ms_per_step=gemm_ms),
        "e2e_decode": e2e,
        "e2e_decode_level1_start": e2e_l1,
        "e2e_decode_paper_as": e2e_as,
        "e2e_decode_reuse": e2e_reuse,
        "e2e_decode_level1_start_reuse": e2e_l1_reuse,
        "decode_bound": probe,
    }
    print(json.dumps(out), flush=True)
    eng.close()


if __name__ == "__main__":
    main()
