"""ctypes binding of ``libatspeed.so`` (include/atspeed.h), same call names.

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  PyTorch provides device memory (weights, workspace, inputs, outputs)
and the stream.  Importing this module raises if the library is not built.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libatspeed.so")

STRICT, RELAXED_EXACT, RELAXED_PAPER = 0, 1, 2
FP32, BF16 = 0, 1
STATUS = {0: "OK", 1: "E_INVALID", 2: "E_SHAPE", 3: "E_WORKSPACE", 4: "E_DEVICE", 5: "E_STATE"}
LAYER_ORDER = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")
SYMBOLS = ("atspeed_workspace_bytes", "atspeed_create", "atspeed_destroy", "atspeed_last_error",
           "atspeed_prefill", "atspeed_draft", "atspeed_get_tree", "atspeed_verify", "atspeed_tree_logits",
           "atspeed_capture_hidden",
           "atspeed_accept", "atspeed_accept_noalloc", "atspeed_decode_topk", "atspeed_logprobs", "atspeed_get_state", "atspeed_set_state",
           "atspeed_set_timing", "atspeed_get_timing", "atspeed_align_data", "atspeed_align_step",
           "atspeed_target_search", "atspeed_mixed_search")
KERNEL_CLASSES = ("qkv", "o", "gu", "down", "lm_head", "attention", "row", "select")


class Dims(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("d_ffn", C.c_int32), ("vocab", C.c_int32), ("item_base", C.c_int32)]


class Config(C.Structure):
    _fields_ = [("target", Dims), ("draft", Dims), ("L", C.c_int32), ("codebook", C.c_int32),
                ("K", C.c_int32), ("N", C.c_int32), ("gamma", C.c_int32), ("max_batch", C.c_int32),
                ("max_prefix", C.c_int32), ("mode", C.c_int32), ("temperature", C.c_float),
                ("seed", C.c_uint64), ("dtype", C.c_int32), ("sd_start_level", C.c_int32),
                ("reuse_tree_kv", C.c_int32), ("stream", C.c_void_p)]


class Weights(C.Structure):
    _fields_ = [("tok_emb", C.c_void_p), ("layers", C.POINTER(C.c_void_p)),
                ("final_norm", C.c_void_p), ("lm_head_item", C.c_void_p)]


class Catalog(C.Structure):
    _fields_ = [("n_items", C.c_int32), ("codes", C.POINTER(C.c_int32))]


class Tree(C.Structure):
    _fields_ = [("max_nodes", C.c_int32), ("n_nodes", C.c_void_p), ("token", C.c_void_p),
                ("parent", C.c_void_p), ("depth", C.c_void_p), ("q_score", C.c_void_p)]


class Stats(C.Structure):
    _fields_ = [("n_steps", C.c_int32), ("accepted", C.POINTER(C.c_int32)), ("t_after", C.POINTER(C.c_int32)),
                ("ms_prefill", C.c_double), ("ms_draft", C.c_double), ("ms_verify", C.c_double),
                ("rows_target", C.c_int64)]


class KernelTimes(C.Structure):
    _fields_ = [("ms", C.c_double * 8), ("launches", C.c_int64 * 8), ("gflop", C.c_double * 8)]


TIME_TARGET_ONLY = 1 << 16


class AlignArgs(C.Structure):
    _fields_ = [("mode", C.c_int32), ("alpha", C.c_float), ("ctx_weight", C.c_void_p), ("label_weight", C.c_void_p),
                ("root_weight", C.c_void_p), ("log_pK", C.c_void_p), ("lp_target", C.c_void_p),
                ("root_target", C.c_void_p), ("master", C.c_void_p), ("adam_m", C.c_void_p), ("adam_v", C.c_void_p),
                ("grad", C.c_void_p), ("hidden_out", C.c_void_p), ("lr", C.c_float), ("beta1", C.c_float),
                ("beta2", C.c_float), ("eps", C.c_float), ("weight_decay", C.c_float), ("step", C.c_int32)]


class AtspeedError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


def load_library(path: str = LIB_PATH) -> C.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built (run __graft_entry__.build())")
    lib = C.CDLL(path)
    vp, i32, pi32, pf = C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p
    lib.atspeed_workspace_bytes.argtypes = [C.POINTER(Config), C.POINTER(Catalog), C.POINTER(C.c_size_t)]
    lib.atspeed_create.argtypes = [C.POINTER(Config), C.POINTER(Weights), C.POINTER(Weights), C.POINTER(Catalog),
                                   vp, C.c_size_t, C.POINTER(vp)]
    lib.atspeed_destroy.argtypes = [vp]
    lib.atspeed_destroy.restype = None
    lib.atspeed_last_error.restype = C.c_char_p
    lib.atspeed_prefill.argtypes = [vp, i32, i32, pi32, pf]
    lib.atspeed_draft.argtypes = [vp]
    lib.atspeed_get_tree.argtypes = [vp, C.POINTER(Tree)]
    lib.atspeed_verify.argtypes = [vp, pi32, pi32, pf]
    lib.atspeed_tree_logits.argtypes = [vp, pf]
    lib.atspeed_capture_hidden.argtypes = [vp, i32, i32, pf, vp, pi32, i32]
    lib.atspeed_accept.argtypes = [vp, pf, pf, pi32, pi32]
    lib.atspeed_accept_noalloc.argtypes = [vp, pf, pf, pi32, pi32]
    lib.atspeed_decode_topk.argtypes = [vp, i32, i32, pi32, pi32, pf, pi32, C.POINTER(Stats)]
    lib.atspeed_logprobs.argtypes = [vp, i32, pf, pf]
    lib.atspeed_get_state.argtypes = [vp, i32, C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                      C.POINTER(C.c_float)]
    lib.atspeed_set_state.argtypes = [vp, i32, C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                      C.POINTER(C.c_float)]
    lib.atspeed_set_timing.argtypes = [vp, i32]
    lib.atspeed_get_timing.argtypes = [vp, C.POINTER(KernelTimes)]
    lib.atspeed_align_data.argtypes = [vp, i32, pi32, pi32, pi32, C.POINTER(AlignArgs)]
    lib.atspeed_align_step.argtypes = [vp, C.POINTER(AlignArgs), C.POINTER(C.c_double)]
    lib.atspeed_target_search.argtypes = [vp, i32, i32, pi32, pi32, pf, pi32, pi32, pi32, pi32]
    lib.atspeed_mixed_search.argtypes = [vp, C.c_float, i32, i32, pi32, pi32, pf, pi32, pi32, pi32, pi32]
    for name in SYMBOLS:
        fn = getattr(lib, name)
        if fn.restype is C.c_int:  # default
            fn.restype = C.c_int
    return lib


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _np_ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(C.POINTER(ctype))


class Engine:
    """One context of the library: weights, workspace and state on one GPU.

    ``target_w`` / ``draft_w`` are weight dicts in the layout of
    ``synth.make_weights`` (uint16 bf16 bit patterns or float32).
    """

    def __init__(self, w, target_w: Dict[str, np.ndarray], draft_w: Optional[Dict[str, np.ndarray]],
                 catalog: np.ndarray, max_batch: Optional[int] = None, max_prefix: Optional[int] = None,
                 device: str = "cuda:0", mode: int = STRICT, stream=None, seed: int = 0, sd_start_level: int = 0,
                 reuse_tree_kv: int = 0):
        import torch
        self.torch = torch
        self.lib = load_library()
        self.w = w
        self.device = torch.device(device)
        self.bf16 = w.dtype == "bf16"
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        cfg = Config()
        for dst, m in ((cfg.target, w.target), (cfg.draft, w.draft if draft_w is not None else None)):
            if m is None:
                continue
            dst.n_layers, dst.d_model, dst.n_heads = m.n_layers, m.d_model, m.n_heads
            dst.d_ffn, dst.vocab, dst.item_base = m.d_ffn, m.vocab, m.item_base
        cfg.L, cfg.codebook, cfg.K, cfg.N, cfg.gamma = w.L, w.codebook, w.K, w.N, w.gamma
        cfg.max_batch = max_batch or w.batch
        cfg.max_prefix = max_prefix or w.prefix_len
        cfg.mode, cfg.temperature, cfg.seed = mode, w.temperature, seed
        cfg.dtype = BF16 if self.bf16 else FP32
        cfg.sd_start_level = sd_start_level
        cfg.reuse_tree_kv = reuse_tree_kv
        cfg.stream = self.stream.cuda_stream
        self.cfg = cfg
        self._keep = []
        self.tw = self._upload(target_w, w.target.n_layers)
        self.target_dev = self._keep[-2]
        self.dw = self._upload(draft_w, w.draft.n_layers) if draft_w is not None else None
        self.draft_dev = self._keep[-2] if draft_w is not None else None   # device tensors of the draft
        cat = np.ascontiguousarray(catalog, dtype=np.int32)
        self._cat_arr = cat
        self.cat = Catalog(cat.shape[0], _np_ptr(cat, C.c_int32))
        nbytes = C.c_size_t(0)
        self._check(self.lib.atspeed_workspace_bytes(C.byref(cfg), C.byref(self.cat), C.byref(nbytes)))
        self.ws = torch.empty(nbytes.value, dtype=torch.uint8, device=self.device)
        base = self.ws.data_ptr()
        off = (-base) % 256
        ctx = C.c_void_p()
        self._check(self.lib.atspeed_create(C.byref(cfg), C.byref(self.tw), C.byref(self.dw) if self.dw else None,
                                            C.byref(self.cat), base + off, nbytes.value - off, C.byref(ctx)))
        self.ctx = ctx

    # -- plumbing
    def _check(self, status: int):
        if status != 0:
            raise AtspeedError(status, self.lib.atspeed_last_error().decode())

    def _dev(self, a: np.ndarray):
        t = self.torch
        if a.dtype == np.uint16:
            return t.from_numpy(a.view(np.int16)).to(self.device).view(t.bfloat16)
        return t.from_numpy(np.ascontiguousarray(a)).to(self.device)

    def _upload(self, W: Dict[str, np.ndarray], n_layers: int) -> Weights:
        dev = {k: self._dev(v) for k, v in W.items()}
        self._keep.append(dev)
        ptrs = (C.c_void_p * (n_layers * 9))()
        for l in range(n_layers):
            for i, name in enumerate(LAYER_ORDER):
                ptrs[l * 9 + i] = dev[f"l{l}.{name}"].data_ptr()
        self._keep.append(ptrs)
        return Weights(dev["tok_emb"].data_ptr(), ptrs, dev["final_norm"].data_ptr(), dev["lm_head_item"].data_ptr())

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.atspeed_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def max_nodes(self) -> int:
        return self.w.K * (self.w.L - 1) + self.w.gamma * self.w.N

    @property
    def n_item(self) -> int:
        return self.w.L * self.w.codebook

    # -- calls
    def atspeed_prefill(self, prefix, root_logits=None):
        B, P = prefix.shape
        self._check(self.lib.atspeed_prefill(self.ctx, B, P, _ptr(prefix), _ptr(root_logits)))

    def atspeed_draft(self):
        self._check(self.lib.atspeed_draft(self.ctx))

    def atspeed_get_tree(self) -> Tree:
        tr = Tree()
        self._check(self.lib.atspeed_get_tree(self.ctx, C.byref(tr)))
        return tr

    def atspeed_verify(self, accepted=None, t_after=None, logits=None):
        self._check(self.lib.atspeed_verify(self.ctx, _ptr(accepted), _ptr(t_after), _ptr(logits)))

    def atspeed_capture_hidden(self, x=None, plan=None, max_rows=0, act=None, model=0, skip=0):
        self._check(self.lib.atspeed_capture_hidden(self.ctx, int(model), int(skip), _ptr(x), _ptr(act), _ptr(plan),
                                                    int(max_rows)))

    def atspeed_tree_logits(self, logits):
        self._check(self.lib.atspeed_tree_logits(self.ctx, _ptr(logits)))

    def atspeed_accept(self, logits, root_logits, accepted=None, t_after=None):
        self._check(self.lib.atspeed_accept(self.ctx, _ptr(logits), _ptr(root_logits), _ptr(accepted), _ptr(t_after)))

    def atspeed_accept_noalloc(self, logits, root_logits, accepted=None, t_after=None):
        self._check(self.lib.atspeed_accept_noalloc(self.ctx, _ptr(logits), _ptr(root_logits), _ptr(accepted),
                                                    _ptr(t_after)))

    def atspeed_decode_topk(self, prefix, items, scores, n_items, stats: Optional[Stats] = None):
        B, P = prefix.shape
        self._check(self.lib.atspeed_decode_topk(self.ctx, B, P, _ptr(prefix), _ptr(items), _ptr(scores),
                                                 _ptr(n_items), C.byref(stats) if stats is not None else None))

    def atspeed_target_search(self, prefix, items, scores, n_items, step_items=None, step_lens=None, step_n=None):
        B, P = prefix.shape
        self._check(self.lib.atspeed_target_search(self.ctx, B, P, _ptr(prefix), _ptr(items), _ptr(scores),
                                                   _ptr(n_items), _ptr(step_items), _ptr(step_lens), _ptr(step_n)))

    def atspeed_mixed_search(self, lam, prefix, items, scores, n_items, step_items=None, step_lens=None, step_n=None):
        B, P = prefix.shape
        self._check(self.lib.atspeed_mixed_search(self.ctx, lam, B, P, _ptr(prefix), _ptr(items), _ptr(scores),
                                                  _ptr(n_items), _ptr(step_items), _ptr(step_lens), _ptr(step_n)))

    def atspeed_logprobs(self, model, lp, root):
        self._check(self.lib.atspeed_logprobs(self.ctx, model, _ptr(lp), _ptr(root)))

    def atspeed_align_data(self, items, lens, n_items, args: AlignArgs):
        """items [B, S, L] int32, lens [B, S] int32 or None, n_items [B] int32 (device)."""
        self._check(self.lib.atspeed_align_data(self.ctx, items.shape[1], _ptr(items), _ptr(lens), _ptr(n_items),
                                                C.byref(args)))

    def atspeed_align_step(self, args: AlignArgs) -> float:
        loss = C.c_double(0.0)
        self._check(self.lib.atspeed_align_step(self.ctx, C.byref(args), C.byref(loss)))
        return loss.value

    def atspeed_get_state(self, B: int):
        K, L = self.w.K, self.w.L
        t = np.zeros(B, np.int32)
        nb = np.zeros(B, np.int32)
        paths = np.zeros((B, K, L), np.int32)
        sc = np.zeros((B, K), np.float32)
        self._check(self.lib.atspeed_get_state(self.ctx, B, _np_ptr(t, C.c_int32), _np_ptr(nb, C.c_int32),
                                               _np_ptr(paths, C.c_int32), _np_ptr(sc, C.c_float)))
        return t, nb, paths, sc

    def atspeed_set_state(self, t, nb, paths, scores):
        t = np.ascontiguousarray(t, np.int32)
        nb = np.ascontiguousarray(nb, np.int32)
        paths = np.ascontiguousarray(paths, np.int32)
        scores = np.ascontiguousarray(scores, np.float32)
        self._check(self.lib.atspeed_set_state(self.ctx, len(t), _np_ptr(t, C.c_int32), _np_ptr(nb, C.c_int32),
                                               _np_ptr(paths, C.c_int32), _np_ptr(scores, C.c_float)))

    def atspeed_set_timing(self, enable=True, target_only=False):
        """enable: True (every kernel class), False (off), or an iterable of
        class names from KERNEL_CLASSES (only those launches are bracketed);
        target_only: leave the draft model's launches out."""
        if enable is True:
            mask = (1 << len(KERNEL_CLASSES)) - 1
        elif not enable:
            mask = 0
        else:
            mask = sum(1 << KERNEL_CLASSES.index(k) for k in set(enable))
        if mask and target_only:
            mask |= TIME_TARGET_ONLY
        self._check(self.lib.atspeed_set_timing(self.ctx, mask))

    def atspeed_get_timing(self) -> Dict[str, tuple]:
        """class -> (ms, launches, algorithmic GFLOP of the target's GEMM launches)."""
        kt = KernelTimes()
        self._check(self.lib.atspeed_get_timing(self.ctx, C.byref(kt)))
        return {k: (kt.ms[i], kt.launches[i], kt.gflop[i]) for i, k in enumerate(KERNEL_CLASSES)}

    # -- tree upload / download (device SoA of the context)
    def tree_tensors(self, B: int):
        """Torch views of the context's tree arrays (n_nodes [B], token/parent/depth [B, T], q_score [B, T])."""
        t = self.torch
        tr = self.atspeed_get_tree()
        T = tr.max_nodes

        def view(ptr, n, dtype):
            # the workspace tensor owns the memory; index it by byte offset
            off = ptr - self.ws.data_ptr()
            return self.ws[off: off + n * 4].view(dtype)

        return (view(tr.n_nodes, B, t.int32), view(tr.token, B * T, t.int32).view(B, T),
                view(tr.parent, B * T, t.int32).view(B, T), view(tr.depth, B * T, t.int32).view(B, T),
                view(tr.q_score, B * T, t.float32).view(B, T))
