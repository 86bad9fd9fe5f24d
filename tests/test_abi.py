"""The C-ABI library loads, exports every declared entry point, and validates
arguments on the host (no GPU needed: these calls never reach the device)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "atspeed.h")


def _lib():
    from paper_2410_05165_amd import binding
    return binding, binding.load_library()


def test_library_exports_every_declared_symbol():
    binding, lib = _lib()
    declared = re.findall(r"ATSPEED_API\s+[\w\s\*]+?\b(atspeed_\w+)\s*\(", open(HEADER).read())
    assert len(declared) >= 13
    assert set(declared) == set(binding.SYMBOLS)
    for name in declared:
        assert hasattr(lib, name), name


def _cfg(binding, **kw):
    c = binding.Config()
    c.target = binding.Dims(2, 128, 4, 512, 1024, 0)
    c.draft = binding.Dims(1, 64, 2, 256, 1024, 0)
    c.L, c.codebook, c.K, c.N, c.gamma = 4, 256, 10, 10, 4
    c.max_batch, c.max_prefix, c.mode, c.temperature, c.seed, c.dtype = 1, 80, 0, 1.0, 0, 0
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def _catalog(binding, n=50, L=4, cb=256, dup=False):
    rng = np.random.default_rng(0)
    codes = rng.integers(0, cb, size=(n, L)).astype(np.int32)
    if dup:
        codes[1] = codes[0]
    return codes, binding.Catalog(n, codes.ctypes.data_as(C.POINTER(C.c_int32)))


def test_workspace_bytes_and_argument_errors():
    binding, lib = _lib()
    codes, cat = _catalog(binding)
    n = C.c_size_t(0)
    assert lib.atspeed_workspace_bytes(C.byref(_cfg(binding)), C.byref(cat), C.byref(n)) == 0
    assert n.value > 0
    bad = [dict(K=0), dict(N=5), dict(L=5), dict(codebook=300), dict(gamma=0), dict(max_batch=0),
           dict(mode=7), dict(dtype=3), dict(sd_start_level=2), dict(reuse_tree_kv=2),
           dict(mode=1, sd_start_level=1), dict(mode=2, sd_start_level=1)]
    for kw in bad:
        st = lib.atspeed_workspace_bytes(C.byref(_cfg(binding, **kw)), C.byref(cat), C.byref(n))
        assert st == 1, (kw, st)
    # shapes: heads must divide d_model; bf16 needs d_head 64/128
    st = lib.atspeed_workspace_bytes(C.byref(_cfg(binding, target=binding.Dims(2, 130, 4, 512, 1024, 0))),
                                     C.byref(cat), C.byref(n))
    assert st == 2
    st = lib.atspeed_workspace_bytes(C.byref(_cfg(binding, dtype=1)), C.byref(cat), C.byref(n))
    assert st == 2
    # vocabulary must hold the item tokens
    st = lib.atspeed_workspace_bytes(C.byref(_cfg(binding, target=binding.Dims(2, 128, 4, 512, 1000, 0))),
                                     C.byref(cat), C.byref(n))
    assert st == 2
    assert lib.atspeed_workspace_bytes(None, C.byref(cat), C.byref(n)) == 1
    assert b"null" in lib.atspeed_last_error()


def test_catalog_validation():
    binding, lib = _lib()
    n = C.c_size_t(0)
    codes, cat = _catalog(binding, dup=True)
    assert lib.atspeed_workspace_bytes(C.byref(_cfg(binding)), C.byref(cat), C.byref(n)) == 1
    assert b"duplicate" in lib.atspeed_last_error()
    codes, cat = _catalog(binding, n=5)          # fewer items than K = 10
    assert lib.atspeed_workspace_bytes(C.byref(_cfg(binding)), C.byref(cat), C.byref(n)) == 1
    codes, cat = _catalog(binding, cb=8)
    codes[3, 2] = 9                              # code outside the codebook
    assert lib.atspeed_workspace_bytes(C.byref(_cfg(binding, codebook=8)), C.byref(cat), C.byref(n)) == 1


def test_create_rejects_bad_workspace_before_any_launch():
    binding, lib = _lib()
    codes, cat = _catalog(binding)
    ctx = C.c_void_p()
    w = binding.Weights()
    assert lib.atspeed_create(C.byref(_cfg(binding)), C.byref(w), None, C.byref(cat), None, 0, C.byref(ctx)) == 3
    assert lib.atspeed_create(C.byref(_cfg(binding)), C.byref(w), None, C.byref(cat), 0x1001, 1 << 40,
                              C.byref(ctx)) == 3  # misaligned
    assert lib.atspeed_create(C.byref(_cfg(binding)), C.byref(w), None, C.byref(cat), 0x100000, 16,
                              C.byref(ctx)) == 3  # too small
    assert lib.atspeed_prefill(None, 1, 1, None, None) == 1
    assert lib.atspeed_verify(None, None, None, None) == 1


def test_tree_kv_reuse_workspace():
    """reuse_tree_kv keeps two sets of the target's per-layer tree K/V and tree
    log-probs instead of one layer's K/V: the workspace grows by the K/V of
    2 * n_layers - 1 layers, one more log-prob buffer, and six small index
    arrays (four slot-sized, two user-sized), up to alignment padding."""
    binding, lib = _lib()
    codes, cat = _catalog(binding)
    n0, n1 = C.c_size_t(0), C.c_size_t(0)
    assert lib.atspeed_workspace_bytes(C.byref(_cfg(binding)), C.byref(cat), C.byref(n0)) == 0
    assert lib.atspeed_workspace_bytes(C.byref(_cfg(binding, reuse_tree_kv=1)), C.byref(cat), C.byref(n1)) == 0
    B, Tm, d, nl, es, nitem = 1, 10 * 3 + 4 * 10, 128, 2, 4, 4 * 256
    kv = 2 * (2 * nl - 1) * B * Tm * d * es
    extra = kv + B * Tm * nitem * 4 + 4 * B * Tm * 4 + 2 * B * 4
    pad = 64 * 256   # each buffer starts on a 256-byte boundary
    assert extra - pad <= n1.value - n0.value <= extra + pad, (n1.value - n0.value, extra)
