"""Pins for the oracle's bf16 emulation and Philox generator (CPU)."""
import json
import math
import os

import numpy as np
import pytest

from oracle.numerics import bf16_bits_to_f64, round_bf16
from oracle import philox

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _all_bf16_values():
    bits = np.arange(1 << 16, dtype=np.uint32)
    # decode by the IEEE layout: sign(1) exponent(8) mantissa(7)
    sign = np.where(bits >> 15, -1.0, 1.0)
    exp = (bits >> 7) & 0xFF
    man = bits & 0x7F
    val = np.where(exp == 0, sign * man * 2.0 ** -133,
                   sign * (1.0 + man / 128.0) * np.exp2(exp.astype(np.float64) - 127))
    finite = exp != 0xFF
    return bits[finite], val[finite]


def test_bf16_decode_known_patterns():
    assert bf16_bits_to_f64(np.array([0x3F80], np.uint16))[0] == 1.0
    assert bf16_bits_to_f64(np.array([0xC000], np.uint16))[0] == -2.0
    assert bf16_bits_to_f64(np.array([0x4049], np.uint16))[0] == 3.140625
    bits, val = _all_bf16_values()
    np.testing.assert_array_equal(bf16_bits_to_f64(bits.astype(np.uint16)), val)


def test_round_bf16_is_nearest_ties_even():
    bits, val = _all_bf16_values()
    order = np.argsort(val, kind="stable")
    sv, sb = val[order], bits[order]
    # drop the duplicate zero (-0 == +0)
    keep = np.concatenate([[True], sv[1:] != sv[:-1]])
    sv, sb = sv[keep], sb[keep]
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(20000) * 10 ** rng.uniform(-6, 6, 20000),
                        # exact midpoints between neighbours: ties must go to the even mantissa
                        (sv[1000:1200] + sv[1001:1201]) / 2])
    got = round_bf16(x)
    i = np.clip(np.searchsorted(sv, x), 1, len(sv) - 1)
    lo, hi = sv[i - 1], sv[i]
    dlo, dhi = x - lo, hi - x
    even_lo = (sb[i - 1] & 1) == 0
    want = np.where(dlo < dhi, lo, np.where(dhi < dlo, hi, np.where(even_lo, lo, hi)))
    np.testing.assert_array_equal(got, want)


def test_philox_known_answers():
    with open(os.path.join(GOLDEN, "philox_kat.json")) as f:
        kat = json.load(f)
    for c in kat["cases"]:
        ctr = [int(x, 16) for x in c["ctr"]]
        key = [int(x, 16) for x in c["key"]]
        out = philox.philox4x32_10(ctr, key)
        assert ["%08x" % v for v in out] == c["out"]


def test_philox_uniforms():
    xs = [philox.philox4x32_10((i, 7, 0, 3), (0x1234, 0x5678))[0] for i in range(20000)]
    u = np.array([philox.uniform(x) for x in xs])
    assert u.min() > 0.0 and u.max() < 1.0
    # every uniform is exactly representable in fp32
    assert np.all(u.astype(np.float32).astype(np.float64) == u)
    # 16-bin chi-square at alpha = 1e-3 (critical value of chi2 with 15 dof = 37.70)
    h = np.bincount((u * 16).astype(int), minlength=16)
    chi2 = float(((h - 1250.0) ** 2 / 1250.0).sum())
    assert chi2 < 37.70
    g = np.array([philox.gumbel(x) for x in xs])
    # Gumbel(0,1): mean = Euler-Mascheroni constant, variance = pi^2 / 6
    assert abs(g.mean() - 0.5772156649) < 0.03
    assert abs(g.var() - math.pi ** 2 / 6) < 0.08
