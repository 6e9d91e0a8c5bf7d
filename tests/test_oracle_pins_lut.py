"""Pins of the oracle's look-up-table (non-uniform nested) VMM.

Sec. 3.3 allows any quantiser with the nested property, naming k-means
style nested weights, whose levels are centred so no midpoint bias is
applied; the appendix on nested weight formats evaluates such weights.
A wrong prefix shift, a table indexed by the wrong output, a level's
table swapped for another's, a stray phi or a skipped channel that still
counts all fail one of these.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import bruteforce as bf
from oracle import grinqh_oracle as orc
from synth import inputs


def _uniform_luts(N, level_bits, s_out):
    """Tables that reproduce the uniform reconstruction with one scale per
    output (s_out[n], powers of two so every entry is exact in fp16)."""
    b_max = level_bits[-1]
    luts = {}
    for b in level_bits:
        if b == 0:
            continue
        c = np.arange(2 ** b, dtype=np.float64)
        vals = c * 2 ** (b_max - b) + orc.midpoint_bias(b, b_max) - 2 ** (b_max - 1)
        luts[b] = (s_out[:, None] * vals[None, :]).astype(np.float16)
        assert np.array_equal(luts[b].astype(np.float64), s_out[:, None] * vals[None, :])
    return luts


@pytest.mark.parametrize("level_bits", [(0, 2, 4, 8), (0, 2, 4, 6, 8), (0, 2, 4, 6), (0, 1, 2, 3, 4)])
def test_lut_with_uniform_tables_is_the_uniform_vmm(level_bits):
    b_max = level_bits[-1]
    N, K = 24, 256
    rng = np.random.default_rng(b_max + len(level_bits))
    codes = rng.integers(0, 2 ** b_max, size=(N, K)).astype(np.uint8)
    s_out = 2.0 ** rng.integers(-9, -5, size=N).astype(np.float64)
    luts = _uniform_luts(N, level_bits, s_out)
    scales = np.repeat(s_out[None, :], K // 128, axis=0).astype(np.float16)
    x = inputs.activations_t3(K, 3, 11, b_max)
    for t in range(3):
        lm = rng.integers(0, len(level_bits), size=K)
        np.testing.assert_allclose(orc.vmm_lut(codes, luts, x[t], lm, level_bits),
                                   orc.vmm(codes, scales, x[t], lm, level_bits),
                                   rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("level_bits", [(0, 2, 4, 8), (0, 2, 4, 6)])
def test_lut_bruteforce(level_bits):
    b_max = level_bits[-1]
    N, K = 3, 6
    rng = np.random.default_rng(31)
    codes = rng.integers(0, 2 ** b_max, size=(N, K))
    luts = inputs.nested_luts(N, level_bits, 12, b_max)
    x = rng.standard_normal(K).astype(np.float16)
    for trial in range(10):
        lm = rng.integers(0, len(level_bits), size=K)
        want = []
        for n in range(N):
            acc = Fraction(0)
            for k in range(K):
                b = level_bits[lm[k]]
                if b == 0:
                    continue
                prefix = int(bf.code_bits(int(codes[n, k]), b_max)[:b], 2)   # the b leading bits
                acc += Fraction(float(x[k])) * Fraction(float(luts[b][n, prefix]))
            want.append(float(acc))
        np.testing.assert_allclose(orc.vmm_lut(codes, luts, x, lm, level_bits), want, rtol=1e-12, atol=1e-15)


def test_lut_all_skipped_and_all_top():
    level_bits = (0, 2, 4, 6, 8)
    N, K = 16, 384
    codes = inputs.random_codes(N, K, 13, 1)
    luts = inputs.nested_luts(N, level_bits, 13, 1)
    x = inputs.activations_t3(K, 1, 13, 1)[0]
    assert np.all(orc.vmm_lut(codes, luts, x, np.zeros(K, dtype=int), level_bits) == 0.0)
    top = np.full(K, len(level_bits) - 1)
    direct = np.array([sum(float(x[k]) * float(luts[8][n, codes[n, k]]) for k in range(K)) for n in range(N)])
    np.testing.assert_allclose(orc.vmm_lut(codes, luts, x, top, level_bits), direct, rtol=1e-12)


def test_nested_luts_are_means_of_their_children():
    level_bits = (0, 2, 4, 6, 8)
    luts = inputs.nested_luts(8, level_bits, 14, 0)
    for b in (2, 4, 6):
        child = luts[b + 2].astype(np.float64).reshape(8, 2 ** b, 4).mean(axis=2)
        # each side rounds to fp16 separately: agree to about one fp16 ulp
        np.testing.assert_allclose(luts[b].astype(np.float64), child, rtol=2.0 ** -10, atol=4e-5)
    assert np.all(np.diff(luts[8].astype(np.float64), axis=1) >= 0)    # sorted centroids
