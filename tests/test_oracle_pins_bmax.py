"""Pins of the oracle at b_max = 4 and 6 (Sec. 3.3: weights stored at
b_max in {4, 6, 8} bits, read in 2-bit segments up to b_max).

Each test would fail for a plausible mistake in the b_max generalisation:
the wrong RTN divisor or offset, phi not zero at the top level, a shift
from 8 instead of b_max, an 8-bit row length, or a wrong plane count.
"""
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import bruteforce as bf
from oracle import grinqh_oracle as orc
from synth import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_rtn_bmax_hand_examples():
    n = 0
    with open(os.path.join(GOLDEN, "rtn_hand_bmax.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            b, ws, s, cs = [p.split() for p in line.split("|")]
            w = np.array([float(v) for v in ws], dtype=np.float16)[None, :]
            q, sc = orc.rtn_quantize(w, group=w.shape[1], b_max=int(b[0]))
            assert float(sc[0, 0]) == float(s[0])
            assert q[0].tolist() == [int(c) for c in cs]
            n += 1
    assert n == 6


@pytest.mark.parametrize("b_max", [4, 6])
def test_rtn_bmax_matches_exact_rational_rtn(b_max):
    rng = np.random.default_rng(70 + b_max)
    for trial in range(30):
        scale = 10.0 ** rng.uniform(-5, 2)
        w = (rng.standard_normal((2, 16)) * scale).astype(np.float16)
        q, sc = orc.rtn_quantize(w, group=8, b_max=b_max)
        assert q.max() < 2 ** b_max
        for nn in range(2):
            for g in range(2):
                codes, s = bf.rtn_group_exact([float(v) for v in w[nn, g * 8:(g + 1) * 8]], b_max)
                assert float(sc[g, nn]) == s
                assert q[nn, g * 8:(g + 1) * 8].tolist() == codes


@pytest.mark.parametrize("b_max", [4, 6])
def test_reconstruction_bmax_against_bin_enumeration(b_max):
    s = 0.25
    for b in range(1, b_max + 1):
        for q in range(2 ** b_max):
            want = float(bf.w_hat(q, Fraction(s), b, b_max))
            got = float(orc.reconstruct(np.array([q]), np.array([s]), b, b_max)[0])
            assert got == want, (q, b)
    # full depth is the plain dequantisation s (q - 2^(b_max-1))
    q = np.arange(2 ** b_max)
    assert np.array_equal(orc.reconstruct(q, np.full(q.shape, s), b_max, b_max),
                          s * (q - 2 ** (b_max - 1)))


@pytest.mark.parametrize("level_bits", [(0, 2, 4), (0, 2, 4, 6), (0, 1, 2, 3, 4)])
def test_vmm_bmax_bruteforce(level_bits):
    b_max = level_bits[-1]
    G, N, K = 4, 3, 8
    rng = np.random.default_rng(sum(level_bits))
    codes = rng.integers(0, 2 ** b_max, size=(N, K)).astype(np.uint8)
    scales = (rng.uniform(0.5, 2.0, size=(K // G, N))).astype(np.float16)
    x = rng.standard_normal(K).astype(np.float16)
    sc_f = [[Fraction(float(scales[g, n])) for n in range(N)] for g in range(K // G)]
    x_f = [Fraction(float(v)) for v in x]
    for trial in range(20):
        levels = rng.integers(0, len(level_bits), size=K)
        want = bf.vmm_exact(codes.astype(int).tolist(), sc_f, x_f, levels.tolist(), level_bits, G)
        got = orc.vmm(codes, scales, x, levels, level_bits, group=G)
        np.testing.assert_allclose(got, [float(v) for v in want], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("b_max", [4, 6])
def test_prefill_bmax_unit_tokens(b_max):
    G, N, K = 128, 4, 256
    rng = np.random.default_rng(b_max)
    codes = rng.integers(0, 2 ** b_max, size=(N, K)).astype(np.uint8)
    scales = inputs.random_scales(N, K, G, 8, b_max).T.copy()
    ks = [0, 127, 128, 255]
    x = np.zeros((len(ks), K), dtype=np.float16)
    for m, k in enumerate(ks):
        x[m, k] = 1.0
    y = orc.prefill(codes, scales, x, b_max=b_max)
    for m, k in enumerate(ks):
        for n in range(N):
            assert y[m, n] == float(scales[k // G, n]) * (int(codes[n, k]) - 2 ** (b_max - 1))


def _bit_reader(packed, K, u, T, b_max, n, k, planes):
    """Independent bit-by-bit read of the first `planes` planes of code (n, k)."""
    t, o = divmod(n, T)
    row = (t * K + k) * (T * b_max // 8)
    plane_bytes = T * u // 8
    val = 0
    for j in range(planes):
        for bit in range(u - 1, -1, -1):
            pos = o * u + bit
            byte = packed[row + j * plane_bytes + pos // 8]
            val = (val << 1) | ((int(byte) >> (pos % 8)) & 1)
    return val


@pytest.mark.parametrize("b_max,u,T", [(4, 2, 256), (6, 2, 256), (6, 2, 512), (6, 1, 512), (4, 1, 512)])
def test_pack_bmax_prefix_property(b_max, u, T):
    rng = np.random.default_rng(b_max * 10 + u)
    N, K = 2 * T, 3
    codes = rng.integers(0, 2 ** b_max, size=(N, K), dtype=np.uint8)
    packed = orc.pack_codes(codes, u, T, b_max)
    assert packed.size == N * K * b_max // 8
    assert np.array_equal(packed, orc.pack_codes_fast(codes, u, T, b_max))
    for n in rng.integers(0, N, size=48):
        for k in range(K):
            for planes in range(0, b_max // u + 1):
                got = _bit_reader(packed, K, u, T, b_max, int(n), k, planes)
                assert got == int(codes[n, k]) >> (b_max - planes * u)
    for depth in range(0, b_max + 1, u):
        qb = orc.unpack_prefix(packed, N, K, u, T, depth, b_max)
        assert np.array_equal(qb, codes.astype(np.int64) >> (b_max - depth))
