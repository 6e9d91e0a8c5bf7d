"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these tests touches the GPU library.  Each one would fail for a
plausible mistake in the oracle (dropped or wrong-signed phi, a wrong shift,
a transposed operand, a wrong group index, a wrong tie-break, an off-by-one
threshold interval, a wrong count rounding, a wrong plane order).
"""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import bruteforce as bf
from oracle import grinqh_oracle as orc
from synth import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            rows.append([part.split() for part in line.split("|")])
    return rows


# ------------------------------------------------------------------ RTN ----
def test_rtn_hand_examples():
    for ws, s, codes in _read_golden("rtn_hand.txt"):
        w = np.array([float(v) for v in ws], dtype=np.float16)[None, :]
        q, sc = orc.rtn_quantize(w, group=w.shape[1])
        assert float(sc[0, 0]) == float(s[0])
        assert q[0].tolist() == [int(c) for c in codes]


def test_rtn_matches_exact_rational_rtn():
    rng = np.random.default_rng(7)
    for trial in range(40):
        scale = 10.0 ** rng.uniform(-6, 2)
        w = (rng.standard_normal((3, 16)) * scale).astype(np.float16)
        if trial % 5 == 0:
            w[0, :] = 0.0
        q, sc = orc.rtn_quantize(w, group=8)
        for n in range(3):
            for g in range(2):
                grp = [float(v) for v in w[n, g * 8:(g + 1) * 8]]
                codes, s = bf.rtn_group_exact(grp)
                assert float(sc[g, n]) == s
                assert q[n, g * 8:(g + 1) * 8].tolist() == codes


def test_rtn_code_range_and_symmetry():
    w = inputs.weights(64, 256, config=99)
    q, sc = orc.rtn_quantize(w)
    assert q.min() >= 1 and q.max() <= 255          # |w/s| <= 127 -> codes 1..255
    q2, sc2 = orc.rtn_quantize(-w)
    assert np.array_equal(sc, sc2)
    assert np.array_equal(q2.astype(int) - 128, -(q.astype(int) - 128))


# ----------------------------------------------------- reconstruction ----
def test_reconstruction_against_bin_enumeration():
    s = 0.5
    for b in range(1, 9):
        for q in range(256):
            want = float(bf.w_hat(q, Fraction(s), b))
            got = float(orc.reconstruct(np.array([q]), np.array([s]), b)[0])
            assert got == want, (q, b)


def test_reconstruction_error_bound_and_mean_shift():
    # phi moves the truncated value from the floor of its bin towards the
    # centre (Sec. 3.3): the error against the full code is at most half a
    # b-bit bin, and over all codes the mean shift is exactly +1/2 code unit
    # (phi = half the bin width, R10).  A dropped phi breaks the bound, a
    # negative phi breaks both.
    q = np.arange(256)
    full = orc.reconstruct(q, np.ones(256), 8)
    assert np.array_equal(full, q - 128.0)
    for b in range(1, 8):
        r = orc.reconstruct(q, np.ones(256), b)
        assert np.max(np.abs(r - full)) <= 2.0 ** (7 - b)
        assert np.mean(r - full) == 0.5
    assert np.all(orc.reconstruct(q, np.ones(256), 0) == 0.0)


def test_nested_code_is_prefix():
    for q in range(256):
        for b in range(0, 9):
            got = int(orc.nested_code(np.array([q]), b)[0])
            want = int(bf.code_bits(q)[:b], 2) if b else 0
            assert got == want


# ----------------------------------------------------------- matvec ----
def _tiny_case(seed, N, K, G):
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 256, size=(N, K), dtype=np.uint8)
    scales = rng.uniform(0.01, 1.0, size=(K // G, N)).astype(np.float16)
    x = rng.standard_normal(K).astype(np.float16)
    return codes, scales, x


@pytest.mark.parametrize("level_bits", [(0, 2, 4, 8), (0, 2, 4, 6, 8), (0, 2, 3, 4, 8)])
def test_vmm_exhaustive_level_maps_bruteforce(level_bits):
    # every level map of a K = 4, two-group (G = 2), N = 3 case, exact arithmetic
    N, K, G = 3, 4, 2
    codes, scales, x = _tiny_case(11, N, K, G)
    sc_f = [[Fraction(float(scales[g, n])) for n in range(N)] for g in range(K // G)]
    x_f = [Fraction(float(v)) for v in x]
    cq = [[int(v) for v in row] for row in codes]
    for levels in itertools.product(range(len(level_bits)), repeat=K):
        want = bf.vmm_exact(cq, sc_f, x_f, list(levels), level_bits, G)
        got = orc.vmm(codes, scales, x, np.array(levels), level_bits, group=G)
        for n in range(N):
            w = float(want[n])
            assert abs(got[n] - w) <= 1e-12 * max(1.0, abs(w)), (levels, n)


def test_vmm_random_maps_bruteforce_larger():
    N, K, G = 5, 16, 4
    level_bits = (0, 2, 4, 6, 8)
    codes, scales, x = _tiny_case(12, N, K, G)
    sc_f = [[Fraction(float(scales[g, n])) for n in range(N)] for g in range(K // G)]
    x_f = [Fraction(float(v)) for v in x]
    cq = [[int(v) for v in row] for row in codes]
    rng = np.random.default_rng(3)
    for _ in range(60):
        levels = rng.integers(0, len(level_bits), size=K)
        want = bf.vmm_exact(cq, sc_f, x_f, levels.tolist(), level_bits, G)
        got = orc.vmm(codes, scales, x, levels, level_bits, group=G)
        for n in range(N):
            assert abs(got[n] - float(want[n])) <= 1e-12 * max(1.0, abs(float(want[n])))


def test_vmm_all_top_is_textbook_dequant_matvec():
    W = inputs.weights(48, 256, config=98)
    x = inputs.activations_t3(256, 1, config=98)[0]
    q, s = orc.rtn_quantize(W)
    y = orc.vmm(q, s, x, np.full(256, 3), (0, 2, 4, 8))
    # symmetric RTN dequantisation s * (q - 128), written directly
    deq = np.empty((48, 256))
    for n in range(48):
        for k in range(256):
            deq[n, k] = float(s[k // 128, n]) * (int(q[n, k]) - 128)
    ref = deq @ x.astype(np.float64)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)
    # and it approximates the unquantised fp16 matvec (RTN error only)
    dense = W.astype(np.float64) @ x.astype(np.float64)
    assert np.max(np.abs(y - dense)) < 0.02 * np.max(np.abs(dense)) + 1e-3


def test_prefill_bruteforce_exact():
    # every channel at 8 bits, each token's row summed exactly in rationals
    G, N, K, M = 128, 5, 256, 3
    codes = inputs.random_codes(N, K, 3, 1)
    scales = inputs.random_scales(N, K, G, 3, 1).T.copy()          # [K/G, N]
    x = inputs.activations_t3(K, M, 3, 1)
    got = orc.prefill(codes, scales, x)
    cq = codes.astype(int).tolist()
    sc_f = [[Fraction(float(scales[g, n])) for n in range(N)] for g in range(K // G)]
    for m in range(M):
        x_f = [Fraction(float(v)) for v in x[m]]
        want = bf.vmm_exact(cq, sc_f, x_f, [1] * K, (0, 8), G)
        np.testing.assert_allclose(got[m], [float(v) for v in want], rtol=1e-12, atol=0)


def test_prefill_unit_tokens_read_single_weights():
    # token m = 2^-3 e_k reads back 2^-3 s[k // 128][n] (q[n][k] - 128) exactly:
    # a transposed operand, a wrong group index or a dropped offset all fail
    G, N, K = 128, 6, 384
    codes = inputs.random_codes(N, K, 4, 2)
    scales = inputs.random_scales(N, K, G, 4, 2).T.copy()
    ks = [0, 1, 127, 128, 200, 383]
    x = np.zeros((len(ks), K), dtype=np.float16)
    for m, k in enumerate(ks):
        x[m, k] = 0.125
    y = orc.prefill(codes, scales, x)
    for m, k in enumerate(ks):
        for n in range(N):
            assert y[m, n] == 0.125 * float(scales[k // G, n]) * (int(codes[n, k]) - 128)


def test_prefill_rows_equal_decode_at_top_level():
    G, N, K, M = 128, 16, 512, 4
    codes = inputs.random_codes(N, K, 5, 3)
    scales = inputs.random_scales(N, K, G, 5, 3).T.copy()
    x = inputs.activations_t3(K, M, 5, 3)
    top = np.full((M, K), 3, dtype=np.uint8)
    np.testing.assert_allclose(orc.prefill(codes, scales, x),
                               orc.vmm_batch(codes, scales, x, top, (0, 2, 4, 8)),
                               rtol=1e-13, atol=1e-13)


def test_vmm_all_skipped_is_zero():
    W = inputs.weights(32, 256, config=97)
    x = inputs.activations_t3(256, 1, config=97)[0]
    q, s = orc.rtn_quantize(W)
    y = orc.vmm(q, s, x, np.zeros(256, dtype=np.uint8), (0, 2, 4, 8))
    assert np.all(y == 0.0)


def test_reconstruct_at_zero_bits_is_zero():
    # R2: a skipped channel contributes exactly 0.  (A 0-bit read has q_b = 0
    # and phi = 2^(b_max-1), so s * phi cancels z = -2^(b_max-1) s exactly:
    # the formula and the skip agree bit for bit.)
    q = np.arange(256, dtype=np.uint8)
    s = np.full(256, 0.0123, dtype=np.float64)
    for b_max in (4, 6, 8):
        assert np.all(orc.reconstruct(q >> (8 - b_max), s, 0, b_max) == 0.0)


def test_vmm_single_level_equals_truncated_uniform_quantiser():
    # all channels at b bits: the layer acts as a uniform b-bit quantiser whose
    # grid is the 8-bit grid coarsened by 2^(8-b), offset by phi.
    W = inputs.weights(16, 256, config=96)
    x = inputs.activations_t3(256, 1, config=96)[0].astype(np.float64)
    q, s = orc.rtn_quantize(W)
    for lvl, b in enumerate((0, 2, 4, 6, 8)):
        y = orc.vmm(q, s, x.astype(np.float16), np.full(256, lvl), (0, 2, 4, 6, 8))
        step = 2 ** (8 - b)
        grid = (q.astype(np.int64) // step) * step + (step // 2 if b < 8 else 0)
        s_full = np.repeat(s.astype(np.float64).T, 128, axis=1)
        ref = (s_full * (grid - 128)) @ x if b else np.zeros(16)
        np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_vmm_linear_in_level_masks():
    W = inputs.weights(24, 384, config=95)
    x = inputs.activations_t3(384, 1, config=95)[0]
    q, s = orc.rtn_quantize(W)
    rng = np.random.default_rng(5)
    lv = rng.integers(0, 5, size=384)
    bits = (0, 2, 4, 6, 8)
    total = orc.vmm(q, s, x, lv, bits)
    parts = sum(orc.vmm(q, s, x, np.where(lv == j, j, 0), bits) for j in range(1, 5))
    np.testing.assert_allclose(total, parts, rtol=1e-12, atol=1e-12)


def test_vmm_batch_is_per_token():
    W = inputs.weights(16, 256, config=94)
    x = inputs.activations_t3(256, 3, config=94)
    q, s = orc.rtn_quantize(W)
    lv = np.random.default_rng(1).integers(0, 4, size=(3, 256))
    yb = orc.vmm_batch(q, s, x, lv, (0, 2, 4, 8))
    for t in range(3):
        assert np.array_equal(yb[t], orc.vmm(q, s, x[t], lv[t], (0, 2, 4, 8)))


# ------------------------------------------------------- assignment ----
def test_threshold_matches_searchsorted_and_boundaries():
    rng = np.random.default_rng(4)
    x = (rng.standard_t(3, size=5000) * 2).astype(np.float16)
    th = np.array([0.25, 0.5, 1.5, 3.0], dtype=np.float32)
    got = orc.assign_threshold(x, th)
    ax = np.abs(x.astype(np.float32))
    want = np.searchsorted(th, ax, side="right")
    assert np.array_equal(got, want)
    # |x| exactly on a threshold goes to the higher level (left-closed)
    edge = np.array([0.25, -0.5, 1.5, 3.0, 0.0, 65504.0], dtype=np.float16)
    assert orc.assign_threshold(edge, th).tolist() == [1, 2, 3, 4, 0, 4]
    # equal thresholds make an empty level; +inf disables the top level
    th2 = np.array([0.5, 0.5, np.inf], dtype=np.float32)
    assert orc.assign_threshold(np.array([0.4, 0.5, 7.0], np.float16), th2).tolist() == [0, 2, 2]


def test_topk_counts_rule():
    for K in (1, 7, 128, 1000, 4096, 14336):
        for p in [(3000, 5000, 1500, 500), (2000, 2000, 3000, 3000), (0, 0, 0, 10000),
                  (2500, 2200, 3100, 2200, 0), (3333, 3333, 3334, 0, 0)]:
            c = orc.topk_counts(K, p)
            assert c.sum() == K and np.all(c >= 0)
            for j in range(len(p)):
                exact = Fraction(sum(p[j:]) * K, 10000)
                half_up = (exact + Fraction(1, 2)).numerator // (exact + Fraction(1, 2)).denominator
                assert int(c[j:].sum()) == half_up


def test_topk_matches_pairwise_ranks_with_ties():
    rng = np.random.default_rng(9)
    for trial in range(30):
        K = int(rng.integers(1, 40))
        vals = np.array([0.0, -0.0, 0.5, -0.5, 1.0, 2.0, -3.0, 65504.0], dtype=np.float16)
        x = rng.choice(vals, size=K).astype(np.float16)
        p = rng.multinomial(10000, [0.25, 0.25, 0.25, 0.25])
        counts = orc.topk_counts(K, p)
        got = orc.assign_topk(x, counts)
        keys = orc.magnitude_key(x).tolist()
        want = bf.topk_levels_pairwise(keys, counts.tolist())
        assert got.tolist() == want
        assert np.array_equal(np.bincount(got, minlength=4), counts)


def test_magnitude_key_orders_every_finite_fp16_like_abs():
    # App. A.1 ranks channels by |x|.  Every finite fp16 bit pattern (both
    # signs, +-0, subnormals, +-65504): the key must order them exactly as
    # |x| in float64 does, with equal keys only for equal magnitudes.
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    x = bits.view(np.float16)
    x = x[np.isfinite(x)]
    key = orc.magnitude_key(x)
    mag = np.abs(x.astype(np.float64))
    order = np.argsort(mag, kind="stable")
    k_sorted, m_sorted = key[order], mag[order]
    assert np.all(np.diff(k_sorted) >= 0)
    # equal magnitude <=> equal key (e.g. -0.0 and +0.0, x and -x)
    same_mag = np.diff(m_sorted) == 0
    same_key = np.diff(k_sorted) == 0
    assert np.array_equal(same_mag, same_key)
    assert key[x == np.float16(-65504.0)][0] == key[x == np.float16(65504.0)][0]


def test_topk_matches_independent_abs_sort_signed_values():
    # Independent route to the top-p partition: a stable sort of -|x| in
    # float64 (ties keep the lower index, reading R7), then levels handed out
    # from the top in rank order.  Signed inputs with negatives, -0.0,
    # subnormals and +-65504, so a key that ignored the sign bit wrongly (or
    # used the signed value) would fail.
    rng = np.random.default_rng(97)
    special = np.array([0.0, -0.0, 6e-8, -6e-8, 1e-5, -1e-5, 0.5, -0.5, 2.0, -3.0,
                        65504.0, -65504.0], dtype=np.float16)
    for trial in range(60):
        K = int(rng.integers(1, 300))
        if trial % 3 == 0:
            x = rng.choice(special, size=K).astype(np.float16)
        elif trial % 3 == 1:
            x = (rng.standard_t(3, K) * 4).astype(np.float16)
        else:
            x = np.where(rng.random(K) < 0.5, rng.choice(special, size=K),
                         rng.standard_normal(K)).astype(np.float16)
        n_lv = int(rng.integers(2, 6))
        p = rng.multinomial(10000, [1.0 / n_lv] * n_lv)
        counts = orc.topk_counts(K, p)
        got = orc.assign_topk(x, counts)
        order = np.argsort(-np.abs(x.astype(np.float64)), kind="stable")
        want = np.empty(K, dtype=np.int64)
        r = 0
        for j in range(n_lv - 1, -1, -1):
            want[order[r:r + counts[j]]] = j
            r += counts[j]
        assert got.tolist() == want.tolist(), (trial, x.tolist())


def test_topk_exact_budget_on_workload_shapes():
    x = inputs.activations_t3(4096, 2, config=93)
    for p in inputs.BUDGETS[inputs.LEVELS_B].values():
        counts = orc.topk_counts(4096, p)
        lv = orc.assign_topk(x, counts)
        for t in range(2):
            assert np.array_equal(np.bincount(lv[t], minlength=5), counts)
            # monotone: larger magnitude never gets a lower level
            key = orc.magnitude_key(x[t])
            order = np.argsort(-key, kind="stable")
            assert np.all(np.diff(lv[t][order].astype(int)) <= 0)


def test_calibration_matches_library_quantiles():
    # type-7 sample quantiles are numpy's 'linear' percentiles; the oracle
    # fixes the position exactly, so the two agree to rounding
    rng = np.random.default_rng(93)
    for n in (128, 1000, 4096):
        samples = [np.abs(rng.standard_t(3, n)).astype(np.float16).astype(np.float64) for _ in range(5)]
        for p in [(2000, 800, 2400, 4800, 0), (0, 0, 0, 10000), (2500, 2500, 2500, 2500), (3333, 3333, 3334)]:
            cum = np.cumsum(p)[:-1]
            lib = np.mean([[np.percentile(a, c / 100.0) for c in cum] for a in samples], axis=0)
            ours = orc.calibrate_thresholds(samples, p)
            np.testing.assert_allclose(ours, lib.astype(np.float32), rtol=2e-7, atol=0)


def test_calibration_exact_small_case():
    # n = 5 magnitudes 1..5, quantiles at 25% and 60%: h = 1.0 and 2.4
    a = np.array([5.0, 1.0, 4.0, 2.0, 3.0])
    th = orc.calibrate_thresholds([a], (2500, 3500, 4000))
    assert th[0] == np.float32(2.0)
    assert th[1] == np.float32(3.0 + 0.4 * 1.0)
    # two samples: the mean of the per-sample values
    th2 = orc.calibrate_thresholds([a, 2 * a], (2500, 7500))
    assert th2[0] == np.float32((2.0 + 4.0) / 2)


def test_calibrated_thresholds_reproduce_fractions_on_one_sample():
    a = np.abs(inputs.activations_t3(4096, 1, config=92)[0].astype(np.float64))
    p = (2000, 2000, 3000, 3000)
    th = orc.calibrate_thresholds([a], p)
    lv = orc.assign_threshold(a.astype(np.float16), th)
    counts = np.bincount(lv, minlength=4)
    target = np.array(p) * 4096 / 10000
    assert np.all(np.abs(counts - target) <= 8)    # ties at fp16 resolution


# ----------------------------------------------------------- layout ----
def _bit_reader(packed, N, K, u, T, n, k, planes):
    """Independent bit-by-bit read of the first `planes` planes of code (n, k)."""
    t, o = divmod(n, T)
    row = (t * K + k) * T
    plane_bytes = T * u // 8
    val = 0
    for j in range(planes):
        for bit in range(u - 1, -1, -1):
            pos = o * u + bit
            byte = packed[row + j * plane_bytes + pos // 8]
            val = (val << 1) | ((int(byte) >> (pos % 8)) & 1)
    return val


def test_pack_golden_const_rows():
    for (u, T), vals in [((int(a), int(b)), [int(v) for v in rest])
                         for (a, b), rest in _read_golden("pack_const_rows.txt")]:
        codes = np.full((T, 2), 0xE4, dtype=np.uint8)
        packed = orc.pack_codes(codes, u, T)
        pb = T * u // 8
        for k in range(2):
            row = packed[k * T:(k + 1) * T]
            for j, v in enumerate(vals):
                assert np.all(row[j * pb:(j + 1) * pb] == v)


@pytest.mark.parametrize("u,T", [(2, 256), (2, 512), (1, 512)])
def test_pack_prefix_property_bitwise(u, T):
    rng = np.random.default_rng(21)
    N, K = 2 * T, 3
    codes = rng.integers(0, 256, size=(N, K), dtype=np.uint8)
    packed = orc.pack_codes(codes, u, T)
    assert np.array_equal(packed, orc.pack_codes_fast(codes, u, T))
    for n in rng.integers(0, N, size=64):
        for k in range(K):
            for planes in range(0, 8 // u + 1):
                got = _bit_reader(packed, N, K, u, T, int(n), k, planes)
                assert got == int(codes[n, k]) >> (8 - planes * u)
    for depth in range(0, 9, u):
        qb = orc.unpack_prefix(packed, N, K, u, T, depth)
        assert np.array_equal(qb, codes.astype(np.int64) >> (8 - depth))


def test_pack_fast_matches_reference_packer_bigger():
    rng = np.random.default_rng(22)
    codes = rng.integers(0, 256, size=(1024, 16), dtype=np.uint8)
    for u, T in [(2, 256), (2, 1024), (1, 512), (1, 1024)]:
        assert np.array_equal(orc.pack_codes(codes, u, T), orc.pack_codes_fast(codes, u, T))


def test_plane_bits_for_level_sets():
    assert orc.plane_bits_for((0, 2, 4, 8)) == 2
    assert orc.plane_bits_for((0, 2, 4, 6, 8)) == 2
    assert orc.plane_bits_for((0, 2, 3, 4, 8)) == 1
