"""GPU parity of libgrinqh against the CPU oracle (run on an MI355X).

Bars: packed codes, scales and level maps bit-exact; y within max-normwise
relative error 1e-3 of the float64 oracle (max_n |y - y_ref| / max_n |y_ref|).
All calls go through the C ABI via the thin binding.
"""
import numpy as np
import pytest

from oracle import grinqh_oracle as orc
from synth import inputs

pytestmark = pytest.mark.gpu
TOL = 1e-3


@pytest.fixture(scope="module")
def g():
    from paper_2606_23419_amd import grinqh
    return grinqh


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


@pytest.fixture
def opts(g):
    """Set launch overrides (grinqh_set_option) for one test, reset after it."""
    touched = []

    def setopt(option, value):
        g.grinqh_set_option(option, int(value))
        touched.append(option)
    yield setopt
    for option in touched:
        g.grinqh_set_option(option, 0)


KERNEL = {"dot2": 1, "v0": 2}   # GRINQH_KERNEL_PER_PLANE, GRINQH_KERNEL_GENERAL


def _dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _host(t):
    return t.detach().cpu().numpy()


def normwise(y, ref):
    ref = np.asarray(ref, dtype=np.float64)
    den = np.max(np.abs(ref))
    num = np.max(np.abs(np.asarray(y, dtype=np.float64) - ref))
    return num / den if den > 0 else num


class Layer:
    """One packed layer: GPU buffers and the oracle's codes/scales."""

    def __init__(self, g, torch, K, N, levels, cfg=50, layer=0, tile_n=0, codes_src=False):
        self.desc = g.grinqh_resolve_desc(g.make_desc(K, N, levels, tile_n=tile_n))
        self.levels = tuple(levels)
        self.b_max = int(levels[-1])
        self.K, self.N = K, N
        if codes_src:
            self.codes = inputs.random_codes(N, K, cfg, layer)
            if self.b_max < 8:
                self.codes = (self.codes & ((1 << self.b_max) - 1)).astype(np.uint8)
            sc_nk = inputs.random_scales(N, K, 128, cfg, layer)
            self.scales = np.ascontiguousarray(sc_nk.T)
            self.pc, self.ps = g.grinqh_pack(self.desc, codes=_dev(torch, self.codes),
                                             scales=_dev(torch, sc_nk))
        else:
            W = inputs.weights(N, K, cfg, layer)
            self.codes, self.scales = orc.rtn_quantize(W, b_max=self.b_max)
            self.pc, self.ps = g.grinqh_pack(self.desc, W=_dev(torch, W))
        torch.cuda.synchronize()

    def check_packed(self):
        u, T = self.desc.plane_bits, self.desc.tile_n
        want = orc.pack_codes_fast(self.codes, u, T, self.b_max)
        got = _host(self.pc)
        assert np.array_equal(got, want), f"packed codes differ at {np.nonzero(got != want)[0][:8]}"
        assert np.array_equal(_host(self.ps).view(np.uint16), self.scales.view(np.uint16))


# ------------------------------------------------------------------ pack ----
@pytest.mark.parametrize("K,N,levels,tile_n", [
    (128, 512, (0, 2, 4, 8), 0), (640, 1024, (0, 2, 4, 6, 8), 256), (256, 2048, (0, 2, 3, 4, 8), 0),
    (384, 2048, (0, 2, 4, 8), 2048), (256, 1024, (0, 2, 3, 4, 8), 1024)])
def test_pack_rtn_bit_exact(g, torch, K, N, levels, tile_n):
    Layer(g, torch, K, N, levels, tile_n=tile_n).check_packed()


def test_pack_codes_source_bit_exact(g, torch):
    Layer(g, torch, 512, 1024, (0, 2, 4, 6, 8), codes_src=True).check_packed()
    Layer(g, torch, 256, 512, (0, 2, 3, 4, 8), codes_src=True).check_packed()


def test_pack_rtn_edge_groups(g, torch):
    # zero groups, a subnormal-only group (scale underflows to 0), ties
    K, N = 256, 512
    W = inputs.weights(N, K, 51).copy()
    W[0, :128] = 0.0
    W[1, :128] = np.float16(2.0 ** -23)
    W[2, :] = np.float16(127.0)
    W[2, 1:5] = np.array([2.5, 3.5, -2.5, -0.0], dtype=np.float16)
    desc = g.grinqh_resolve_desc(g.make_desc(K, N, (0, 2, 4, 8)))
    pc, ps = g.grinqh_pack(desc, W=_dev(torch, W))
    q, s = orc.rtn_quantize(W)
    assert np.array_equal(_host(pc), orc.pack_codes_fast(q, 2, desc.tile_n))
    assert np.array_equal(_host(ps).view(np.uint16), s.view(np.uint16))


# ---------------------------------------------------------------- assign ----
@pytest.mark.parametrize("K", [128, 640, 4096, 14336])
def test_assign_threshold_bit_exact(g, torch, K):
    desc = g.make_desc(K, 512, (0, 2, 4, 6, 8))
    x = inputs.activations_t3(K, 3, 52)
    th = np.array([0.3, 0.7, 1.5, 4.0], dtype=np.float32)
    x[0, :4] = np.array([0.3, -0.7, 1.5, 4.0], dtype=np.float16).astype(np.float16)
    lm = g.grinqh_assign(desc, _dev(torch, x), g.GRINQH_ASSIGN_THRESHOLD, thresholds=th)
    assert np.array_equal(_host(lm), orc.assign_threshold(x, th))


@pytest.mark.parametrize("K", [128, 640, 1024, 4096, 14336])
@pytest.mark.parametrize("levels", [(0, 2, 4, 8), (0, 2, 4, 6, 8), (0, 2, 3, 4, 8)])
def test_assign_topk_bit_exact(g, torch, K, levels):
    desc = g.make_desc(K, 512, levels)
    x = inputs.activations_t3(K, 4, 53) if K != 14336 else inputs.activations_swiglu(K, 4, 53)
    for p in inputs.BUDGETS[tuple(levels)].values():
        counts = g.grinqh_topk_counts(K, p)
        lm = g.grinqh_assign(desc, _dev(torch, x), g.GRINQH_ASSIGN_TOPK, counts=counts)
        assert np.array_equal(_host(lm), orc.assign_topk(x, counts))


@pytest.mark.parametrize("case", ["ties", "all_equal", "zeros", "signed_zero", "extreme_counts"])
def test_assign_topk_adversarial(g, torch, case):
    K = 1024
    rng = np.random.default_rng(54)
    desc = g.make_desc(K, 512, (0, 2, 4, 8))
    if case == "ties":
        x = rng.choice(np.array([0.5, -0.5, 1.0, 2.0, -2.0, 0.0], np.float16), size=(3, K))
    elif case == "all_equal":
        x = np.full((2, K), -1.25, dtype=np.float16)
    elif case == "zeros":
        x = np.zeros((2, K), dtype=np.float16)
    elif case == "signed_zero":
        x = np.where(rng.random((2, K)) < 0.5, np.float16(0.0), np.float16(-0.0)).astype(np.float16)
        x[:, ::7] = np.float16(3.0)
    else:
        x = inputs.activations_t3(K, 2, 55)
    x = x.astype(np.float16)
    plist = [(2000, 2000, 3000, 3000), (0, 0, 0, 10000), (10000, 0, 0, 0), (3333, 3333, 3334, 0)]
    for p in plist:
        counts = g.grinqh_topk_counts(K, p)
        lm = g.grinqh_assign(desc, _dev(torch, x), g.GRINQH_ASSIGN_TOPK, counts=counts)
        assert np.array_equal(_host(lm), orc.assign_topk(x, counts)), (case, p)
    # counts of a single channel at each level
    counts = [K - 3, 1, 1, 1]
    lm = g.grinqh_assign(desc, _dev(torch, x), g.GRINQH_ASSIGN_TOPK, counts=counts)
    assert np.array_equal(_host(lm), orc.assign_topk(x, counts))


# ------------------------------------------------------------------- vmm ----
def _vmm_case(g, torch, L, x, lm):
    y = g.grinqh_vmm(L.desc, L.pc, L.ps, _dev(torch, x), _dev(torch, lm))
    torch.cuda.synchronize()
    ref = orc.vmm_batch(L.codes, L.scales, x, lm, L.levels)
    return _host(y), ref


@pytest.mark.parametrize("K,N,levels,tile_n", [
    (128, 512, (0, 2, 4, 8), 0), (640, 1024, (0, 2, 4, 6, 8), 256), (1024, 1024, (0, 2, 4, 8), 0),
    (384, 2048, (0, 2, 3, 4, 8), 0), (896, 2048, (0, 2, 4, 6, 8), 1024), (256, 2048, (0, 2, 4, 8), 2048),
    (640, 3072, (0, 2, 4, 6, 8), 1024)])
@pytest.mark.parametrize("B", [1, 2, 4])
def test_vmm_topk_parity(g, torch, K, N, levels, tile_n, B):
    L = Layer(g, torch, K, N, levels, tile_n=tile_n)
    x = inputs.activations_t3(K, B, 56, 1)
    for p in inputs.BUDGETS[tuple(levels)].values():
        counts = g.grinqh_topk_counts(K, p)
        lm = _host(g.grinqh_assign(L.desc, _dev(torch, x), g.GRINQH_ASSIGN_TOPK, counts=counts))
        assert np.array_equal(lm, orc.assign_topk(x, counts)), p
        y, ref = _vmm_case(g, torch, L, x, lm)
        assert normwise(y, ref) <= TOL, (p, normwise(y, ref))


@pytest.mark.parametrize("levels", [(0, 2, 4, 8), (0, 2, 4, 6, 8), (0, 2, 3, 4, 8)])
def test_vmm_random_level_maps(g, torch, levels):
    K, N = 1152, 1024
    L = Layer(g, torch, K, N, levels, cfg=57)
    rng = np.random.default_rng(57)
    for B in (1, 3):
        x = inputs.activations_t3(K, B, 57, 2)
        lm = rng.integers(0, len(levels), size=(B, K)).astype(np.uint8)
        y, ref = _vmm_case(g, torch, L, x, lm)
        assert normwise(y, ref) <= TOL


def test_vmm_all_skipped_is_exactly_zero(g, torch):
    L = Layer(g, torch, 512, 1024, (0, 2, 4, 8), cfg=58)
    x = inputs.activations_t3(512, 2, 58)
    y, _ = _vmm_case(g, torch, L, x, np.zeros((2, 512), np.uint8))
    assert np.all(y == 0.0)


def test_vmm_all_top_is_dequant_matvec(g, torch):
    L = Layer(g, torch, 512, 1024, (0, 2, 4, 8), cfg=59)
    x = inputs.activations_t3(512, 1, 59)
    y, _ = _vmm_case(g, torch, L, x, np.full((1, 512), 3, np.uint8))
    s_full = np.repeat(L.scales.astype(np.float64).T, 128, axis=1)
    ref = (s_full * (L.codes.astype(np.float64) - 128)) @ x[0].astype(np.float64)
    assert normwise(y[0], ref) <= TOL


def test_vmm_single_level_and_mixed_tokens(g, torch):
    levels = (0, 2, 4, 6, 8)
    L = Layer(g, torch, 768, 1024, levels, cfg=60)
    x = inputs.activations_t3(768, 4, 60)
    lm = np.stack([np.full(768, j, np.uint8) for j in (1, 2, 3, 4)])
    y, ref = _vmm_case(g, torch, L, x, lm)
    for t in range(4):
        assert normwise(y[t], ref[t]) <= TOL


def test_vmm_batch_equals_single_tokens(g, torch):
    levels = (0, 2, 4, 6, 8)
    L = Layer(g, torch, 1024, 1024, levels, cfg=61)
    x = inputs.activations_t3(1024, 4, 61)
    rng = np.random.default_rng(61)
    lm = rng.integers(0, 5, size=(4, 1024)).astype(np.uint8)
    yb, ref = _vmm_case(g, torch, L, x, lm)
    for t in range(4):
        y1, _ = _vmm_case(g, torch, L, x[t:t + 1], lm[t:t + 1])
        assert normwise(y1[0], ref[t]) <= TOL
        assert normwise(yb[t], ref[t]) <= TOL


def test_vmm_accumulate_flag_and_clamped_levels(g, torch):
    L = Layer(g, torch, 512, 512, (0, 2, 4, 8), cfg=62)
    x = inputs.activations_t3(512, 1, 62)
    lm = np.random.default_rng(62).integers(0, 4, size=(1, 512)).astype(np.uint8)
    y0 = torch.full((1, 512), 1.5, dtype=torch.float32, device="cuda")
    g.grinqh_vmm(L.desc, L.pc, L.ps, _dev(torch, x), _dev(torch, lm), y=y0, accumulate=True)
    ref = orc.vmm_batch(L.codes, L.scales, x, lm, L.levels) + 1.5
    assert normwise(_host(y0), ref) <= TOL
    # a level value above the top level is read as the top level
    lm_hi = lm.copy()
    lm_hi[lm_hi == 3] = 200
    y, _ = _vmm_case(g, torch, L, x, lm_hi)
    assert normwise(y, orc.vmm_batch(L.codes, L.scales, x, lm, L.levels)) <= TOL


@pytest.mark.parametrize("levels", [(0, 2, 4, 8), (0, 2, 3, 4, 8)])
def test_vmm_threshold_fused(g, torch, levels):
    K, N = 1024, 1024
    L = Layer(g, torch, K, N, levels, cfg=63)
    x = inputs.activations_t3(K, 3, 63)
    th = np.sort(np.abs(x[0].astype(np.float32)))[[300, 500, 800, 1000][:len(levels) - 1]]
    lm_out = torch.zeros((3, K), dtype=torch.uint8, device="cuda")
    y = g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, _dev(torch, x), th, level_map_out=lm_out)
    torch.cuda.synchronize()
    lm = orc.assign_threshold(x, th)
    assert np.array_equal(_host(lm_out), lm)
    ref = orc.vmm_batch(L.codes, L.scales, x, lm, levels)
    assert normwise(_host(y), ref) <= TOL


def _topk_fused_case(g, torch, L, x, counts, accumulate_check=False):
    """Fused top-k VMM against the oracle (level map bit-exact, y normwise) and
    against the two-launch path (assign, then VMM)."""
    K = L.K
    lm_out = torch.full((1, K), 255, dtype=torch.uint8, device="cuda")
    xd = _dev(torch, x)
    y = g.grinqh_vmm_topk(L.desc, L.pc, L.ps, xd, counts, level_map_out=lm_out)
    lm2 = g.grinqh_assign(L.desc, xd, g.GRINQH_ASSIGN_TOPK, counts=counts)
    y2 = g.grinqh_vmm(L.desc, L.pc, L.ps, xd, lm2)
    torch.cuda.synchronize()
    lm = orc.assign_topk(x, counts)
    assert np.array_equal(_host(lm_out), lm), counts
    # same kernel and level map; the groups' partial sums meet in atomics, so
    # the two agree to float32 rounding of the order of additions
    assert normwise(_host(y), _host(y2)) <= 1e-6, counts
    ref = orc.vmm_batch(L.codes, L.scales, x, lm, L.levels)
    assert normwise(_host(y), ref) <= TOL, (counts, normwise(_host(y), ref))
    if accumulate_check:
        y0 = torch.from_numpy(np.full((1, L.N), 0.75, np.float32)).cuda()
        g.grinqh_vmm_topk(L.desc, L.pc, L.ps, xd, counts, y=y0, accumulate=True)
        torch.cuda.synchronize()
        assert normwise(_host(y0) - 0.75, ref) <= TOL


@pytest.mark.parametrize("K,N,levels,tile_n", [
    (128, 512, (0, 2, 4, 8), 512), (640, 1024, (0, 2, 4, 6, 8), 256), (1152, 2048, (0, 2, 4, 8), 1024),
    (4096, 4096, (0, 2, 4, 6, 8), 512), (4096, 1024, (0, 2, 4, 6), 256), (2048, 2048, (0, 2, 4), 512),
    (14336, 1024, (0, 2, 4, 6, 8), 1024), (16384, 512, (0, 2, 4, 8), 512)])
def test_vmm_topk_fused(g, torch, K, N, levels, tile_n):
    L = Layer(g, torch, K, N, levels, cfg=64, tile_n=tile_n)
    x = (inputs.activations_swiglu if K >= 4096 else inputs.activations_t3)(K, 1, 64)
    for i, p in enumerate(inputs.BUDGETS[tuple(levels)].values()):
        _topk_fused_case(g, torch, L, x, g.grinqh_topk_counts(K, p), accumulate_check=i == 0)


@pytest.mark.parametrize("case", ["ties", "all_equal", "zeros", "signed_zero", "extreme_counts"])
def test_vmm_topk_fused_adversarial(g, torch, case):
    K, N = 1024, 1024
    L = Layer(g, torch, K, N, (0, 2, 4, 8), cfg=65, tile_n=512)
    rng = np.random.default_rng(65)
    if case == "ties":
        x = rng.choice(np.array([0.5, -0.5, 1.0, 2.0, -2.0, 0.0], np.float16), size=(1, K))
    elif case == "all_equal":
        x = np.full((1, K), -1.25, dtype=np.float16)
    elif case == "zeros":
        x = np.zeros((1, K), dtype=np.float16)
    elif case == "signed_zero":
        x = np.where(rng.random((1, K)) < 0.5, np.float16(0.0), np.float16(-0.0)).astype(np.float16)
        x[:, ::7] = np.float16(3.0)
    else:
        x = inputs.activations_t3(K, 1, 66)
    x = x.astype(np.float16)
    for p in [(2000, 2000, 3000, 3000), (0, 0, 0, 10000), (10000, 0, 0, 0), (3333, 3333, 3334, 0)]:
        _topk_fused_case(g, torch, L, x, g.grinqh_topk_counts(K, p))
    for counts in ([K - 3, 1, 1, 1], [0, K - 2, 1, 1], [1, 1, 1, K - 3], [K - 511, 0, 511, 0]):
        _topk_fused_case(g, torch, L, x, counts)


@pytest.mark.parametrize("K,N,levels,tile_n", [
    (640, 1024, (0, 2, 4, 6, 8), 256), (1152, 2048, (0, 2, 4, 8), 512), (4096, 2048, (0, 2, 4, 6, 8), 1024)])
def test_vmm_topk_fused_shared_lists(g, torch, opts, K, N, levels, tile_n):
    """The top-k selecting kernel with the workgroup-shared lists (two groups
    per workgroup, as on the MLP projections)."""
    opts(g.GRINQH_OPT_GROUPS_PER_WG, 2)
    L = Layer(g, torch, K, N, levels, cfg=69, tile_n=tile_n)
    x = inputs.activations_t3(K, 1, 69)
    for p in inputs.BUDGETS[tuple(levels)].values():
        _topk_fused_case(g, torch, L, x, g.grinqh_topk_counts(K, p))


@pytest.mark.parametrize("name,K,N,xkind", [
    ("gate|up 4096->28672 (shared lists)", 4096, 28672, "t3"),
    ("down 14336->4096", 14336, 4096, "swiglu")])
def test_vmm_topk_fused_full_size_every_output(g, torch, name, K, N, xkind):
    """Every output of one fused top-k launch at a full MLP shape."""
    levels = inputs.LEVELS_B
    L = Layer(g, torch, K, N, levels, cfg=70, layer=K + N, codes_src=True)
    x = (inputs.activations_swiglu if xkind == "swiglu" else inputs.activations_t3)(K, 1, 70, K + N)
    counts = g.grinqh_topk_counts(K, inputs.BUDGETS[levels][4])
    lm_out = torch.zeros((1, K), dtype=torch.uint8, device="cuda")
    y = _host(g.grinqh_vmm_topk(L.desc, L.pc, L.ps, _dev(torch, x), counts, level_map_out=lm_out))
    lm = orc.assign_topk(x, counts)
    assert np.array_equal(_host(lm_out), lm), name
    ref = oracle_all_outputs(L.codes, L.scales, x, lm, levels)
    err = normwise(y, ref)
    print(f"{name}: normwise {err:.2e}, elementwise {elementwise(y, ref):.2e}")
    assert err <= TOL, (name, err)


def test_vmm_topk_fused_ties_across_threads(g, torch):
    """Runs of equal magnitudes that straddle the per-thread key runs, with cuts
    landing inside a run: the channel-order tie break decides the level map."""
    K, N = 4096, 1024
    L = Layer(g, torch, K, N, (0, 2, 4, 6, 8), cfg=67, tile_n=512)
    x = inputs.activations_t3(K, 1, 67).astype(np.float16)
    x[0, 1000:1100] = np.float16(7.5)
    x[0, 3000:3050] = np.float16(-7.5)
    x[0, 10:4000:13] = np.float16(2.25)
    ax = np.abs(x[0].astype(np.float32))
    n75, n225 = int((ax == 7.5).sum()), int((ax == 2.25).sum())
    above75 = int((ax > 7.5).sum())
    above225 = int((ax > 2.25).sum())
    cases = [
        [K - (above75 + 70), 0, 0, 0, above75 + 70],                       # cut inside the 7.5 run
        [K - (above225 + 7), 0, 0, above225 + 7 - (above75 + 3), above75 + 3],
        [K - (above75 + n75), 0, 0, 0, above75 + n75],                     # cut at the end of a run
        [K - (above75 + 1), 0, 0, 0, above75 + 1],                         # first of a run
    ]
    for counts in cases:
        assert sum(counts) == K and min(counts) >= 0, counts
        _topk_fused_case(g, torch, L, x, counts)


# ------------------------------------------------------- calibration ----
@pytest.mark.parametrize("K", [128, 1152, 4096, 14336])
def test_calibrate_matches_oracle(g, torch, K):
    levels = inputs.LEVELS_B
    d = g.make_desc(K, 1024, levels)
    S = 12
    x = inputs.activations_t3(K, S, 67, K)
    rng = np.random.default_rng(K)
    x[3] = rng.integers(-3, 4, K).astype(np.float16)          # heavy ties
    x[5] = np.float16(0.5)                                     # one value
    samples = [np.abs(r.astype(np.float64)) for r in x]
    budgets = list(inputs.BUDGETS[levels].values()) + [(0, 0, 0, 0, 10000), (10000, 0, 0, 0, 0),
                                                       (1, 1, 1, 1, 9996)]
    for p in budgets:
        th = _host(g.grinqh_calibrate(d, _dev(torch, x), p))
        ref = orc.calibrate_thresholds(samples, p)
        assert np.array_equal(th, ref), (K, p, th, ref)


def test_calibrated_threshold_path_hits_budget(g, torch):
    # calibrate on one set of tokens, grade held-out tokens inside the VMM
    levels = inputs.LEVELS_B
    K, N = 4096, 1024
    L = Layer(g, torch, K, N, levels, cfg=68)
    calib = inputs.activations_t3(K, 64, 68, 1)
    test = inputs.activations_t3(K, 8, 68, 2)
    p = inputs.BUDGETS[levels][4]
    th = _host(g.grinqh_calibrate(L.desc, _dev(torch, calib), p))
    lm_out = torch.zeros((8, K), dtype=torch.uint8, device="cuda")
    xd = _dev(torch, test)
    ys = [g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, xd[t:t + 1], th, level_map_out=lm_out[t:t + 1])
          for t in range(8)]
    torch.cuda.synchronize()
    lm = orc.assign_threshold(test, th)
    assert np.array_equal(_host(lm_out), lm)
    y = np.concatenate([_host(v) for v in ys])
    assert normwise(y, orc.vmm_batch(L.codes, L.scales, test, lm, levels)) <= TOL
    achieved = float(np.asarray(levels)[lm].mean())
    assert abs(achieved - 4.0) < 0.25, achieved


# ------------------------------------------ full-size workload shapes ----
FULL = [
    ("cfg1 1024x1024", 1024, 1024, inputs.LEVELS_A, "t3"),
    ("cfg2 q 4096x4096", 4096, 4096, inputs.LEVELS_B, "t3"),
    ("cfg2 k 4096->1024", 4096, 1024, inputs.LEVELS_B, "t3"),
    ("cfg3 up 4096->14336", 4096, 14336, inputs.LEVELS_B, "t3"),
    ("cfg3 down 14336->4096", 14336, 4096, inputs.LEVELS_B, "swiglu"),
    ("cfg4 qkv 4096->6144", 4096, 6144, inputs.LEVELS_C, "t3"),
    ("cfg4 down 12288->4096", 12288, 4096, inputs.LEVELS_C, "swiglu"),
    # the merged projections the benchmarks run (two groups per workgroup)
    ("cfg3 gate|up 4096->28672", 4096, 28672, inputs.LEVELS_B, "t3"),
    ("cfg4 gate|up 4096->24576", 4096, 24576, inputs.LEVELS_C, "t3"),
]


@pytest.mark.parametrize("name,K,N,levels,xkind", FULL, ids=[f[0] for f in FULL])
def test_full_size_pack_and_sampled_vmm(g, torch, name, K, N, levels, xkind):
    L = Layer(g, torch, K, N, levels, cfg=70, layer=K + N)
    L.check_packed()
    gen = inputs.activations_swiglu if xkind == "swiglu" else inputs.activations_t3
    x = gen(K, 2, 70, K + N)
    rows = np.sort(np.random.default_rng(K + N).choice(N, size=96, replace=False))
    for p in inputs.BUDGETS[tuple(levels)].values():
        counts = g.grinqh_topk_counts(K, p)
        lm = g.grinqh_assign(L.desc, _dev(torch, x), g.GRINQH_ASSIGN_TOPK, counts=counts)
        lm_h = _host(lm)
        assert np.array_equal(lm_h, orc.assign_topk(x, counts))
        y = _host(g.grinqh_vmm(L.desc, L.pc, L.ps, _dev(torch, x), lm))
        ref = orc.vmm_batch(L.codes[rows], L.scales[:, rows], x, lm_h, levels)
        # sampled outputs against the oracle, and the whole vector's scale
        assert normwise(y[:, rows], ref) <= TOL, (name, p)
        assert np.all(np.isfinite(y))
    # one token (the batch-1 plane-pair kernel), from the level map and with
    # the grading fused in (thresholds at the last budget's cut points)
    y1 = _host(g.grinqh_vmm(L.desc, L.pc, L.ps, _dev(torch, x[:1]), lm[:1]))
    ref1 = orc.vmm_batch(L.codes[rows], L.scales[:, rows], x[:1], lm_h[:1], levels)
    assert normwise(y1[:, rows], ref1) <= TOL, (name, "B=1")
    ax = np.sort(np.abs(x[0].astype(np.float32)))[::-1]
    n = len(levels)
    th = np.sort(ax[np.linspace(K // 8, K - K // 8, n - 1).astype(int)]).astype(np.float32)
    lm_out = torch.zeros((1, K), dtype=torch.uint8, device="cuda")
    yt = _host(g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, _dev(torch, x[:1]), th, level_map_out=lm_out))
    lmt = orc.assign_threshold(x[:1], th)
    assert np.array_equal(_host(lm_out), lmt)
    reft = orc.vmm_batch(L.codes[rows], L.scales[:, rows], x[:1], lmt, levels)
    assert normwise(yt[:, rows], reft) <= TOL, (name, "threshold B=1")
    # four tokens at once (the batched kernel, per-token cross-wave sums)
    x4 = gen(K, 4, 71, K + N)
    lm4 = g.grinqh_assign(L.desc, _dev(torch, x4), g.GRINQH_ASSIGN_TOPK, counts=counts)
    y4 = _host(g.grinqh_vmm(L.desc, L.pc, L.ps, _dev(torch, x4), lm4))
    ref4 = orc.vmm_batch(L.codes[rows], L.scales[:, rows], x4, _host(lm4), levels)
    assert normwise(y4[:, rows], ref4) <= TOL, (name, "B=4")


def oracle_all_outputs(codes, scales, x, lm, levels, chunk=2048):
    """The float64 oracle over every output, a block of outputs at a time
    (the dense float64 weights of a 4096 x 28672 layer would take 0.9 GB)."""
    N = codes.shape[0]
    return np.concatenate([orc.vmm_batch(codes[n:n + chunk], scales[:, n:n + chunk], x, lm, levels)
                           for n in range(0, N, chunk)], axis=1)


def elementwise(y, ref):
    """Largest |y_n - ref_n| / max(|ref_n|, 1e-2 max|ref|) (reported, not gated)."""
    y, ref = np.asarray(y, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    den = np.maximum(np.abs(ref), 1e-2 * np.abs(ref).max(axis=-1, keepdims=True))
    return float((np.abs(y - ref) / den).max())


# every output of one full-size shape per kernel instance the benchmarks run
EVERY = [
    ("batch1 T=256 k 4096->1024", 4096, 1024, inputs.LEVELS_B, "t3", 1),
    ("batch1 T=512 qkv 4096->6144", 4096, 6144, inputs.LEVELS_B, "t3", 1),
    ("batch1 T=1024 gate|up 4096->28672", 4096, 28672, inputs.LEVELS_B, "t3", 1),
    ("batch1 T=1024 down 14336->4096", 14336, 4096, inputs.LEVELS_B, "swiglu", 1),
    ("per-plane B=2 qkv 4096->6144", 4096, 6144, inputs.LEVELS_B, "t3", 2),
    ("per-plane B=4 down 14336->4096", 14336, 4096, inputs.LEVELS_B, "swiglu", 4),
    ("1-bit planes qkv 4096->6144", 4096, 6144, inputs.LEVELS_C, "t3", 1),
    ("b_max 6 batch1 gate|up 4096->28672", 4096, 28672, (0, 2, 4, 6), "t3", 1),
    ("b_max 4 batch1 down 14336->4096", 14336, 4096, (0, 2, 4), "swiglu", 1),
]


@pytest.mark.parametrize("name,K,N,levels,xkind,B", EVERY, ids=[e[0] for e in EVERY])
def test_full_size_every_output(g, torch, name, K, N, levels, xkind, B):
    # thresholds calibrated on separate tokens (the runtime path), grading
    # fused into the VMM, level maps written out and checked bit for bit
    L = Layer(g, torch, K, N, levels, cfg=75, layer=K + N, codes_src=True)
    gen = inputs.activations_swiglu if xkind == "swiglu" else inputs.activations_t3
    x = gen(K, B, 75, K + N)
    calib = gen(K, 64, 76, K + N)
    budget = 4 if 4 in inputs.BUDGETS[tuple(levels)] else 3
    th = _host(g.grinqh_calibrate(L.desc, _dev(torch, calib), inputs.BUDGETS[tuple(levels)][budget]))
    lm_out = torch.zeros((B, K), dtype=torch.uint8, device="cuda")
    y = _host(g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, _dev(torch, x), th, level_map_out=lm_out))
    lm = orc.assign_threshold(x, th)
    assert np.array_equal(_host(lm_out), lm)
    ref = oracle_all_outputs(L.codes, L.scales, x, lm, levels)
    err = normwise(y, ref)
    print(f"{name}: normwise {err:.2e}, elementwise {elementwise(y, ref):.2e}")
    assert err <= TOL, (name, err)


def test_large_k_every_path(g, torch):
    # K = 98304 (768 groups): channel indices past 16 bits and tiles of
    # 48 MB, through the fused threshold VMM (level map written out), the
    # standalone assignment + level-map VMM, two tokens (union depth) and a
    # prefill; every output against the oracle, computed a block of outputs
    # at a time.  Thresholds come from the oracle's calibration (the GPU
    # calibration takes K <= 16384).
    K, N, levels = 98304, 1024, inputs.LEVELS_B
    L = Layer(g, torch, K, N, levels, cfg=83, layer=1, tile_n=512, codes_src=True)
    x = inputs.activations_t3(K, 2, 83, 1)
    calib = inputs.activations_t3(K, 8, 84, 1)
    th = orc.calibrate_thresholds([np.abs(r.astype(np.float64)) for r in calib], inputs.BUDGETS[levels][4])
    xd = _dev(torch, x)
    lm_out = torch.zeros((1, K), dtype=torch.uint8, device="cuda")
    y1 = _host(g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, xd[:1], th, level_map_out=lm_out))
    lm = orc.assign_threshold(x, th)
    assert np.array_equal(_host(lm_out), lm[:1])
    lm2 = g.grinqh_assign(L.desc, xd, g.GRINQH_ASSIGN_THRESHOLD, thresholds=th)
    assert np.array_equal(_host(lm2), lm)
    y2 = _host(g.grinqh_vmm(L.desc, L.pc, L.ps, xd[:1], lm2[:1]))
    yb = _host(g.grinqh_vmm(L.desc, L.pc, L.ps, xd, lm2))           # B = 2, union depth
    ref = oracle_all_outputs(L.codes, L.scales, x, lm, levels, chunk=256)
    assert normwise(y1, ref[:1]) <= TOL
    assert normwise(y2, ref[:1]) <= TOL
    assert normwise(yb, ref) <= TOL
    xp = inputs.activations_t3(K, 3, 85, 1)
    yp = _host(g.grinqh_prefill(L.desc, L.pc, L.ps, _dev(torch, xp)))
    refp = np.concatenate([orc.prefill(L.codes[n:n + 256], L.scales[:, n:n + 256], xp)
                           for n in range(0, N, 256)], axis=1)
    assert normwise(yp, refp) <= TOL


@pytest.mark.parametrize("tile_n", [512, 1024])
def test_large_n_every_path(g, torch, tile_n):
    # N = 131072 (128 or 256 tiles in one launch) over two groups, through the
    # same paths; every output against the oracle
    K, N, levels = 256, 131072, inputs.LEVELS_B
    L = Layer(g, torch, K, N, levels, cfg=86, layer=tile_n, tile_n=tile_n, codes_src=True)
    x = inputs.activations_t3(K, 2, 86, tile_n)
    calib = inputs.activations_t3(K, 16, 87, tile_n)
    th = _host(g.grinqh_calibrate(L.desc, _dev(torch, calib), inputs.BUDGETS[levels][4]))
    xd = _dev(torch, x)
    lm = orc.assign_threshold(x, th)
    y1 = _host(g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, xd[:1], th))
    lm2 = g.grinqh_assign(L.desc, xd, g.GRINQH_ASSIGN_THRESHOLD, thresholds=th)
    assert np.array_equal(_host(lm2), lm)
    yb = _host(g.grinqh_vmm(L.desc, L.pc, L.ps, xd, lm2))
    ref = oracle_all_outputs(L.codes, L.scales, x, lm, levels, chunk=16384)
    assert normwise(y1, ref[:1]) <= TOL
    assert normwise(yb, ref) <= TOL
    xp = inputs.activations_t3(K, 5, 88, tile_n)
    yp = _host(g.grinqh_prefill(L.desc, L.pc, L.ps, _dev(torch, xp)))
    assert normwise(yp, orc.prefill(L.codes, L.scales, xp)) <= TOL


def test_decode_layers_graph_replays_match_oracle(g, torch):
    # Two layers of the decode step (merged q|k|v, o, merged gate|up, down at
    # 4 bits, thresholds calibrated per input, grading fused) captured as one
    # HIP graph with the output buffer cleared inside it, replayed three times
    # with eager work and synchronisation between; every replay checked
    # against the oracle on every output of every linear.
    levels = inputs.LEVELS_B
    shapes = [("qkv", 4096, 6144, 0, "t3"), ("o", 4096, 4096, 1, "t3"),
              ("gate_up", 4096, 28672, 2, "t3"), ("down", 14336, 4096, 3, "swiglu")]
    layers = [{name: Layer(g, torch, K, N, levels, cfg=77, layer=10 * li + xin, codes_src=True)
               for name, K, N, xin, _ in shapes} for li in range(2)]
    xs, ths = {}, {}
    p = inputs.BUDGETS[levels][4]
    for name, K, N, xin, kind in shapes:
        gen = inputs.activations_swiglu if kind == "swiglu" else inputs.activations_t3
        xs[xin] = gen(K, 1, 77, xin)
        ths[xin] = _host(g.grinqh_calibrate(layers[0][name].desc, _dev(torch, gen(K, 32, 78, xin)), p))
    xd = {k: _dev(torch, v) for k, v in xs.items()}
    width = sum(N for _, _, N, _, _ in shapes)
    arena = torch.zeros(2 * width, dtype=torch.float32, device="cuda")
    outs, off = [], 0
    for li in range(2):
        per = {}
        for name, _, N, _, _ in shapes:
            per[name] = arena[off:off + N].view(1, N)
            off += N
        outs.append(per)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())

    def step():
        arena.zero_()
        for li in range(2):
            for name, _, _, xin, _ in shapes:
                Ly = layers[li][name]
                g.grinqh_vmm_threshold(Ly.desc, Ly.pc, Ly.ps, xd[xin], ths[xin], y=outs[li][name],
                                       accumulate=True)

    with torch.cuda.stream(s):
        step()
    torch.cuda.synchronize()
    refs = {}
    for li in range(2):
        for name, _, _, xin, _ in shapes:
            Ly = layers[li][name]
            lm = orc.assign_threshold(xs[xin], ths[xin])
            refs[li, name] = oracle_all_outputs(Ly.codes, Ly.scales, xs[xin], lm, levels)
    gr = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gr, stream=s):
        step()
    for rep in range(3):
        arena.fill_(float("nan"))              # eager work between replays
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            gr.replay()
        torch.cuda.synchronize()
        for li in range(2):
            for name, _, _, _, _ in shapes:
                err = normwise(_host(outs[li][name]), refs[li, name])
                assert err <= TOL, (rep, li, name, err)


def test_topk_and_prefill_graph_replays(g, torch, opts):
    # The top-k paths (selection inside the VMM, and assignment launch + VMM)
    # on a merged q|k|v and a down projection at 4 bits, and a prefill on the
    # 8-wave 256 x 256 tile, captured as one HIP graph and replayed three
    # times with eager work between: level maps bit-exact with the oracle's
    # top-k on every replay, outputs within the tolerance of the oracle, and
    # the prefill (fixed summation order) equal bit for bit to its eager run.
    levels = inputs.LEVELS_B
    p = inputs.BUDGETS[levels][4]
    shapes = [("qkv", 4096, 6144, inputs.activations_t3), ("down", 14336, 4096, inputs.activations_swiglu)]
    L = {name: Layer(g, torch, K, N, levels, cfg=81, layer=li, codes_src=True)
         for li, (name, K, N, _) in enumerate(shapes)}
    xs = {name: gen(K, 1, 81, li) for li, (name, K, _, gen) in enumerate(shapes)}
    counts = {name: g.grinqh_topk_counts(K, p) for name, K, _, _ in shapes}
    xd = {name: _dev(torch, v) for name, v in xs.items()}
    y_f = {name: torch.zeros((1, N), dtype=torch.float32, device="cuda") for name, _, N, _ in shapes}
    y_2 = {name: torch.zeros((1, N), dtype=torch.float32, device="cuda") for name, _, N, _ in shapes}
    lm_f = {name: torch.full((1, K), 255, dtype=torch.uint8, device="cuda") for name, K, _, _ in shapes}
    lm_2 = {name: torch.full((1, K), 255, dtype=torch.uint8, device="cuda") for name, K, _, _ in shapes}
    opts(g.GRINQH_OPT_PREFILL_TILE, 1)              # 256 x 256, 8 waves
    Kp, Np, M = 384, 1024, 300
    Lp = Layer(g, torch, Kp, Np, (0, 2, 4, 8), cfg=82, layer=1)
    xp = inputs.activations_t3(Kp, M, 82, 1)
    xpd = _dev(torch, xp)
    yp = torch.zeros((M, Np), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())

    def step():
        for name, _, _, _ in shapes:
            y_f[name].zero_()
            g.grinqh_vmm_topk(L[name].desc, L[name].pc, L[name].ps, xd[name], counts[name],
                              y=y_f[name], level_map_out=lm_f[name], accumulate=True)
            g.grinqh_assign(L[name].desc, xd[name], g.GRINQH_ASSIGN_TOPK, counts=counts[name],
                            out=lm_2[name])
            g.grinqh_vmm(L[name].desc, L[name].pc, L[name].ps, xd[name], lm_2[name], y=y_2[name])
        g.grinqh_prefill(Lp.desc, Lp.pc, Lp.ps, xpd, y=yp)

    with torch.cuda.stream(s):
        step()
    torch.cuda.synchronize()
    yp_eager = _host(yp).copy()
    assert normwise(yp_eager, orc.prefill(Lp.codes, Lp.scales, xp)) <= TOL
    lms, refs = {}, {}
    for name, _, _, _ in shapes:
        lms[name] = orc.assign_topk(xs[name], counts[name])
        refs[name] = oracle_all_outputs(L[name].codes, L[name].scales, xs[name], lms[name], levels)
    gr = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gr, stream=s):
        step()
    for rep in range(3):
        for name, _, _, _ in shapes:                # eager work between replays
            y_f[name].fill_(float("nan"))
            y_2[name].fill_(float("nan"))
            lm_f[name].fill_(255)
            lm_2[name].fill_(255)
        yp.fill_(float("nan"))
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            gr.replay()
        torch.cuda.synchronize()
        for name, _, _, _ in shapes:
            assert np.array_equal(_host(lm_f[name]), lms[name]), (rep, name, "fused")
            assert np.array_equal(_host(lm_2[name]), lms[name]), (rep, name, "assignment launch")
            assert normwise(_host(y_f[name]), refs[name]) <= TOL, (rep, name, "fused")
            assert normwise(_host(y_2[name]), refs[name]) <= TOL, (rep, name, "assignment launch")
        assert np.array_equal(_host(yp).view(np.uint32), yp_eager.view(np.uint32)), rep


@pytest.mark.parametrize("kernel", ["pp", "dot2"])
@pytest.mark.parametrize("gw", ["1", "2", "3", "4"])
@pytest.mark.parametrize("tile_n", [256, 512, 1024])
def test_vmm_groups_per_workgroup(g, torch, gw, tile_n, kernel, opts):
    # K = 1152 is 9 groups: every gw > 1 leaves a ragged last workgroup.  At
    # B = 1 the plane-pair kernel runs unless the per-plane kernel is forced.
    opts(g.GRINQH_OPT_GROUPS_PER_WG, gw)
    if kernel == "dot2":
        opts(g.GRINQH_OPT_VMM_KERNEL, g.GRINQH_KERNEL_PER_PLANE)
    levels = (0, 2, 4, 6, 8)
    K, N = 1152, 1024
    L = Layer(g, torch, K, N, levels, cfg=64, tile_n=tile_n)
    rng = np.random.default_rng(64)
    for B in (1, 2, 4):
        x = inputs.activations_t3(K, B, 64, B)
        lm = rng.integers(0, 5, size=(B, K)).astype(np.uint8)
        y, ref = _vmm_case(g, torch, L, x, lm)
        assert normwise(y, ref) <= TOL, (gw, tile_n, B, normwise(y, ref))


@pytest.mark.parametrize("gw", ["1", "2"])
@pytest.mark.parametrize("tile_n", [256, 512, 1024])
@pytest.mark.parametrize("levels", [(0, 2, 4, 6, 8), (0, 2, 4, 6), (0, 2, 4)])
def test_vmm_batch1_depth_classes(g, torch, gw, tile_n, levels, opts):
    # The batch-1 kernel sorts each wave's rows into those read to 3-4 planes
    # and those read to 1-2, and pads each class to whole batches: a group
    # with nothing to read, one at full depth, and random depths, for b_max
    # 8, 6 and 4, through the level-map and the fused-threshold entry points.
    # K = 1152 is 9 groups: a ragged last workgroup at gw = 2.
    opts(g.GRINQH_OPT_GROUPS_PER_WG, gw)
    K, N = 1152, 1024
    L = Layer(g, torch, K, N, levels, cfg=69, tile_n=tile_n)
    rng = np.random.default_rng(69)
    n = len(levels)
    lm = rng.integers(0, n, size=(1, K)).astype(np.uint8)
    lm[0, :128] = 0                            # a first group with nothing to read
    lm[0, 256:384] = n - 1                     # and one at full depth
    lm[0, 512:544] = 1                         # a wave slice with only shallow rows
    x = inputs.activations_t3(K, 1, 69, int(gw))
    y, ref = _vmm_case(g, torch, L, x, lm)
    assert normwise(y, ref) <= TOL, (gw, tile_n, levels, normwise(y, ref))
    # fused grading: thresholds at quantiles of |x|, level map written out
    ax = np.sort(np.abs(x[0].astype(np.float32)))
    th = ax[np.linspace(0, K - 1, n + 1).astype(int)[1:-1]]
    lm_out = torch.zeros((1, K), dtype=torch.uint8, device="cuda")
    yt = g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, _dev(torch, x), th, level_map_out=lm_out)
    torch.cuda.synchronize()
    lmt = orc.assign_threshold(x, th)
    assert np.array_equal(_host(lm_out), lmt)
    assert normwise(_host(yt), orc.vmm_batch(L.codes, L.scales, x, lmt, levels)) <= TOL


@pytest.mark.parametrize("K,N,tile_n", [(1152, 1024, 512), (4096, 4096, 512), (2048, 8192, 256)])
def test_vmm_entry_points_and_accumulate(g, torch, K, N, tile_n):
    # Both entry points on a small grid and a large one, B = 1 and B = 2,
    # and the benchmarks' call: accumulate onto a non-zero y with the level
    # map written out.
    levels = (0, 2, 4, 6, 8)
    L = Layer(g, torch, K, N, levels, cfg=73, tile_n=tile_n)
    rng = np.random.default_rng(73)
    for B in (1, 2):
        lm = rng.integers(0, len(levels), size=(B, K)).astype(np.uint8)
        x = inputs.activations_t3(K, B, 73, B)
        y = g.grinqh_vmm(L.desc, L.pc, L.ps, _dev(torch, x), _dev(torch, lm), )
        torch.cuda.synchronize()
        ref = orc.vmm_batch(L.codes, L.scales, x, lm, levels)
        assert normwise(_host(y), ref) <= TOL, (K, N, B)
        ax = np.sort(np.abs(x.astype(np.float32)).ravel())
        th = ax[np.linspace(0, ax.size - 1, len(levels) + 1).astype(int)[1:-1]]
        yt = g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, _dev(torch, x), th, )
        torch.cuda.synchronize()
        lmt = orc.assign_threshold(x, th)
        reft = orc.vmm_batch(L.codes, L.scales, x, lmt, levels)
        assert normwise(_host(yt), reft) <= TOL, (K, N, B)
        # the benchmarks' call: accumulate onto a non-zero y, level map written out
        y0 = rng.standard_normal((B, N)).astype(np.float32)
        ya = _dev(torch, y0)
        lo = torch.zeros((B, K), dtype=torch.uint8, device="cuda")
        g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, _dev(torch, x), th, y=ya, level_map_out=lo,
                               accumulate=True, )
        torch.cuda.synchronize()
        assert np.array_equal(_host(lo), lmt)
        assert normwise(_host(ya) - y0, reft) <= TOL, (K, N, B, "accumulate")


@pytest.mark.parametrize("gw", ["1", "2", "3", "4"])
@pytest.mark.parametrize("levels,tile_n", [((0, 2, 4, 6, 8), 256), ((0, 2, 4, 6, 8), 512),
                                           ((0, 2, 4, 6, 8), 1024), ((0, 2, 4, 6), 512),
                                           ((0, 2, 3, 4, 8), 512), ((0, 2, 3, 4, 8), 1024)])
def test_vmm_per_plane_depth_mix(g, torch, gw, levels, tile_n, opts):
    # The per-plane kernel (batches, 1-bit planes, and 2-bit planes at B = 1
    # when forced): per-token depths, lone last planes paired across rows
    # (odd and even counts of them), ragged workgroups (K = 1152), through
    # the level-map and the fused-threshold entry points.
    opts(g.GRINQH_OPT_GROUPS_PER_WG, gw)
    opts(g.GRINQH_OPT_VMM_KERNEL, g.GRINQH_KERNEL_PER_PLANE)
    K, N = 1152, 1024
    L = Layer(g, torch, K, N, levels, cfg=71, tile_n=tile_n)
    rng = np.random.default_rng(71)
    n = len(levels)
    for B in (1, 2, 4):
        lm = rng.integers(0, n, size=(B, K)).astype(np.uint8)
        lm[:, :128] = 0                        # a first group with nothing to read
        lm[0, 128:256] = n - 1                 # one token at full depth in the next
        x = inputs.activations_t3(K, B, 71, B)
        y, ref = _vmm_case(g, torch, L, x, lm)
        assert normwise(y, ref) <= TOL, (gw, levels, tile_n, B, normwise(y, ref))
        ax = np.sort(np.abs(x.astype(np.float32)).ravel())
        th = ax[np.linspace(0, ax.size - 1, n + 1).astype(int)[1:-1]]
        lm_out = torch.zeros((B, K), dtype=torch.uint8, device="cuda")
        yt = g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, _dev(torch, x), th, level_map_out=lm_out)
        torch.cuda.synchronize()
        lmt = orc.assign_threshold(x, th)
        assert np.array_equal(_host(lm_out), lmt)
        assert normwise(_host(yt), orc.vmm_batch(L.codes, L.scales, x, lmt, levels)) <= TOL, (gw, B)


@pytest.mark.parametrize("kernel", ["pp", "dot2"])
def test_vmm_precision_margin(g, torch, kernel, opts):
    # the contract is 1e-3; the fp32 accumulation should sit far below it
    if kernel == "dot2":
        opts(g.GRINQH_OPT_VMM_KERNEL, g.GRINQH_KERNEL_PER_PLANE)
    levels = (0, 2, 4, 6, 8)
    K, N = 4096, 1024
    L = Layer(g, torch, K, N, levels, cfg=65, tile_n=256)
    x = inputs.activations_t3(K, 2, 65)
    worst = 0.0
    for p in inputs.BUDGETS[levels].values():
        counts = g.grinqh_topk_counts(K, p)
        lm = _host(g.grinqh_assign(L.desc, _dev(torch, x), g.GRINQH_ASSIGN_TOPK, counts=counts))
        y, ref = _vmm_case(g, torch, L, x, lm)
        worst = max(worst, normwise(y, ref))
    print(f"worst normwise error {worst:.2e}")
    assert worst <= 1e-4


@pytest.mark.parametrize("tile_n", [256, 512, 1024])
@pytest.mark.parametrize("gw", ["1", "2", "4"])
def test_vmm_groups_with_no_active_channel(g, torch, tile_n, gw, opts):
    # groups whose channels are all skipped, next to active ones in the same
    # workgroup: such a group has no plane rows to read but still runs its
    # epilogue (regression: its padding once left the batch unwritten)
    opts(g.GRINQH_OPT_GROUPS_PER_WG, gw)
    levels = (0, 2, 4, 6, 8)
    K, N = 1024, 1024
    L = Layer(g, torch, K, N, levels, cfg=66, tile_n=tile_n)
    rng = np.random.default_rng(66)
    lm = rng.integers(0, 5, size=(1, K)).astype(np.uint8)
    lm[0, 128:384] = 0          # groups 1 and 2 fully skipped
    lm[0, 896:] = 0             # group 7 fully skipped
    x = inputs.activations_t3(K, 1, 66)
    y, ref = _vmm_case(g, torch, L, x, lm)
    assert normwise(y, ref) <= TOL


# --------------------------------------------------------------- prefill ----
def rowwise(y, ref):
    """Largest over rows of max_n |y - ref| / max_n |ref|."""
    y, ref = np.asarray(y, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    den = np.maximum(np.abs(ref).max(axis=1), 1e-30)
    return float((np.abs(y - ref).max(axis=1) / den).max())


def prefill_bound_ok(y, codes, scales, x):
    """Elementwise error bound of a dense fp16 GEMM over the dequantised
    weights: each weight rounds once to fp16 (relative 2^-11), products are
    exact in fp32 and K of them are summed in fp32, so
    |y - Y| <= (2^-11 + K 2^-24) sum_k |x_k| |w_hat_k| (+ a tiny absolute
    term for fp16 subnormal weights)."""
    K = x.shape[1]
    W = np.abs((codes.astype(np.float64) - 128) *
               np.repeat(np.asarray(scales, dtype=np.float16).astype(np.float64).T, 128, axis=1))
    mag = np.abs(x.astype(np.float64)) @ W.T
    ref = orc.prefill(codes, scales, x)
    gamma = 2.0 ** -11 + K * 2.0 ** -24
    slack = 2.0 ** -24 * np.abs(x.astype(np.float64)).sum(axis=1, keepdims=True)
    return bool(np.all(np.abs(np.asarray(y, dtype=np.float64) - ref) <= gamma * mag + slack))

PREFILL = [  # K, N, levels, tile_n, M
    (128, 256, (0, 2, 4, 8), 256, 1),
    (384, 512, (0, 2, 4, 8), 512, 200),
    (640, 1024, (0, 2, 4, 6, 8), 1024, 130),
    (1152, 512, (0, 2, 4, 8), 256, 257),
    (256, 2048, (0, 2, 4, 8), 2048, 64),
    (256, 2048, (0, 2, 3, 4, 8), 2048, 77),    # 1-bit planes
    (256, 1024, (0, 2, 3, 4, 8), 512, 300),    # 1-bit planes
]


@pytest.mark.parametrize("K,N,levels,tile_n,M", PREFILL)
def test_prefill_parity(g, torch, K, N, levels, tile_n, M):
    L = Layer(g, torch, K, N, levels, cfg=60, layer=K + M, tile_n=tile_n)
    assert L.desc.plane_bits == (1 if 3 in levels else 2)
    x = inputs.activations_t3(K, M, 60, K + M)
    y = _host(g.grinqh_prefill(L.desc, L.pc, L.ps, _dev(torch, x)))
    ref = orc.prefill(L.codes, L.scales, x)
    assert normwise(y, ref) <= TOL
    assert prefill_bound_ok(y, L.codes, L.scales, x)


def test_prefill_codes_source_all_code_values(g, torch):
    # uniform codes reach every byte value, including 0 and 255
    K, N, M = 512, 1024, 129
    L = Layer(g, torch, K, N, (0, 2, 4, 8), cfg=61, layer=1, codes_src=True)
    assert L.codes.min() == 0 and L.codes.max() == 255
    x = inputs.activations_swiglu(K, M, 61, 1)
    y = _host(g.grinqh_prefill(L.desc, L.pc, L.ps, _dev(torch, x)))
    assert normwise(y, orc.prefill(L.codes, L.scales, x)) <= TOL
    assert prefill_bound_ok(y, L.codes, L.scales, x)


@pytest.mark.parametrize("tile", [0, 1, 2, 3])   # automatic, then each tile forced
def test_prefill_accumulate_and_reproducible(g, torch, tile, opts):
    if tile:
        opts(g.GRINQH_OPT_PREFILL_TILE, tile)
    K, N, M = 384, 512, 150
    L = Layer(g, torch, K, N, (0, 2, 4, 8), cfg=62, layer=2)
    x = inputs.activations_t3(K, M, 62, 2)
    xd = _dev(torch, x)
    y1 = _host(g.grinqh_prefill(L.desc, L.pc, L.ps, xd))
    y2 = _host(g.grinqh_prefill(L.desc, L.pc, L.ps, xd))
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))
    base = np.random.default_rng(3).standard_normal((M, N)).astype(np.float32)
    yd = _dev(torch, base)
    g.grinqh_prefill(L.desc, L.pc, L.ps, xd, y=yd, accumulate=True)
    ref = orc.prefill(L.codes, L.scales, x) + base.astype(np.float64)
    assert normwise(_host(yd), ref) <= TOL
    # the kernel adds its sum to y once: y + base in fp32
    assert np.array_equal(_host(yd), (base + y1).astype(np.float32))


def test_prefill_rows_match_decode_at_top_level(g, torch):
    # the two stages read one packed copy: a prefill row is the decode VMM
    # with every channel at the top level
    K, N, M = 1024, 2048, 4
    levels = (0, 2, 4, 6, 8)
    L = Layer(g, torch, K, N, levels, cfg=63, layer=3)
    x = inputs.activations_t3(K, M, 63, 3)
    xd = _dev(torch, x)
    y = _host(g.grinqh_prefill(L.desc, L.pc, L.ps, xd))
    top = _dev(torch, np.full((M, K), len(levels) - 1, dtype=np.uint8))
    yv = _host(g.grinqh_vmm(L.desc, L.pc, L.ps, xd, top))
    assert normwise(y, yv) <= TOL


PREFILL_FULL = [  # name, K, N, levels, M
    ("qkv 4096->6144 M2048", 4096, 6144, inputs.LEVELS_B, 2048),
    ("gate_up 4096->28672 M512", 4096, 28672, inputs.LEVELS_B, 512),
    ("gate_up 4096->28672 M2048 (split rounds)", 4096, 28672, inputs.LEVELS_B, 2048),
    ("down 14336->4096 M300", 14336, 4096, inputs.LEVELS_B, 300),
]


@pytest.mark.parametrize("cus,K,N,levels,tile_n,M", [
    (64, 128, 5120, (0, 2, 4, 8), 512, 2048),       # 160 tiles: 128 at 256x256, then 4 columns at 256x128
    (64, 256, 5120, (0, 2, 3, 4, 8), 512, 1900),    # 1-bit planes, ragged last row block
    (80, 128, 6144, (0, 2, 4, 6, 8), 1024, 1800)])  # 192 tiles: 160, then 4 columns
def test_prefill_split_rounds(g, torch, opts, cus, K, N, levels, tile_n, M):
    """A launch whose 256x256 tiles leave a part-filled last round runs whole
    rounds at 256x256 and the remaining columns at 256x128."""
    opts(g.GRINQH_OPT_PREFILL_CUS, cus)
    L = Layer(g, torch, K, N, levels, cfg=68, tile_n=tile_n)
    x = inputs.activations_t3(K, M, 68, 3)
    y = g.grinqh_prefill(L.desc, L.pc, L.ps, _dev(torch, x))
    torch.cuda.synchronize()
    ref = orc.prefill(L.codes, L.scales, x)
    assert rowwise(_host(y), ref) <= TOL
    assert prefill_bound_ok(_host(y), L.codes, L.scales, x)
    opts(g.GRINQH_OPT_PREFILL_CUS, 0)
    y2 = g.grinqh_prefill(L.desc, L.pc, L.ps, _dev(torch, x))
    torch.cuda.synchronize()
    assert rowwise(_host(y2), _host(y)) <= 1e-6


@pytest.mark.parametrize("name,K,N,levels,M", PREFILL_FULL, ids=[f[0] for f in PREFILL_FULL])
def test_prefill_full_size_sampled(g, torch, name, K, N, levels, M):
    L = Layer(g, torch, K, N, levels, cfg=71, layer=K + N)
    gen = inputs.activations_swiglu if K > N else inputs.activations_t3
    x = gen(K, M, 71, K + N)
    y = _host(g.grinqh_prefill(L.desc, L.pc, L.ps, _dev(torch, x)))
    assert np.all(np.isfinite(y))
    r = np.random.default_rng(K + N)
    rows = np.sort(r.choice(M, size=min(M, 48), replace=False))
    cols = np.sort(r.choice(N, size=256, replace=False))
    ref = orc.prefill(L.codes[cols], L.scales[:, cols], x[rows])
    assert normwise(y[np.ix_(rows, cols)], ref) <= TOL, name
    assert prefill_bound_ok(y[np.ix_(rows, cols)], L.codes[cols], L.scales[:, cols], x[rows]), name


@pytest.mark.parametrize("tile", ["0", "1", "2"])
@pytest.mark.parametrize("K,N,levels,tile_n,M", [
    (128, 512, (0, 2, 4, 8), 256, 1),          # one group: the pipeline's tail only
    (384, 1024, (0, 2, 4, 8), 256, 300),       # ragged M over 2 or 3 row blocks
    (640, 1024, (0, 2, 3, 4, 8), 512, 257),    # 1-bit planes
    (256, 2048, (0, 2, 4, 6, 8), 2048, 64),
])
def test_prefill_tile_configs(g, torch, tile, K, N, levels, tile_n, M, opts):
    opts(g.GRINQH_OPT_PREFILL_TILE, int(tile) + 1)
    L = Layer(g, torch, K, N, levels, cfg=64, layer=K + M, tile_n=tile_n)
    x = inputs.activations_t3(K, M, 64, K + M)
    y = _host(g.grinqh_prefill(L.desc, L.pc, L.ps, _dev(torch, x)))
    assert normwise(y, orc.prefill(L.codes, L.scales, x)) <= TOL
    assert prefill_bound_ok(y, L.codes, L.scales, x)



# ------------------------------------------------ b_max = 4 and 6 storage ----
# Sec. 3.3 stores the codes at b_max in {4, 6, 8} bits; the top level reads
# all of them.  Every entry point runs on the narrower rows.
BMAX_LEVELS = [(0, 2, 4), (0, 2, 4, 6), (0, 1, 2, 3, 4), (0, 2, 3, 4, 6)]


@pytest.mark.parametrize("levels", BMAX_LEVELS)
@pytest.mark.parametrize("codes_src", [False, True])
def test_pack_bmax_bit_exact(g, torch, levels, codes_src):
    for tile_n in (0, 512, 1024):
        L = Layer(g, torch, 384, 2048, levels, cfg=80, layer=tile_n, tile_n=tile_n, codes_src=codes_src)
        assert L.desc.plane_bits == orc.plane_bits_for(levels)
        assert L.pc.numel() == 384 * 2048 * L.b_max // 8
        L.check_packed()


@pytest.mark.parametrize("levels", BMAX_LEVELS)
@pytest.mark.parametrize("kernel", ["auto", "dot2", "v0"])
def test_vmm_bmax_random_level_maps(g, torch, levels, kernel, opts):
    if kernel != "auto":
        opts(g.GRINQH_OPT_VMM_KERNEL, KERNEL[kernel])
    K, N = 1152, 1024
    L = Layer(g, torch, K, N, levels, cfg=81, codes_src=True)
    rng = np.random.default_rng(81)
    for B in (1, 2, 4):
        x = inputs.activations_t3(K, B, 81, B)
        lm = rng.integers(0, len(levels), size=(B, K)).astype(np.uint8)
        y, ref = _vmm_case(g, torch, L, x, lm)
        assert normwise(y, ref) <= TOL, (B, normwise(y, ref))
    # every channel at the top level is the plain dequantised matvec at b_max
    x = inputs.activations_t3(K, 1, 81, 9)
    top = np.full((1, K), len(levels) - 1, dtype=np.uint8)
    y, ref = _vmm_case(g, torch, L, x, top)
    assert normwise(y, ref) <= TOL


@pytest.mark.parametrize("levels", [(0, 2, 4), (0, 2, 4, 6)])
def test_vmm_bmax_topk_and_threshold(g, torch, levels):
    K, N = 4096, 4096
    L = Layer(g, torch, K, N, levels, cfg=82)
    x = inputs.activations_t3(K, 2, 82, 1)
    for p in inputs.BUDGETS[tuple(levels)].values():
        counts = g.grinqh_topk_counts(K, p)
        lm = _host(g.grinqh_assign(L.desc, _dev(torch, x), g.GRINQH_ASSIGN_TOPK, counts=counts))
        y, ref = _vmm_case(g, torch, L, x, lm)
        assert normwise(y, ref) <= TOL, p
    th = np.sort(np.abs(x[0].astype(np.float32)))[[1000, 2000, 3000][:len(levels) - 1]]
    lm_out = torch.zeros((2, K), dtype=torch.uint8, device="cuda")
    y = g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, _dev(torch, x), th, level_map_out=lm_out)
    torch.cuda.synchronize()
    lm = orc.assign_threshold(x, th)
    assert np.array_equal(_host(lm_out), lm)
    assert normwise(_host(y), orc.vmm_batch(L.codes, L.scales, x, lm, levels)) <= TOL


@pytest.mark.parametrize("levels", BMAX_LEVELS)
@pytest.mark.parametrize("tile", ["0", "1", "2"])
def test_prefill_bmax(g, torch, levels, tile, opts):
    opts(g.GRINQH_OPT_PREFILL_TILE, int(tile) + 1)
    K, N, M = 384, 1024, 200
    L = Layer(g, torch, K, N, levels, cfg=83, layer=int(tile), tile_n=512)
    x = inputs.activations_t3(K, M, 83, int(tile))
    y = _host(g.grinqh_prefill(L.desc, L.pc, L.ps, _dev(torch, x)))
    ref = orc.prefill(L.codes, L.scales, x, b_max=L.b_max)
    assert normwise(y, ref) <= TOL


# ------------------------------------------ look-up-table nested weights ----
class LutLayer:
    """Packed codes (no scales) and per-output nested tables of one layer."""

    def __init__(self, g, torch, K, N, levels, cfg=90, layer=0, tile_n=0, tables=None):
        self.desc = g.grinqh_resolve_desc(g.make_desc(K, N, levels, tile_n=tile_n))
        self.levels = tuple(levels)
        b_max = int(levels[-1])
        self.codes = inputs.random_codes(N, K, cfg, layer)
        if b_max < 8:
            self.codes = (self.codes & ((1 << b_max) - 1)).astype(np.uint8)
        self.tables = tables if tables is not None else inputs.nested_luts(N, levels, cfg, layer)
        self.pc, _ = g.grinqh_pack(self.desc, codes=_dev(torch, self.codes))
        self.luts = g.lut_table_array(self.desc, self.tables, device="cuda")
        torch.cuda.synchronize()

    def run(self, g, torch, x, lm, **kw):
        y = g.grinqh_vmm_lut(self.desc, self.pc, self.luts, _dev(torch, x), _dev(torch, lm), **kw)
        torch.cuda.synchronize()
        return _host(y)

    def ref(self, x, lm):
        return orc.vmm_lut_batch(self.codes, self.tables, x, lm, self.levels)


LUT_CASES = [  # K, N, levels, tile_n
    (1152, 1024, (0, 2, 4, 8), 256),
    (1152, 1024, (0, 2, 4, 6, 8), 512),
    (640, 2048, (0, 2, 4, 6), 1024),
    (384, 2048, (0, 2, 4), 2048),
    (640, 1024, (0, 1, 2, 3, 4), 512),
    (512, 2048, (0, 2, 3, 4, 8), 1024),
]


@pytest.mark.parametrize("K,N,levels,tile_n", LUT_CASES)
def test_vmm_lut_parity(g, torch, K, N, levels, tile_n):
    L = LutLayer(g, torch, K, N, levels, layer=K + N, tile_n=tile_n)
    rng = np.random.default_rng(K + N)
    for B in (1, 3):
        x = inputs.activations_t3(K, B, 90, B)
        lm = rng.integers(0, len(levels), size=(B, K)).astype(np.uint8)
        assert normwise(L.run(g, torch, x, lm), L.ref(x, lm)) <= TOL, B
    x = inputs.activations_t3(K, 1, 90, 7)
    top = np.full((1, K), len(levels) - 1, dtype=np.uint8)
    assert normwise(L.run(g, torch, x, top), L.ref(x, top)) <= TOL
    assert np.all(L.run(g, torch, x, np.zeros((1, K), dtype=np.uint8)) == 0.0)


@pytest.mark.parametrize("K,N,levels,tile_n", LUT_CASES)
def test_vmm_lut_threshold_fused(g, torch, K, N, levels, tile_n):
    # grading fused into the LUT VMM: levels bit-exact against the oracle's
    # threshold assignment (written out once per row), y against the oracle
    L = LutLayer(g, torch, K, N, levels, layer=K + N + 1, tile_n=tile_n)
    n = len(levels)
    for B in (1, 3):
        x = inputs.activations_t3(K, B, 91, B)
        ax = np.sort(np.abs(x.astype(np.float32)).ravel())
        th = ax[np.linspace(0, ax.size - 1, n + 1).astype(int)[1:-1]]
        lm_out = torch.full((B, K), 255, dtype=torch.uint8, device="cuda")
        y = g.grinqh_vmm_lut_threshold(L.desc, L.pc, L.luts, _dev(torch, x), th, level_map_out=lm_out)
        torch.cuda.synchronize()
        lm = orc.assign_threshold(x, th)
        assert np.array_equal(_host(lm_out), lm), B
        assert normwise(_host(y), L.ref(x, lm)) <= TOL, B


@pytest.mark.parametrize("levels", [(0, 2, 4, 8), (0, 2, 4, 6)])
def test_vmm_lut_with_uniform_tables_is_the_uniform_vmm(g, torch, levels):
    # tables holding the uniform reconstruction (one power-of-two scale per
    # output, exact in fp16) make the two GPU paths compute the same thing
    K, N = 1024, 1024
    b_max = levels[-1]
    rng = np.random.default_rng(91)
    s_out = 2.0 ** rng.integers(-9, -5, size=N).astype(np.float64)
    tables = {}
    for b in levels[1:]:
        c = np.arange(2 ** b, dtype=np.float64)
        vals = c * 2 ** (b_max - b) + orc.midpoint_bias(b, b_max) - 2 ** (b_max - 1)
        tables[b] = (s_out[:, None] * vals[None, :]).astype(np.float16)
    L = LutLayer(g, torch, K, N, levels, layer=3, tables=tables)
    sc_nk = np.repeat(s_out[:, None], K // 128, axis=1).astype(np.float16)
    pc, ps = g.grinqh_pack(L.desc, codes=_dev(torch, L.codes), scales=_dev(torch, sc_nk))
    x = inputs.activations_t3(K, 2, 91, 0)
    lm = rng.integers(0, len(levels), size=(2, K)).astype(np.uint8)
    y_lut = L.run(g, torch, x, lm)
    y_uni = _host(g.grinqh_vmm(L.desc, pc, ps, _dev(torch, x), _dev(torch, lm)))
    assert normwise(y_lut, y_uni) <= 1e-5
    assert normwise(y_lut, orc.vmm_batch(L.codes, np.ascontiguousarray(sc_nk.T), x, lm, levels)) <= TOL


@pytest.mark.parametrize("gps", ["1", "3", "16"])
def test_vmm_lut_full_size_topk(g, torch, gps, opts):
    opts(g.GRINQH_OPT_LUT_GROUPS, gps)
    K, N, levels = 4096, 4096, inputs.LEVELS_B
    L = LutLayer(g, torch, K, N, levels, layer=4)
    x = inputs.activations_t3(K, 1, 92, 0)
    counts = g.grinqh_topk_counts(K, inputs.BUDGETS[levels][4])
    lm = _host(g.grinqh_assign(L.desc, _dev(torch, x), g.GRINQH_ASSIGN_TOPK, counts=counts))
    rows = np.sort(np.random.default_rng(92).choice(N, size=128, replace=False))
    y = L.run(g, torch, x, lm)
    ref = orc.vmm_lut_batch(L.codes[rows], {b: t[rows] for b, t in L.tables.items()}, x, lm, levels)
    assert normwise(y[:, rows], ref) <= TOL


def test_vmm_lut_accumulate(g, torch):
    K, N, levels = 512, 1024, (0, 2, 4, 8)
    L = LutLayer(g, torch, K, N, levels, layer=5)
    x = inputs.activations_t3(K, 2, 93, 0)
    lm = np.random.default_rng(93).integers(0, 4, size=(2, K)).astype(np.uint8)
    base = np.random.default_rng(94).standard_normal((2, N)).astype(np.float32)
    yd = _dev(torch, base)
    L.run(g, torch, x, lm, y=yd, accumulate=True)
    assert normwise(_host(yd), L.ref(x, lm) + base) <= TOL


@pytest.mark.parametrize("levels", [(0, 2, 3, 4, 8), (0, 1, 2, 3, 4), (0, 3, 6)])
@pytest.mark.parametrize("tile_n", [512, 1024])
def test_vmm_one_bit_planes_dot2(g, torch, levels, tile_n, opts):
    # 1-bit planes through the per-plane kernel: each plane a work item at
    # its own weight, per-token depths exact for B > 1
    opts(g.GRINQH_OPT_VMM_KERNEL, g.GRINQH_KERNEL_PER_PLANE)
    K, N = 1152, 2048
    L = Layer(g, torch, K, N, levels, cfg=84, layer=tile_n, tile_n=tile_n)
    assert L.desc.plane_bits == 1
    rng = np.random.default_rng(tile_n)
    for B in (1, 2, 3, 4):
        x = inputs.activations_t3(K, B, 84, B)
        lm = rng.integers(0, len(levels), size=(B, K)).astype(np.uint8)
        y, ref = _vmm_case(g, torch, L, x, lm)
        assert normwise(y, ref) <= TOL, (B, normwise(y, ref))
    th = np.sort(np.abs(x[0].astype(np.float32)))[[300, 600, 900, 1100][:len(levels) - 1]]
    y = g.grinqh_vmm_threshold(L.desc, L.pc, L.ps, _dev(torch, x), th)
    torch.cuda.synchronize()
    assert normwise(_host(y), orc.vmm_batch(L.codes, L.scales, x, orc.assign_threshold(x, th), levels)) <= TOL
