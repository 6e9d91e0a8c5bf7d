"""grinqh_calibrate_noalloc, the calibration entry point that allocates
nothing (its per-sample scratch is a static device array of the library),
against grinqh_calibrate with a caller-provided scratch, through the C ABI.
Two calls in a row, the second with fewer samples and a smaller K: the
static scratch keeps the first call's contents, and the result must not
depend on them."""
import ctypes

import numpy as np
import pytest

from synth import inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def g():
    from paper_2606_23419_amd import grinqh
    return grinqh


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


def _both(g, torch, K, S, levels, p, seed):
    d = g.grinqh_resolve_desc(g.make_desc(K, 512, levels))
    x = torch.from_numpy(inputs.activations_t3(K, S, 90, seed)).cuda()
    n = len(levels) - 1
    per_sample = torch.empty((S, n), dtype=torch.float64, device="cuda")
    want = g.grinqh_calibrate(d, x, p, per_sample=per_sample)
    # the no-alloc entry point called through the C ABI directly
    theta = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
    arr = (ctypes.c_int32 * len(p))(*p)
    st = g.lib.grinqh_calibrate_noalloc(ctypes.byref(d), ctypes.c_void_p(x.data_ptr()), S, arr,
                                         ctypes.c_void_p(theta.data_ptr()),
                                         ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, g.grinqh_last_error()
    torch.cuda.synchronize()
    return want.cpu().numpy(), theta.cpu().numpy()


def test_calibrate_noalloc_matches_workspace_entry_point(g, torch):
    # first call: many samples, large K (fills much of the scratch)
    a, b = _both(g, torch, 4096, 4096, (0, 2, 4, 6, 8), (2000, 800, 2400, 4800, 0), 1)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    # second call: fewer samples, smaller K, other levels; stale entries of
    # the first call sit beyond what it writes and must not be read
    a, b = _both(g, torch, 1024, 7, (0, 2, 4, 8), (2000, 2000, 3000, 3000), 2)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert np.all(np.isfinite(b))


def test_calibrate_noalloc_rejects_oversize(g, torch):
    d = g.grinqh_resolve_desc(g.make_desc(1024, 512, (0, 2, 4, 6, 8)))
    x = torch.zeros((32769, 1024), dtype=torch.float16, device="cuda")   # 32769 * 4 > 131072
    with pytest.raises(g.GrinqhError) as e:
        g.grinqh_calibrate_noalloc(d, x, (2000, 800, 2400, 4800, 0))
    assert e.value.status == g.GRINQH_ESIZE
    assert "static scratch" in g.grinqh_last_error()
