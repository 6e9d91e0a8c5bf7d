"""Thin Python binding of libgrinqh (argument marshalling only).

Every function has the name of the C entry point it calls (include/grinqh.h)
and does no arithmetic of the method: it checks tensor dtypes, devices and
shapes, allocates outputs with torch (device memory is plumbing here), passes
raw pointers and the current HIP stream, and turns a negative status into
``GrinqhError``.  There is no fallback: if libgrinqh.so is missing or fails to
load, importing this module raises.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgrinqh.so")

GRINQH_OK = 0
GRINQH_EINVAL = -1
GRINQH_EUNSUPPORTED = -2
GRINQH_ESIZE = -3
GRINQH_EHIP = -4
GRINQH_SRC_FP16_RTN = 0
GRINQH_SRC_CODES_U8 = 1
GRINQH_ASSIGN_THRESHOLD = 0
GRINQH_ASSIGN_TOPK = 1
GRINQH_VMM_ACCUMULATE = 1
GRINQH_OPT_VMM_KERNEL = 1
GRINQH_OPT_GROUPS_PER_WG = 2
GRINQH_OPT_PREFILL_TILE = 3
GRINQH_OPT_LUT_GROUPS = 4
GRINQH_OPT_PREFILL_CUS = 5
GRINQH_KERNEL_AUTO = 0
GRINQH_KERNEL_PER_PLANE = 1
GRINQH_KERNEL_GENERAL = 2
MAX_LEVELS = 9

EXPORTED = (
    "grinqh_resolve_desc", "grinqh_packed_bytes", "grinqh_pack", "grinqh_topk_counts",
    "grinqh_workspace_bytes", "grinqh_calibrate", "grinqh_assign", "grinqh_vmm",
    "grinqh_vmm_threshold", "grinqh_prefill", "grinqh_lut_entries", "grinqh_vmm_lut",
    "grinqh_vmm_lut_threshold", "grinqh_set_option", "grinqh_calibrate_noalloc",
    "grinqh_stream_read", "grinqh_vmm_topk", "grinqh_last_error",
)


class GrinqhError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"grinqh status {status}: {message}")
        self.status = status


class LayerDesc(ctypes.Structure):
    _fields_ = [
        ("K", ctypes.c_int32), ("N", ctypes.c_int32), ("group", ctypes.c_int32),
        ("n_levels", ctypes.c_int32), ("level_bits", ctypes.c_uint8 * MAX_LEVELS),
        ("reserved_", ctypes.c_uint8 * 3), ("plane_bits", ctypes.c_int32),
        ("tile_n", ctypes.c_int32),
    ]

    def levels(self):
        return tuple(int(self.level_bits[i]) for i in range(self.n_levels))

    def __repr__(self):
        return (f"LayerDesc(K={self.K}, N={self.N}, levels={self.levels()}, "
                f"plane_bits={self.plane_bits}, tile_n={self.tile_n})")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2606_23419_amd.build.build()")
    lib = ctypes.CDLL(LIB_PATH)
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    dp = ctypes.POINTER(LayerDesc)
    i32 = ctypes.c_int32
    sig = {
        "grinqh_resolve_desc": [dp, dp],
        "grinqh_packed_bytes": [dp, ctypes.POINTER(sz), ctypes.POINTER(sz)],
        "grinqh_pack": [dp, ctypes.c_int, vp, vp, vp, vp, vp],
        "grinqh_topk_counts": [i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)],
        "grinqh_workspace_bytes": [dp, i32, ctypes.POINTER(sz)],
        "grinqh_calibrate": [dp, vp, i32, ctypes.POINTER(i32), vp, vp, vp],
        "grinqh_assign": [dp, ctypes.c_int, vp, i32, ctypes.POINTER(ctypes.c_float),
                          ctypes.POINTER(i32), vp, vp, sz, vp],
        "grinqh_vmm": [dp, vp, vp, vp, vp, i32, vp, i32, vp, sz, vp],
        "grinqh_vmm_threshold": [dp, vp, vp, vp, i32, ctypes.POINTER(ctypes.c_float), vp, vp,
                                 i32, vp, sz, vp],
        "grinqh_prefill": [dp, vp, vp, vp, i32, vp, i32, vp],
        "grinqh_lut_entries": [dp, ctypes.POINTER(sz)],
        "grinqh_vmm_lut": [dp, vp, vp, vp, vp, i32, vp, i32, vp],
        "grinqh_vmm_lut_threshold": [dp, vp, vp, vp, i32, ctypes.POINTER(ctypes.c_float), vp, vp, i32, vp],
        "grinqh_set_option": [ctypes.c_int, ctypes.c_int],
        "grinqh_calibrate_noalloc": [dp, vp, i32, ctypes.POINTER(i32), vp, vp],
        "grinqh_stream_read": [vp, sz, vp, vp],
        "grinqh_vmm_topk": [dp, vp, vp, vp, i32, ctypes.POINTER(i32), vp, vp, i32, vp, sz, vp],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.grinqh_last_error.argtypes = []
    lib.grinqh_last_error.restype = ctypes.c_char_p
    return lib


lib = _load()


def _check(status: int):
    if status != GRINQH_OK:
        raise GrinqhError(status, lib.grinqh_last_error().decode())


def make_desc(K: int, N: int, level_bits, plane_bits: int = 0, tile_n: int = 0,
              group: int = 128) -> LayerDesc:
    d = LayerDesc()
    d.K, d.N, d.group = int(K), int(N), int(group)
    lb = [int(b) for b in level_bits]
    d.n_levels = len(lb)
    for i, b in enumerate(lb[:MAX_LEVELS]):
        d.level_bits[i] = b
    d.plane_bits, d.tile_n = int(plane_bits), int(tile_n)
    return d


def grinqh_last_error() -> str:
    return lib.grinqh_last_error().decode()


def grinqh_set_option(option: int, value: int) -> None:
    """Process-wide launch override for tests and measurements (see grinqh.h)."""
    _check(lib.grinqh_set_option(int(option), int(value)))


def _host_array(vals, n, ctype, name):
    """A ctypes array of exactly n host values: the C side reads n entries."""
    vals = list(vals)
    if len(vals) != n:
        raise ValueError(f"{name} has {len(vals)} entries, expected {n}")
    return (ctype * n)(*vals)


def grinqh_resolve_desc(desc: LayerDesc) -> LayerDesc:
    out = LayerDesc()
    _check(lib.grinqh_resolve_desc(ctypes.byref(desc), ctypes.byref(out)))
    return out


def grinqh_packed_bytes(desc: LayerDesc):
    c, s = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib.grinqh_packed_bytes(ctypes.byref(desc), ctypes.byref(c), ctypes.byref(s)))
    return int(c.value), int(s.value)


def grinqh_topk_counts(K: int, p_bp):
    n = len(p_bp)
    arr = _host_array([int(v) for v in p_bp], n, ctypes.c_int32, "p_bp")
    out = (ctypes.c_int32 * n)()
    _check(lib.grinqh_topk_counts(int(K), n, arr, out))
    return [int(v) for v in out]


def grinqh_workspace_bytes(desc: LayerDesc, B: int) -> int:
    b = ctypes.c_size_t()
    _check(lib.grinqh_workspace_bytes(ctypes.byref(desc), int(B), ctypes.byref(b)))
    return int(b.value)


# ----------------------------------------------------------- device calls --
def _torch():
    import torch
    return torch


def _dev(t, dtype, name, shape=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def grinqh_pack(desc: LayerDesc, W=None, codes=None, scales=None, out_codes=None,
                out_scales=None, stream=None):
    """Pack fp16 W[N, K] (RTN inside) or uint8 codes[N, K] + fp16 scales[N, K/128].

    Returns (packed_codes uint8 [K*N], packed_scales fp16 [K/128, N])."""
    torch = _torch()
    rd = grinqh_resolve_desc(desc)
    nc, ns = grinqh_packed_bytes(rd)
    if (W is None) == (codes is None):
        raise ValueError("pass exactly one of W and codes")
    ref = W if W is not None else codes
    dev = ref.device
    if out_codes is None:
        out_codes = torch.empty(nc, dtype=torch.uint8, device=dev)
    if out_scales is None:
        out_scales = torch.empty((rd.K // 128, rd.N), dtype=torch.float16, device=dev)
    pc = _dev(out_codes, torch.uint8, "out_codes", (nc,))
    ps = _dev(out_scales, torch.float16, "out_scales", (rd.K // 128, rd.N))
    if W is not None:
        src = _dev(W, torch.float16, "W", (rd.N, rd.K))
        st = lib.grinqh_pack(ctypes.byref(rd), GRINQH_SRC_FP16_RTN, src, None, pc, ps,
                             _stream(stream))
    else:
        src = _dev(codes, torch.uint8, "codes", (rd.N, rd.K))
        sc = _dev(scales, torch.float16, "scales", (rd.N, rd.K // 128)) if scales is not None else None
        st = lib.grinqh_pack(ctypes.byref(rd), GRINQH_SRC_CODES_U8, src, sc, pc,
                             ps if scales is not None else None, _stream(stream))
    _check(st)
    return out_codes, out_scales


def _thresholds(rd, vals):
    return _host_array([float(v) for v in vals], rd.n_levels - 1, ctypes.c_float, "thresholds")


def grinqh_calibrate(desc: LayerDesc, x, p_bp, per_sample=None, theta=None, stream=None):
    """Thresholds theta_1..theta_n (fp32 device tensor) calibrated on the fp16
    samples x [S, K] for the precision distribution p_bp (basis points)."""
    torch = _torch()
    rd = grinqh_resolve_desc(desc)
    if x.dim() == 1:
        x = x.view(1, -1)
    S = int(x.shape[0])
    n = rd.n_levels - 1
    xp = _dev(x, torch.float16, "x", (S, rd.K))
    if per_sample is None:
        per_sample = torch.empty((S, n), dtype=torch.float64, device=x.device)
    if theta is None:
        theta = torch.empty((n,), dtype=torch.float32, device=x.device)
    pp = _dev(per_sample, torch.float64, "per_sample", (S, n))
    tp = _dev(theta, torch.float32, "theta", (n,))
    arr = _host_array([int(v) for v in p_bp], rd.n_levels, ctypes.c_int32, "p_bp")
    _check(lib.grinqh_calibrate(ctypes.byref(rd), xp, S, arr, pp, tp, _stream(stream)))
    return theta


def grinqh_calibrate_noalloc(desc: LayerDesc, x, p_bp, theta=None, stream=None):
    """grinqh_calibrate with the library's static scratch: no workspace is
    passed (theta is allocated here only when the caller passes none)."""
    torch = _torch()
    rd = grinqh_resolve_desc(desc)
    if x.dim() == 1:
        x = x.view(1, -1)
    S = int(x.shape[0])
    n = rd.n_levels - 1
    xp = _dev(x, torch.float16, "x", (S, rd.K))
    if theta is None:
        theta = torch.empty((n,), dtype=torch.float32, device=x.device)
    tp = _dev(theta, torch.float32, "theta", (n,))
    arr = _host_array([int(v) for v in p_bp], rd.n_levels, ctypes.c_int32, "p_bp")
    _check(lib.grinqh_calibrate_noalloc(ctypes.byref(rd), xp, S, arr, tp, _stream(stream)))
    return theta


def grinqh_assign(desc: LayerDesc, x, mode: int, thresholds=None, counts=None, out=None,
                  stream=None):
    """Level map uint8 [B, K] for fp16 x [B, K] (threshold or top-k mode)."""
    torch = _torch()
    rd = grinqh_resolve_desc(desc)
    if x.dim() == 1:
        x = x.view(1, -1)
    B = int(x.shape[0])
    xp = _dev(x, torch.float16, "x", (B, rd.K))
    if out is None:
        out = torch.empty((B, rd.K), dtype=torch.uint8, device=x.device)
    op = _dev(out, torch.uint8, "out", (B, rd.K))
    th = _thresholds(rd, thresholds) if thresholds is not None else None
    cn = _host_array([int(c) for c in counts], rd.n_levels, ctypes.c_int32, "counts") \
        if counts is not None else None
    _check(lib.grinqh_assign(ctypes.byref(rd), int(mode), xp, B, th, cn, op, None, 0,
                             _stream(stream)))
    return out


def _vmm_flags(accumulate):
    return GRINQH_VMM_ACCUMULATE if accumulate else 0


def grinqh_vmm(desc: LayerDesc, packed_codes, packed_scales, x, level_map, y=None,
               accumulate: bool = False, stream=None):
    """y fp32 [B, N] = nested-precision VMM of fp16 x [B, K] with level_map [B, K]."""
    torch = _torch()
    rd = grinqh_resolve_desc(desc)
    if x.dim() == 1:
        x = x.view(1, -1)
    if level_map.dim() == 1:
        level_map = level_map.view(1, -1)
    B = int(x.shape[0])
    cp = _dev(packed_codes, torch.uint8, "packed_codes", (rd.K * rd.N * rd.level_bits[rd.n_levels - 1] // 8,))
    sp = _dev(packed_scales, torch.float16, "packed_scales", (rd.K // 128, rd.N))
    xp = _dev(x, torch.float16, "x", (B, rd.K))
    lp = _dev(level_map, torch.uint8, "level_map", (B, rd.K))
    if y is None:
        y = torch.empty((B, rd.N), dtype=torch.float32, device=x.device)
    yp = _dev(y, torch.float32, "y", (B, rd.N))
    flags = _vmm_flags(accumulate)
    _check(lib.grinqh_vmm(ctypes.byref(rd), cp, sp, xp, lp, B, yp, flags, None, 0,
                          _stream(stream)))
    return y


def grinqh_vmm_threshold(desc: LayerDesc, packed_codes, packed_scales, x, thresholds, y=None,
                         level_map_out=None, accumulate: bool = False, stream=None):
    """The VMM with threshold grading fused in; optionally writes the level map."""
    torch = _torch()
    rd = grinqh_resolve_desc(desc)
    if x.dim() == 1:
        x = x.view(1, -1)
    B = int(x.shape[0])
    cp = _dev(packed_codes, torch.uint8, "packed_codes", (rd.K * rd.N * rd.level_bits[rd.n_levels - 1] // 8,))
    sp = _dev(packed_scales, torch.float16, "packed_scales", (rd.K // 128, rd.N))
    xp = _dev(x, torch.float16, "x", (B, rd.K))
    lo = _dev(level_map_out, torch.uint8, "level_map_out", (B, rd.K)) \
        if level_map_out is not None else None
    if y is None:
        y = torch.empty((B, rd.N), dtype=torch.float32, device=x.device)
    yp = _dev(y, torch.float32, "y", (B, rd.N))
    flags = _vmm_flags(accumulate)
    _check(lib.grinqh_vmm_threshold(ctypes.byref(rd), cp, sp, xp, B, _thresholds(rd, thresholds), lo,
                                    yp, flags, None, 0, _stream(stream)))
    return y


def grinqh_vmm_topk(desc: LayerDesc, packed_codes, packed_scales, x, counts, y=None,
                    level_map_out=None, accumulate: bool = False, stream=None):
    """The batch-1 VMM with exact top-k assignment fused in (counts per level,
    summing to K); optionally writes the level map."""
    torch = _torch()
    rd = grinqh_resolve_desc(desc)
    if x.dim() == 1:
        x = x.view(1, -1)
    B = int(x.shape[0])
    cp = _dev(packed_codes, torch.uint8, "packed_codes", (rd.K * rd.N * rd.level_bits[rd.n_levels - 1] // 8,))
    sp = _dev(packed_scales, torch.float16, "packed_scales", (rd.K // 128, rd.N))
    xp = _dev(x, torch.float16, "x", (B, rd.K))
    cn = _host_array([int(c) for c in counts], rd.n_levels, ctypes.c_int32, "counts")
    lo = _dev(level_map_out, torch.uint8, "level_map_out", (B, rd.K)) \
        if level_map_out is not None else None
    if y is None:
        y = torch.empty((B, rd.N), dtype=torch.float32, device=x.device)
    yp = _dev(y, torch.float32, "y", (B, rd.N))
    flags = _vmm_flags(accumulate)
    _check(lib.grinqh_vmm_topk(ctypes.byref(rd), cp, sp, xp, B, cn, lo, yp, flags, None, 0,
                               _stream(stream)))
    return y


def grinqh_prefill(desc: LayerDesc, packed_codes, packed_scales, x, y=None,
                   accumulate: bool = False, stream=None):
    """Y fp32 [M, N] = X W_hat^T at all 8 bits for fp16 X [M, K] (prefill)."""
    torch = _torch()
    rd = grinqh_resolve_desc(desc)
    if x.dim() == 1:
        x = x.view(1, -1)
    M = int(x.shape[0])
    cp = _dev(packed_codes, torch.uint8, "packed_codes", (rd.K * rd.N * rd.level_bits[rd.n_levels - 1] // 8,))
    sp = _dev(packed_scales, torch.float16, "packed_scales", (rd.K // 128, rd.N))
    xp = _dev(x, torch.float16, "x", (M, rd.K))
    if y is None:
        y = torch.empty((M, rd.N), dtype=torch.float32, device=x.device)
    yp = _dev(y, torch.float32, "y", (M, rd.N))
    flags = GRINQH_VMM_ACCUMULATE if accumulate else 0
    _check(lib.grinqh_prefill(ctypes.byref(rd), cp, sp, xp, M, yp, flags, _stream(stream)))
    return y


def grinqh_lut_entries(desc: LayerDesc) -> int:
    n = ctypes.c_size_t()
    _check(lib.grinqh_lut_entries(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def lut_table_array(desc: LayerDesc, tables, device=None):
    """Concatenate per-level fp16 tables {b: [N, 2^b]} in level order into
    the 1-D table array of grinqh_vmm_lut (host-side layout helper)."""
    torch = _torch()
    rd = grinqh_resolve_desc(desc)
    parts = [torch.as_tensor(tables[int(rd.level_bits[l])]).reshape(-1)
             for l in range(1, rd.n_levels)]
    out = torch.cat(parts).to(torch.float16)
    assert out.numel() == grinqh_lut_entries(rd)
    return out.to(device) if device is not None else out


def grinqh_vmm_lut(desc: LayerDesc, packed_codes, luts, x, level_map, y=None,
                   accumulate: bool = False, stream=None):
    """y fp32 [B, N] of the look-up-table nested VMM (see grinqh.h)."""
    torch = _torch()
    rd = grinqh_resolve_desc(desc)
    if x.dim() == 1:
        x = x.view(1, -1)
    if level_map.dim() == 1:
        level_map = level_map.view(1, -1)
    B = int(x.shape[0])
    cp = _dev(packed_codes, torch.uint8, "packed_codes",
              (rd.K * rd.N * rd.level_bits[rd.n_levels - 1] // 8,))
    lp = _dev(luts, torch.float16, "luts", (grinqh_lut_entries(rd),))
    xp = _dev(x, torch.float16, "x", (B, rd.K))
    mp = _dev(level_map, torch.uint8, "level_map", (B, rd.K))
    if y is None:
        y = torch.empty((B, rd.N), dtype=torch.float32, device=x.device)
    yp = _dev(y, torch.float32, "y", (B, rd.N))
    flags = GRINQH_VMM_ACCUMULATE if accumulate else 0
    _check(lib.grinqh_vmm_lut(ctypes.byref(rd), cp, lp, xp, mp, B, yp, flags, _stream(stream)))
    return y


def grinqh_vmm_lut_threshold(desc: LayerDesc, packed_codes, luts, x, thresholds, y=None,
                             level_map_out=None, accumulate: bool = False, stream=None):
    """The LUT VMM with threshold grading fused in; optionally writes the level map."""
    torch = _torch()
    rd = grinqh_resolve_desc(desc)
    if x.dim() == 1:
        x = x.view(1, -1)
    B = int(x.shape[0])
    cp = _dev(packed_codes, torch.uint8, "packed_codes",
              (rd.K * rd.N * rd.level_bits[rd.n_levels - 1] // 8,))
    lp = _dev(luts, torch.float16, "luts", (grinqh_lut_entries(rd),))
    xp = _dev(x, torch.float16, "x", (B, rd.K))
    lo = _dev(level_map_out, torch.uint8, "level_map_out", (B, rd.K)) \
        if level_map_out is not None else None
    if y is None:
        y = torch.empty((B, rd.N), dtype=torch.float32, device=x.device)
    yp = _dev(y, torch.float32, "y", (B, rd.N))
    flags = GRINQH_VMM_ACCUMULATE if accumulate else 0
    _check(lib.grinqh_vmm_lut_threshold(ctypes.byref(rd), cp, lp, xp, B, _thresholds(rd, thresholds), lo, yp,
                                        flags, _stream(stream)))
    return y


def grinqh_stream_read(src, sink, stream=None):
    """Stream-read the uint8 device tensor src (measurement infrastructure)."""
    torch = _torch()
    sp = _dev(src, torch.uint8, "src")
    kp = _dev(sink, torch.int32, "sink", (1,))
    _check(lib.grinqh_stream_read(sp, src.numel(), kp, _stream(stream)))
