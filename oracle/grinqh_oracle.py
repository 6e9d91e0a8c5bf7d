"""CPU oracle for GRINQH's nested-precision decode VMM.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  It shares no code
with the GPU library (``paper_2606_23419_amd``) and imports nothing from it.

It is a plain, slow, obviously correct statement of what the hot path computes,
in numpy with float64 wherever floating point is involved, following the paper
(GRINQH, arXiv 2606.23419) step by step:

1. uniform symmetric RTN quantisation at b_max = 8 bits, group size G = 128
   along the input dimension (Sec. 3.3 "Storage Layout and Weight Loading";
   Sec. 4 "Models and Baselines": symmetric configurations, G = 128);
2. nesting: the b-bit code is the b most significant bits of the 8-bit code
   (Sec. 3.3; App. E.1: truncation, i.e. slicing, instead of rounding);
3. reconstruction with the midpoint bias term,
   w_hat = s * (q_b * 2^(b_max - b) + phi) + z, phi = 2^(b_max - b - 1)
   (Sec. 3.3 "Weight Reconstruction and Bias Correction");
4. per-token precision assignment, either by thresholds (Sec. 3.1: b_i = b_k
   iff |x_i| lies in [theta_k, theta_(k+1)), theta_0 = 0, theta_(n+1) = inf) or
   by the top-p partition of |x| into the fractions P (App. A.1);
5. the matvec y = W_hat x, accumulated in float64 (a skipped channel, level 0,
   contributes nothing: Sec. 3, "bypassing the loading");
6. the packed nested layout, written from the layout definition below, so the
   GPU packer's bytes can be compared byte for byte.

Readings taken where the paper is silent or inconsistent:

* R1  phi at b = b_max is 0: no bits are dropped, so there is no floor to undo.
* R2  level 0 contributes exactly 0 (skip), not s*phi + z.
* R3  symmetric, offset-binary codes: q in [0, 255], z = -128 s.
* R4  RTN: s = fp16_rne(fp32(max|w|) / 127); q = clamp(rint_half_even(
      fp32(w) / fp32(s)), -128, 127) + 128; a group with s == 0 gets q = 128.
* R5  groups of 128 consecutive input channels, one scale per (group, output).
* R6  n interior thresholds theta_1..theta_n (non-decreasing fp32), compared
      against |x| widened exactly from fp16 to fp32; equality goes to the
      higher level (left-closed intervals).
* R7  top-k order: |x| descending, ties broken by the lower channel index.
* R8  P (basis points) -> integer counts: with U_j = sum_{i >= j} p_i,
      C_j = floor((U_j * K + 5000) / 10000) channels are at level >= j.
* R9  bit planes of uniform width u (2, or 1 when a level width is odd);
      a depth-b read loads the first b/u planes of the row (Sec. 3.3 uses
      u = 2; the odd level set {0,2,3,4,8} needs u = 1).
* R10 phi is the paper's 2^(b_max - b - 1), half a b-bit bin above the floor,
      not the exact centre of the integer bin.
* R19 b_max is the top level's width (the paper's b_n = b_max) and may be 4,
      6 or 8 (Sec. 3.3 evaluates all three): RTN divides by 2^(b_max-1) - 1,
      codes are offset by 2^(b_max-1), phi is 0 at b = b_max, and a stored
      row holds b_max/u planes (tile_n * b_max / 8 bytes).
"""
from __future__ import annotations

import numpy as np

B_MAX = 8            # the default b_max; 4 and 6 are also stored (Sec. 3.3; R19)
OFFSET = 128          # z = -OFFSET * s at b_max = 8; 2^(b_max-1) in general (R3)


# ---------------------------------------------------------------------------
# 1. RTN quantisation (Sec. 3.3 / Sec. 4; readings R3, R4, R5)
# ---------------------------------------------------------------------------
def rtn_quantize(W16: np.ndarray, group: int = 128, b_max: int = B_MAX):
    """Quantise fp16 weights W[N, K] to b_max-bit offset-binary codes (R4):
    s = fp16(fp32(max|w|) / (2^(b_max-1) - 1)), q = clamp(rint(w / s),
    -2^(b_max-1), 2^(b_max-1) - 1) + 2^(b_max-1).

    Returns (codes uint8 [N, K], scales fp16 [K // group, N]).
    """
    W16 = np.asarray(W16, dtype=np.float16)
    N, K = W16.shape
    assert K % group == 0
    half = 2 ** (b_max - 1)
    G = K // group
    w32 = W16.astype(np.float32).reshape(N, G, group)
    amax = np.max(np.abs(w32), axis=2)                                   # fp32 [N, G]
    s16 = (amax / np.float32(half - 1)).astype(np.float32).astype(np.float16)
    s32 = s16.astype(np.float32)
    zero = (s32 == 0.0)[:, :, None]
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.rint(w32 / s32[:, :, None])                 # fp32 IEEE divide, half-even
    r = np.clip(np.where(zero, 0.0, r), -half, half - 1)   # a zero-scale group -> code 2^(b_max-1)
    codes = (r.astype(np.int32) + half).astype(np.uint8)
    return codes.reshape(N, K), np.ascontiguousarray(s16.T)


# ---------------------------------------------------------------------------
# 2./3. Nesting and reconstruction (Sec. 3.3; readings R1, R2, R10)
# ---------------------------------------------------------------------------
def nested_code(q: np.ndarray, b: int, b_max: int = B_MAX) -> np.ndarray:
    """q_b: the integer formed by the b most significant bits of the b_max-bit q."""
    q = np.asarray(q, dtype=np.int64)
    return q >> (b_max - b)


def midpoint_bias(b: int, b_max: int = B_MAX) -> float:
    """phi for a b-bit read: 2^(b_max - b - 1), and 0 at full depth (R1)."""
    if b >= b_max:
        return 0.0
    return float(2 ** (b_max - b - 1))


def reconstruct(q: np.ndarray, s: np.ndarray, b: int, b_max: int = B_MAX) -> np.ndarray:
    """w_hat = s * (q_b * 2^(b_max - b) + phi) + z with z = -2^(b_max-1) s (float64).

    b = 0 is a skipped channel and reconstructs to exactly 0 (R2).
    """
    s = np.asarray(s, dtype=np.float64)
    if b == 0:
        return np.zeros(np.broadcast(np.asarray(q), s).shape, dtype=np.float64)
    qb = nested_code(q, b, b_max).astype(np.float64)
    z = -float(2 ** (b_max - 1)) * s
    return s * (qb * float(2 ** (b_max - b)) + midpoint_bias(b, b_max)) + z


# ---------------------------------------------------------------------------
# 4. Precision assignment (Sec. 3.1 and App. A.1; readings R6, R7, R8)
# ---------------------------------------------------------------------------
def magnitude_key(x16: np.ndarray) -> np.ndarray:
    """Integer key whose order is the order of |x| for finite fp16 x."""
    bits = np.asarray(x16, dtype=np.float16).view(np.uint16).astype(np.int64)
    return bits & 0x7FFF


def assign_threshold(x16: np.ndarray, thetas) -> np.ndarray:
    """Level index per channel: the k with |x| in [theta_k, theta_(k+1)).

    ``thetas`` are the n interior thresholds theta_1..theta_n (fp32); the
    boundary thresholds theta_0 = 0 and theta_(n+1) = +inf are added here.
    """
    th = [0.0] + [float(np.float32(t)) for t in thetas] + [np.inf]
    n = len(th) - 2
    ax = np.abs(np.asarray(x16, dtype=np.float16).astype(np.float32)).astype(np.float64)
    out = np.zeros(ax.shape, dtype=np.uint8)
    for k in range(n + 1):
        inside = (th[k] <= ax) & (ax < th[k + 1])
        out[inside] = k
    return out


def topk_counts(K: int, p_bp) -> np.ndarray:
    """Per-level channel counts c_0..c_n for distribution P in basis points (R8)."""
    p_bp = [int(v) for v in p_bp]
    assert sum(p_bp) == 10000 and all(v >= 0 for v in p_bp)
    n = len(p_bp) - 1
    C = [0] * (n + 2)
    for j in range(n + 1):
        U = sum(p_bp[j:])
        C[j] = (U * K + 5000) // 10000
    C[n + 1] = 0
    return np.array([C[j] - C[j + 1] for j in range(n + 1)], dtype=np.int64)


def assign_topk(x16: np.ndarray, counts) -> np.ndarray:
    """Top-p partition of |x| (App. A.1): the c_n largest magnitudes get level n,
    the next c_(n-1) get level n-1, and so on; ties go to the lower index (R7)."""
    x16 = np.asarray(x16, dtype=np.float16)
    counts = [int(c) for c in counts]
    K = x16.shape[-1]
    assert sum(counts) == K
    n = len(counts) - 1
    level_of_rank = np.empty(K, dtype=np.uint8)
    r = 0
    for j in range(n, -1, -1):
        level_of_rank[r:r + counts[j]] = j
        r += counts[j]
    flat = x16.reshape(-1, K)
    out = np.empty(flat.shape, dtype=np.uint8)
    idx = np.arange(K)
    for t in range(flat.shape[0]):
        key = magnitude_key(flat[t])
        order = np.lexsort((idx, -key))        # primary: key descending; then index
        out[t, order] = level_of_rank
    return out.reshape(x16.shape)


# ---------------------------------------------------------------------------
# 5. Dequantise and matvec (Sec. 3.3 reconstruction; float64 accumulation)
# ---------------------------------------------------------------------------
def dequantize(codes: np.ndarray, scales: np.ndarray, levels: np.ndarray,
               level_bits, group: int = 128) -> np.ndarray:
    """W_hat[n, k] for one token's level map (float64 [N, K]).  The top
    level's width is b_max (the paper's b_n = b_max, Sec. 3.1)."""
    b_max = int(level_bits[-1])
    codes = np.asarray(codes)
    N, K = codes.shape
    s_full = np.repeat(np.asarray(scales, dtype=np.float16).astype(np.float64).T,
                       group, axis=1)                          # [N, K]
    W = np.zeros((N, K), dtype=np.float64)
    levels = np.asarray(levels).reshape(K)
    for lvl, b in enumerate(level_bits):
        cols = np.nonzero(levels == lvl)[0]
        if cols.size == 0 or b == 0:
            continue
        W[:, cols] = reconstruct(codes[:, cols], s_full[:, cols], int(b), b_max)
    return W


def vmm(codes, scales, x16, levels, level_bits, group: int = 128) -> np.ndarray:
    """y = W_hat(levels) x for one token (float64 [N])."""
    x = np.asarray(x16, dtype=np.float16).astype(np.float64).reshape(-1)
    W = dequantize(codes, scales, levels, level_bits, group)
    return W @ x


def vmm_batch(codes, scales, x16, levels, level_bits, group: int = 128) -> np.ndarray:
    """Tokens are independent: y[t] = W_hat(levels[t]) x[t]  (float64 [B, N])."""
    x16 = np.atleast_2d(np.asarray(x16, dtype=np.float16))
    levels = np.atleast_2d(np.asarray(levels))
    return np.stack([vmm(codes, scales, x16[t], levels[t], level_bits, group)
                     for t in range(x16.shape[0])])


def prefill(codes, scales, x16, group: int = 128, b_max: int = B_MAX) -> np.ndarray:
    """Stage-decoupled prefill (Sec. 3: the prompt is processed with the
    weights at the fixed top precision b_max; Sec. 4 "Prefill vs. Decoding
    Evaluation": unpack at b_max, dense matrix-matrix product).  Every channel
    of every token is read at b_max bits, so W_hat = s (q - 2^(b_max-1))
    (R1, R3) and Y = X W_hat^T for the M tokens in x16 [M, K] (float64 [M, N])."""
    codes = np.asarray(codes)
    N, K = codes.shape
    s_full = np.repeat(np.asarray(scales, dtype=np.float16).astype(np.float64).T,
                       group, axis=1)                          # [N, K]
    W = reconstruct(codes, s_full, b_max, b_max)
    X = np.atleast_2d(np.asarray(x16, dtype=np.float16)).astype(np.float64)
    return X @ W.T


def vmm_lut(codes, luts, x16, levels, level_bits) -> np.ndarray:
    """Non-uniform nested weights read through look-up tables (Sec. 3.3: the
    format only needs the nested property, which k-means-style nested weights
    have; their levels are centred, so there is no phi; App. "Evaluation of
    Nested Weight Formats").  luts[b] is an fp16 [N, 2^b] table per level
    width b; a channel at level l (b = level_bits[l] > 0) reads the b most
    significant bits q_b of the b_max-bit code and weighs x_k by
    luts[b][n][q_b]; level 0 is skipped.  One token: float64 [N]."""
    b_max = int(level_bits[-1])
    codes = np.asarray(codes).astype(np.int64)
    N, K = codes.shape
    x = np.asarray(x16, dtype=np.float16).astype(np.float64).reshape(-1)
    levels = np.asarray(levels).reshape(K)
    W = np.zeros((N, K), dtype=np.float64)
    rows = np.arange(N)[:, None]
    for lvl, b in enumerate(level_bits):
        b = int(b)
        cols = np.nonzero(levels == lvl)[0]
        if cols.size == 0 or b == 0:
            continue
        qb = nested_code(codes[:, cols], b, b_max)                  # [N, |cols|]
        W[:, cols] = np.asarray(luts[b], dtype=np.float16).astype(np.float64)[rows, qb]
    return W @ x


def vmm_lut_batch(codes, luts, x16, levels, level_bits) -> np.ndarray:
    """Tokens are independent (float64 [B, N])."""
    x16 = np.atleast_2d(np.asarray(x16, dtype=np.float16))
    levels = np.atleast_2d(np.asarray(levels))
    return np.stack([vmm_lut(codes, luts, x16[t], levels[t], level_bits) for t in range(x16.shape[0])])


# ---------------------------------------------------------------------------
# 6. Packed nested layout (Sec. 3.3 and App. C.1, as re-laid-out for CDNA4)
# ---------------------------------------------------------------------------
def plane_bits_for(level_bits) -> int:
    """u = 2 when every level is an even number of bits, else 1 (R9)."""
    return 2 if all(int(b) % 2 == 0 for b in level_bits) else 1


def pack_codes(codes: np.ndarray, plane_bits: int, tile_n: int, b_max: int = B_MAX) -> np.ndarray:
    """Pack b_max-bit codes[N, K] into the tile-major, row-prefix, bit-plane layout.

    Definition (written out bit by bit on purpose):
      * N is cut into tiles of ``tile_n`` outputs; tile t covers outputs
        t*tile_n .. t*tile_n + tile_n - 1;
      * the row of (tile t, channel k) is R = tile_n*b_max/8 bytes starting at
        byte (t*K + k) * R;
      * it holds P = b_max/u planes, most significant first; plane j (1-based)
        starts at byte (j-1) * tile_n*u/8 of the row and holds, for local
        output o, the u-bit field (q >> (b_max - j*u)) & (2^u - 1) at bit o*u
        of the plane (byte floor(o*u/8), bit (o*u) mod 8, little-endian bits).
    """
    u = int(plane_bits)
    codes = np.asarray(codes, dtype=np.uint8)
    N, K = codes.shape
    assert N % tile_n == 0 and 8 % u == 0 and b_max % u == 0
    P = b_max // u
    R = tile_n * b_max // 8
    plane_bytes = tile_n * u // 8
    out = np.zeros(N * K * b_max // 8, dtype=np.uint8)
    mask = (1 << u) - 1
    for t in range(N // tile_n):
        for k in range(K):
            row = (t * K + k) * R
            for o in range(tile_n):
                q = int(codes[t * tile_n + o, k])
                for j in range(1, P + 1):
                    field = (q >> (b_max - j * u)) & mask
                    bit = o * u
                    byte = row + (j - 1) * plane_bytes + bit // 8
                    out[byte] |= field << (bit % 8)
    return out


def pack_codes_fast(codes: np.ndarray, plane_bits: int, tile_n: int, b_max: int = B_MAX) -> np.ndarray:
    """Same bytes as ``pack_codes``, vectorised over outputs (for large tests).

    Equality with ``pack_codes`` is itself tested on small inputs.
    """
    u = int(plane_bits)
    codes = np.asarray(codes, dtype=np.uint8)
    N, K = codes.shape
    P = b_max // u
    per_byte = 8 // u
    T = N // tile_n
    c = codes.reshape(T, tile_n, K).transpose(0, 2, 1)            # [T, K, tile_n]
    mask = (1 << u) - 1
    planes = []
    for j in range(1, P + 1):
        f = ((c >> (b_max - j * u)) & mask).astype(np.uint16)      # [T, K, tile_n]
        f = f.reshape(T, K, tile_n // per_byte, per_byte)
        byte = np.zeros(f.shape[:3], dtype=np.uint16)
        for e in range(per_byte):
            byte |= f[..., e] << (e * u)
        planes.append(byte.astype(np.uint8))
    return np.concatenate(planes, axis=2).reshape(-1)


def unpack_prefix(packed: np.ndarray, N: int, K: int, plane_bits: int, tile_n: int,
                  depth_bits: int, b_max: int = B_MAX) -> np.ndarray:
    """Read the first depth_bits/u planes of every row and rebuild q_b [N, K]."""
    u = int(plane_bits)
    assert depth_bits % u == 0
    planes = depth_bits // u
    per_byte = 8 // u
    plane_bytes = tile_n * u // 8
    T = N // tile_n
    rows = np.asarray(packed, dtype=np.uint8).reshape(T, K, tile_n * b_max // 8)
    q = np.zeros((T, K, tile_n), dtype=np.int64)
    mask = (1 << u) - 1
    for j in range(1, planes + 1):
        pb = rows[:, :, (j - 1) * plane_bytes: j * plane_bytes].astype(np.int64)
        f = np.stack([(pb >> (e * u)) & mask for e in range(per_byte)], axis=-1)
        q = (q << u) | f.reshape(T, K, tile_n)
    return q.transpose(0, 2, 1).reshape(N, K)


def calibrate_thresholds(samples_abs, p_bp) -> np.ndarray:
    """Offline threshold calibration (Sec. 3.2; App. A.1; reading R16).

    For every calibration sample the thresholds are the magnitudes that split
    |x| into the fractions P: theta_k is the sample quantile (type 7 of
    Hyndman and Fan) of that sample's magnitudes at q_k = U_k / 10000,
    U_k = sum_{j<k} p_j in basis points.  With the n magnitudes sorted
    ascending (a_0 <= ... <= a_(n-1)), the position h = (n-1) U_k / 10000 is
    taken exactly: lo = floor(h), frac = the fraction of h as a float64
    quotient of integers, and theta = a_lo + frac * (a_(lo+1) - a_lo) in
    float64 (a_(lo+1) = a_lo when lo = n-1).  The per-sample thresholds are
    then averaged in float64, summed in sample order, and rounded to fp32.
    Returns theta_1..theta_n.
    """
    p = [int(v) for v in p_bp]
    n_th = len(p) - 1
    acc = np.zeros(n_th, dtype=np.float64)
    count = 0
    for a in samples_abs:
        srt = np.sort(np.asarray(a, dtype=np.float64).reshape(-1))
        n = srt.size
        ths = np.empty(n_th, dtype=np.float64)
        for k in range(1, n_th + 1):
            U = sum(p[:k])
            num = (n - 1) * U                      # h = num / 10000, exactly
            lo = num // 10000
            frac = np.float64(num % 10000) / np.float64(10000.0)
            lo_v = srt[lo]
            hi_v = srt[min(lo + 1, n - 1)]
            ths[k - 1] = lo_v + frac * (hi_v - lo_v)
        acc = acc + ths
        count += 1
    return (acc / np.float64(count)).astype(np.float32)