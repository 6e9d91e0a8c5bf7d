"""Seeded synthetic inputs for the nested-precision decode VMM.

This module only draws random numbers and names workload shapes.  It holds
none of the method's arithmetic (no quantisation, no assignment, no
reconstruction) so that both the CPU oracle's tests and the GPU path can take
their inputs from it without sharing any computation.

Workload recipe (stands in for the paper's Llama3-8B / Qwen3-8B weights and
activations, which are not available; Sec. 4 "Experimental Setup"):

* weights  W[n, k]: float64 N(0, 0.02) rounded to fp16 (RNE), torch
  ``Linear.weight`` layout [N, K];
* attention / o-proj / MLP-input activations: Student-t with 3 degrees of
  freedom per element; a fixed set of round(0.01 K) outlier channels per
  layer (same for every token) is multiplied by 20 before the fp16 cast.
  This gives the heavy-tailed, outlier-channel structure that the dynamic
  assignment of Sec. 3.1 relies on;
* down-projection input: SiLU(g) * u with g, u iid N(0, 1) in fp32, cast to
  fp16 (the product of the gate and up branches of a SwiGLU MLP).

Every stream is a numpy ``Generator(PCG64)`` built from
``SeedSequence(seed, spawn_key=(config, layer, role))`` so that each
(config, layer, role) triple draws the same numbers on any machine.
"""
from __future__ import annotations

import numpy as np

ROLE_W = 0
ROLE_X = 1
ROLE_OUTLIER = 2
ROLE_CALIB = 3
ROLE_CODES = 4


def rng(config: int, layer: int, role: int, seed: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence(seed, spawn_key=(int(config), int(layer), int(role)))
    return np.random.Generator(np.random.PCG64(ss))


def weights(N: int, K: int, config: int = 1, layer: int = 0, seed: int = 0) -> np.ndarray:
    """fp16 [N, K] weights drawn from N(0, 0.02)."""
    g = rng(config, layer, ROLE_W, seed)
    return g.normal(0.0, 0.02, size=(N, K)).astype(np.float16)


def random_codes(N: int, K: int, config: int = 1, layer: int = 0, seed: int = 0) -> np.ndarray:
    """uint8 [N, K] uniformly random 8-bit codes (for the pre-quantised entry)."""
    g = rng(config, layer, ROLE_CODES, seed)
    return g.integers(0, 256, size=(N, K), dtype=np.uint8)


def random_scales(N: int, K: int, group: int = 128, config: int = 1, layer: int = 0,
                  seed: int = 0) -> np.ndarray:
    """fp16 [N, K/group] positive scales (the pre-quantised entry's scale input)."""
    g = rng(config, layer, ROLE_CODES, seed + 1)
    return g.uniform(1e-4, 4e-4, size=(N, K // group)).astype(np.float16)


def outlier_channels(K: int, config: int = 1, layer: int = 0, seed: int = 0) -> np.ndarray:
    g = rng(config, layer, ROLE_OUTLIER, seed)
    n_out = int(round(0.01 * K))
    return np.sort(g.choice(K, size=n_out, replace=False))


def activations_t3(K: int, tokens: int, config: int = 1, layer: int = 0, seed: int = 0,
                   role: int = ROLE_X) -> np.ndarray:
    """fp16 [tokens, K]: Student-t(3) with 1% outlier channels scaled x20."""
    g = rng(config, layer, role, seed)
    x = g.standard_t(3.0, size=(tokens, K))
    idx = outlier_channels(K, config, layer, seed)
    x[:, idx] *= 20.0
    return x.astype(np.float16)


def activations_swiglu(K: int, tokens: int, config: int = 1, layer: int = 0, seed: int = 0,
                       role: int = ROLE_X) -> np.ndarray:
    """fp16 [tokens, K]: SiLU(g) * u with g, u iid N(0, 1), computed in fp32."""
    gen = rng(config, layer, role, seed)
    gg = gen.standard_normal(size=(tokens, K)).astype(np.float32)
    uu = gen.standard_normal(size=(tokens, K)).astype(np.float32)
    silu = gg / (np.float32(1.0) + np.exp(-gg))
    return (silu * uu).astype(np.float16)


def nested_luts(N: int, level_bits, config: int = 1, layer: int = 0, seed: int = 0):
    """Synthetic per-output nested look-up tables, shaped like any-precision
    (nested k-means) weights: for every output n, 2^b_max sorted centroids of
    a N(0, 0.02) row at the top width b_max = level_bits[-1]; the table of a
    narrower width b holds, for each b-bit prefix c, the mean of the
    2^(b_max-b) centroids under it.  Returns {b: fp16 [N, 2^b]} for every
    b > 0 in level_bits."""
    b_max = int(level_bits[-1])
    g = rng(config, layer, ROLE_CODES, seed + 2)
    top = np.sort(g.normal(0.0, 0.02, size=(N, 2 ** b_max)), axis=1)
    out = {}
    for b in level_bits:
        b = int(b)
        if b == 0:
            continue
        out[b] = top.reshape(N, 2 ** b, 2 ** (b_max - b)).mean(axis=2).astype(np.float16)
    return out


# --------------------------------------------------------------------------
# Level sets and precision distributions (basis points, sum 10000).
# The {0,2,4,6,8} rows marked "sweep" are rows of the paper's precision
# distribution sweep table (App. A.2, b_max = 8 column); the others are
# budgets chosen here to hit the named average bits (sum p_i b_i).
# --------------------------------------------------------------------------
LEVELS_A = (0, 2, 4, 8)
LEVELS_B = (0, 2, 4, 6, 8)
LEVELS_C = (0, 2, 3, 4, 8)
LEVELS_D = (0, 2, 4, 6)       # b_max = 6
LEVELS_E = (0, 2, 4)          # b_max = 4

BUDGETS = {
    LEVELS_A: {
        2: (3000, 5000, 1500, 500),
        3: (2000, 4000, 2500, 1500),
        4: (2000, 2000, 3000, 3000),
        8: (0, 0, 0, 10000),
    },
    LEVELS_B: {
        2: (3000, 4500, 2000, 500, 0),
        3: (2500, 2200, 3100, 2200, 0),      # sweep row 9
        4: (2000, 800, 2400, 4800, 0),       # sweep row 29
        6: (2000, 0, 0, 2000, 6000),
        8: (0, 0, 0, 0, 10000),              # sweep row 60
    },
    LEVELS_C: {
        2: (3000, 4000, 2000, 500, 500),
        3: (2000, 3000, 2000, 1500, 1500),
        4: (2000, 1000, 2000, 2000, 3000),
    },
    # rows of the same sweep table, b_max = 6 and b_max = 4 columns
    LEVELS_D: {
        3: (2500, 2200, 3100, 2200),          # sweep row 9, 3.00 bits
        4: (2000, 800, 2400, 4800),           # sweep row 29, 4.00 bits
        6: (0, 0, 0, 10000),
    },
    LEVELS_E: {
        2: (3500, 2500, 4000),                # sweep row 52, 2.10 bits
        3: (2500, 100, 7400),                 # sweep row 30, 2.98 bits
        4: (0, 0, 10000),                     # sweep row 1
    },
}


# Layer shapes (K -> N) of the workloads.
LLAMA3_8B = {
    "q": (4096, 4096), "k": (4096, 1024), "v": (4096, 1024), "o": (4096, 4096),
    "gate": (4096, 14336), "up": (4096, 14336), "down": (14336, 4096),
}
QWEN3_8B = {
    "qkv": (4096, 6144), "o": (4096, 4096), "gate": (4096, 12288), "up": (4096, 12288),
    "down": (12288, 4096),
}
