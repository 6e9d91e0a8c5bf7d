"""Benchmark of the nested-precision decode VMM on one MI355X.

Default workload: the Llama3-8B attention projections at batch 1 (q, o
4096x4096; k, v 4096->1024), 256 synthetic tokens, top-k assignment at an
average budget of 4 bits over the levels {0,2,4,6,8}.  One step is the whole
hot path for every token: grade the attention input (one assignment shared by
q, k and v), run the q, k, v VMMs, grade the o-projection input, run the o VMM.
The step is captured once as a HIP graph and replayed.  The packed weights
rotate over enough distinct copies (> 512 MiB) that the 256 MiB last-level
cache cannot serve them between uses.

Output: one JSON line.  `value` is whole-step throughput in GB/s of required
bytes (sum over every VMM of the bytes its level map requires: code prefixes,
scales of groups with an active channel, x, y, level map); `roofline` is for
the VMM kernel alone, timed with HIP events on its own stream.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from synth import inputs  # noqa: E402

HBM_PEAK_GBS = 8000.0
MALL_ROTATE_BYTES = 512 << 20
PROFILES = os.path.join(ROOT, "profiles")
# sources whose change invalidates a stored traffic measurement of the VMM kernel
VMM_SOURCES = ("paper_2606_23419_amd/csrc/vmm_dot2.hip", "paper_2606_23419_amd/csrc/vmm.hip",
               "paper_2606_23419_amd/csrc/grinqh_internal.h")

WORKLOADS = {
    # name: (config id, layers [(name, K, N, input id)], level set, budget)
    "llama3-8b-attn": (2, [("q", 4096, 4096, 0), ("k", 4096, 1024, 0), ("v", 4096, 1024, 0),
                           ("o", 4096, 4096, 1)], inputs.LEVELS_B, 4),
    "llama3-8b-attn-b3": (2, [("q", 4096, 4096, 0), ("k", 4096, 1024, 0), ("v", 4096, 1024, 0),
                              ("o", 4096, 4096, 1)], inputs.LEVELS_B, 3),
    "llama3-8b-mlp": (3, [("gate", 4096, 14336, 0), ("up", 4096, 14336, 0),
                          ("down", 14336, 4096, 1)], inputs.LEVELS_B, 4),
    "qwen3-8b-layer": (4, [("qkv", 4096, 6144, 0), ("o", 4096, 4096, 1), ("gate", 4096, 12288, 2),
                           ("up", 4096, 12288, 2), ("down", 12288, 4096, 3)], inputs.LEVELS_C, 3),
    "single-1024": (1, [("w", 1024, 1024, 0)], inputs.LEVELS_A, 4),
}


def vmm_source_sha() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in VMM_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stored_traffic(workload: str, budget: int):
    """HBM bytes per VMM launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary of this workload, or None when there is none or the
    kernel sources changed since it was taken."""
    path = os.path.join(PROFILES, f"k_vmm_dot2_traffic_{workload}_b{budget}.md")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith(("#", "|", " ")):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("source_sha256_16") != vmm_source_sha():
        return None
    try:
        return float(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration(mib: int, reps: int):
    """A plain device-to-device copy of known size, for scaling the HBM byte
    counters (run under rocprofv3 --pmc)."""
    import torch
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "reps": reps}), flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama3-8b-attn", choices=sorted(WORKLOADS))
    ap.add_argument("--budget", type=int, default=None, help="override the average-bit budget")
    ap.add_argument("--tokens", type=int, default=256)
    ap.add_argument("--tile-n", type=int, default=0)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--vmm-only-reps", type=int, default=5)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain copy of MIB MiB (counter calibration) and exit")
    ap.add_argument("--vmm-source-sha", action="store_true",
                    help="print the hash of the VMM kernel sources and exit")
    return ap.parse_args()


def bytes_required(level_map: np.ndarray, level_bits, K: int, N: int) -> np.ndarray:
    """Per-token algorithmic bytes of one VMM (B = 1): the code prefixes the
    levels ask for, the scales of groups with any active channel, x (fp16),
    y (fp32) and the level map (uint8)."""
    bits = np.asarray(level_bits, dtype=np.int64)[level_map.astype(np.int64)]   # [T, K]
    code = bits.sum(axis=1) * N // 8
    active_groups = (level_map.reshape(level_map.shape[0], K // 128, 128) > 0).any(axis=2).sum(axis=1)
    return code + active_groups * N * 2 + 2 * K + 4 * N + K


def cpu_baseline(wl, budget, tokens_sample: int):
    """Time the oracle (assignment + dequantise + float64 matvec) on host cores."""
    from threadpoolctl import threadpool_limits
    from oracle import grinqh_oracle as orc

    cfg, layers, levels, _ = wl
    p = inputs.BUDGETS[levels][budget]
    xs = {}
    codes = {}
    for li, (name, K, N, xin) in enumerate(layers):
        W = inputs.weights(N, K, cfg, li)
        codes[name] = orc.rtn_quantize(W)
        if xin not in xs:
            gen = inputs.activations_swiglu if name == "down" else inputs.activations_t3
            xs[xin] = gen(K, tokens_sample, cfg, 100 + xin)
    total_bytes = 0
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        for t in range(tokens_sample):
            lms = {}
            for li, (name, K, N, xin) in enumerate(layers):
                if xin not in lms:
                    lms[xin] = orc.assign_topk(xs[xin][t], orc.topk_counts(K, p))
                q, s = codes[name]
                orc.vmm(q, s, xs[xin][t], lms[xin], levels)
                total_bytes += int(bytes_required(lms[xin][None, :], levels, K, N)[0])
        dt = time.perf_counter() - t0
    return {"value": round(total_bytes / dt / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{tokens_sample} tokens x {len(layers)} VMMs (+assignment) of the same workload, "
                      f"numpy float64, 1 thread; {dt:.1f} s"}


def main():
    args = parse()
    if args.vmm_source_sha:
        print(vmm_source_sha())
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the nested-precision "
              "VMM path has no multi-GPU mode in this build.", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration(args.copy_calibration, reps=10)
        return

    import torch
    from paper_2606_23419_amd import grinqh as g

    dev = torch.device("cuda:0")
    wl = WORKLOADS[args.workload]
    cfg, layers, levels, budget = wl
    if args.budget is not None:
        budget = args.budget
    p_bp = inputs.BUDGETS[levels][budget]
    T = args.tokens

    # ---- layers: pack once, then replicate to defeat the last-level cache
    descs, packed = {}, {}
    layer_bytes = 0
    for li, (name, K, N, _) in enumerate(layers):
        d = g.grinqh_resolve_desc(g.make_desc(K, N, levels, tile_n=args.tile_n))
        W = torch.from_numpy(inputs.weights(N, K, cfg, li)).to(dev)
        pc, ps = g.grinqh_pack(d, W=W)
        del W
        descs[name], packed[name] = d, (pc, ps)
        layer_bytes += pc.numel() + ps.numel() * 2
    R = max(1, -(-MALL_ROTATE_BYTES // layer_bytes))
    copies = [{n: (packed[n][0].clone(), packed[n][1].clone()) for n in packed} for _ in range(R - 1)]
    copies.insert(0, packed)

    # ---- inputs and outputs
    n_inputs = max(xin for *_, xin in layers) + 1
    xs = []
    for xin in range(n_inputs):
        name, K = next((n, k) for n, k, _, i in layers if i == xin)
        gen = inputs.activations_swiglu if name == "down" else inputs.activations_t3
        xs.append(torch.from_numpy(gen(K, T, cfg, 100 + xin)).to(dev))
    lm = [torch.empty(x.shape, dtype=torch.uint8, device=dev) for x in xs]
    counts = [g.grinqh_topk_counts(int(x.shape[1]), p_bp) for x in xs]
    ybufs = {name: torch.zeros((T, N), dtype=torch.float32, device=dev) for name, _, N, _ in layers}

    def _desc_for(xin):
        return next(descs[n] for n, _, _, i in layers if i == xin)

    def step(vmm_only=False):
        if not vmm_only:
            for b in ybufs.values():
                b.zero_()
        for t in range(T):
            c = copies[t % R]
            for xin in range(n_inputs):
                if not vmm_only:
                    g.grinqh_assign(_desc_for(xin), xs[xin][t:t + 1], g.GRINQH_ASSIGN_TOPK,
                                    counts=counts[xin], out=lm[xin][t:t + 1])
                for name, K, N, xi in layers:
                    if xi == xin:
                        g.grinqh_vmm(descs[name], c[name][0], c[name][1], xs[xin][t:t + 1],
                                     lm[xin][t:t + 1], y=ybufs[name][t:t + 1], accumulate=True)

    # ---- eager run (reference for the graph replays), then capture
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.synchronize()
    eager = {n: b.clone() for n, b in ybufs.items()}
    lm_host = [m.cpu().numpy() for m in lm]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        step()
    for _ in range(2):
        graph.replay()
        torch.cuda.synchronize()
        for n, b in ybufs.items():
            # partial sums meet in atomics, so replays agree to rounding, not bits
            err = float((b - eager[n]).abs().max() / eager[n].abs().max())
            if not err <= 1e-5:
                raise RuntimeError(f"graph replay of {n} differs from the eager step ({err:.2e})")
    for m, h in zip(lm, lm_host):
        if not np.array_equal(m.cpu().numpy(), h):
            raise RuntimeError("graph replay changed a level map")

    # ---- required bytes per step (from the level maps actually used)
    req = {}
    for name, K, N, xin in layers:
        req[name] = bytes_required(lm_host[xin], levels, K, N)           # [T]
    step_bytes = int(sum(int(v.sum()) for v in req.values()))
    n_vmm = T * len(layers)
    avg_bits = {xin: float(np.asarray(levels)[lm_host[xin]].mean()) for xin in range(n_inputs)}

    # ---- timed region: whole step
    with torch.cuda.stream(s):
        for _ in range(args.warmup):
            graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        e0.record(s)
        for _ in range(args.steps):
            graph.replay()
        e1.record(s)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps

    # ---- VMM kernel alone: a graph of the step's VMM launches on stream s
    vgraph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(vgraph, stream=s):
        step(vmm_only=True)
    with torch.cuda.stream(s):
        vgraph.replay()
    torch.cuda.synchronize()
    v0, v1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(s):
        v0.record(s)
        for _ in range(args.vmm_only_reps):
            vgraph.replay()
        v1.record(s)
    torch.cuda.synchronize()
    us_per_vmm = v0.elapsed_time(v1) * 1e3 / (args.vmm_only_reps * n_vmm)
    bytes_per_vmm = step_bytes / n_vmm
    achieved = bytes_per_vmm / (us_per_vmm * 1e-6) / 1e9

    # per-layer VMM times (graph of one layer's launches)
    per_layer = {}
    for name, K, N, xin in layers:
        lg = torch.cuda.CUDAGraph()
        with torch.cuda.graph(lg, stream=s):
            for t in range(T):
                c = copies[t % R]
                g.grinqh_vmm(descs[name], c[name][0], c[name][1], xs[xin][t:t + 1],
                             lm[xin][t:t + 1], y=ybufs[name][t:t + 1], accumulate=True)
        with torch.cuda.stream(s):
            lg.replay()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s)
            for _ in range(args.vmm_only_reps):
                lg.replay()
            b.record(s)
        torch.cuda.synchronize()
        us = a.elapsed_time(b) * 1e3 / (args.vmm_only_reps * T)
        mean_req = float(req[name].mean())
        per_layer[name] = {"K": K, "N": N, "us_per_vmm": round(us, 3),
                           "required_bytes": int(mean_req),
                           "GBps": round(mean_req / (us * 1e-6) / 1e9, 1),
                           "tile_n": int(descs[name].tile_n)}

    value = step_bytes / (ms_step * 1e-3) / 1e9
    out = {
        "metric": "µs per decode VMM and effective HBM GB/s (% of peak) vs avg bits, batch 1",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8 codes, fp16 x, f32 accumulate",
        "data": "synthetic (seeded N(0,0.02) weights RTN-quantised; Student-t(3) activations "
                "with 1% x20 outlier channels)",
        "config": {"workload": args.workload, "layers": {n: [K, N] for n, K, N, _ in layers},
                   "tokens": T, "batch": 1, "levels": list(levels), "budget_bits": budget,
                   "assignment": "top-k", "P_bp": list(p_bp), "weight_copies": R,
                   "avg_bits": {f"input{k}": round(v, 4) for k, v in avg_bits.items()}},
        "us_per_vmm": round(us_per_vmm, 3),
        "per_layer": per_layer,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": stored_traffic(args.workload, budget)},
        "algorithmic_bytes_per_vmm": round(bytes_per_vmm, 1),
    }
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(wl, budget, tokens_sample=8)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
