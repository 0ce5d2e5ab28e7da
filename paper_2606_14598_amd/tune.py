"""Offline tile sweep: time every GEMM tile on each workload shape and write the
per-shape table (tile_table.inc) the library compiles in.

The paper tunes its kernel per (M, N, K) with an autotuner over 36 configurations at
first call (Section 3, "Why autotuning is load-bearing"); here the search runs once,
offline, on the target GPU, and its result is a constant table in the library.

Two sets of shapes: the workload shapes (one entry each, for their exact M) and the
paper's five model shapes over its token counts (Section 3, "Target architecture";
Section 5), which get token-count buckets: each swept M owns the range up to the
midpoints with its neighbours.

Usage (on an MI355X): python -m paper_2606_14598_amd.tune --out tile_table.inc
       [--json r.json] [--set all|workloads|paper] [--iters N]
"""
from __future__ import annotations

import argparse
import json
import os
import re
import sys

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import paper_2606_14598_amd as w8a8  # noqa: E402
import synth_inputs as si  # noqa: E402

HEADER = """// Offline-chosen GEMM tile per shape: {M lower bound, M upper bound, N, K, tile id}.
// Written by paper_2606_14598_amd/tune.py from a timed sweep of every tile on MI355X;
// shapes not listed use the fallback rule in gemm_i8.hip, whose cost model takes each
// tile's per-round cost from kTileCost below.
"""

CUS = 256


def time_ms(fn, iters=20, warmup=3, warm_ms=0.0, min_timed_ms=2.0):
    """Mean ms per call of fn: `iters` calls captured once in a HIP graph and replayed,
    so microsecond kernels are timed without the host's per-launch overhead. The graph
    is replayed for `warm_ms` before timing, and timed over at least `min_timed_ms`."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for _ in range(iters):
                fn()
    st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    st.record()
    g.replay()
    en.record()
    torch.cuda.synchronize()
    once = max(st.elapsed_time(en), 1e-3)
    for _ in range(int(warm_ms / once)):
        g.replay()
    reps = max(3, int(min_timed_ms / once) + 1)
    torch.cuda.synchronize()
    st.record()
    for _ in range(reps):
        g.replay()
    en.record()
    torch.cuda.synchronize()
    return st.elapsed_time(en) / (reps * iters)


def shapes(which: str = "all"):
    """(shape, M lower bound, M upper bound) of every entry to tune."""
    seen = set()
    if which in ("all", "workloads"):
        for c in sorted(si.WORKLOADS):
            for s in si.WORKLOADS[c]:
                key = (s.M, s.N, s.K)
                if key not in seen:
                    seen.add(key)
                    yield s, s.M, s.M
    if which in ("all", "paper"):
        ms = sorted(si.PAPER_M)
        for name, _, _ in si.PAPER_SHAPES:
            for i, M in enumerate(ms):
                lo = 257 if i == 0 else (ms[i - 1] + M) // 2 + 1
                hi = (1 << 62) if i == len(ms) - 1 else (M + ms[i + 1]) // 2
                yield si.paper_shape(name, M), lo, hi


def _dev_bf16(bits, dev):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)


def sweep(iters: int, which: str = "all"):
    """Time every tile on every shape, on the shape's own synthetic inputs quantized by
    the library: the matrix cores' sustained rate depends on the operand bits
    (switching power), so uniform random or constant codes would mislead. The
    weight-streaming tiles (made for M <= 128) are skipped above 128 tokens, and the
    split-K tiles where their unsplit tile already gives two workgroups per CU. The chip's
    power management needs ~15-20 ms of sustained load to settle after an idle gap (the
    input generation between shapes is one), so each shape first runs 30 ms of work,
    and every tile is timed twice, in two passes, keeping the faster."""
    dev = torch.device("cuda:0")
    results = []
    for s, lo, hi in shapes(which):
        x, w, bb = si.make_inputs(s)
        xd = _dev_bf16(x, dev)
        del x
        xq, sx = w8a8.quantize_act(xd)
        del xd
        wq, sw = w8a8.quantize_weight(_dev_bf16(w, dev))
        b = _dev_bf16(bb, dev)
        row = {"name": s.name, "M": s.M, "N": s.N, "K": s.K, "m_lo": lo, "m_hi": hi,
               "default": w8a8.tile_name(w8a8.default_tile(s.M, s.N, s.K)), "ms": {}}
        y = torch.empty((s.M, s.N), dtype=torch.bfloat16, device=dev)
        nws = max(w8a8.gemm_workspace_bytes(s.M, s.N, s.K, t) for t in range(w8a8.tile_count()))
        ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
        it = iters if s.ops < 5e14 else max(3, iters // 4)
        def wanted(t):
            name = w8a8.tile_name(t)
            if s.M > 128 and name.startswith(("skinny", "wsx")):
                return False
            d = _tile_dims(name)
            # split-K only pays where the unsplit tiles leave CUs idle
            if "_k" in name and -(-s.M // d[0]) * -(-s.N // d[1]) >= 2 * CUS:
                return False
            return True
        cand = [t for t in range(w8a8.tile_count()) if wanted(t)]
        first = w8a8.select_tile(s.M, s.N, s.K)
        time_ms(lambda: w8a8.gemm(xq, sx, wq, sw, b, tile=first, out=y, workspace=ws), it,
                warm_ms=30.0)
        for _ in range(2):
            for t in cand:
                name = w8a8.tile_name(t)
                ms = time_ms(lambda: w8a8.gemm(xq, sx, wq, sw, b, tile=t, out=y, workspace=ws),
                             it)
                row["ms"][name] = min(ms, row["ms"].get(name, ms))
        best = min(row["ms"], key=row["ms"].get)
        row["best"] = best
        row["best_tops"] = 2 * s.M * s.N * s.K / (row["ms"][best] * 1e-3) / 1e12
        print(json.dumps(row), flush=True)
        results.append(row)
        del xq, sx, wq, sw, b, y, ws
        torch.cuda.empty_cache()
    return results


def _tile_dims(name):
    m = re.match(r"m(\d+)n(\d+)k(\d+)", name)
    return tuple(int(g) for g in m.groups()) if m else None


def tile_costs(results, names):
    """Per-round cost model of each LDS-staged tile, fitted to the sweep: a launch of T
    workgroups takes ceil(T / CUS) rounds, each costing c + d * (K * TM * TN / 1e9) ms
    (c: the fixed part of a round -- launch share, prologue, epilogue; d: the
    per-multiply-accumulate part). Least squares on relative error over the swept shapes
    with more than 128 tokens; c is held at 0 if it fits negative. (0, 0) for the
    weight-streaming and split-K tiles (not modeled)."""
    out = []
    for n in names:
        d = _tile_dims(n)
        rows, ys = [], []
        if d is not None and "_k" not in n:
            for r in results:
                if r["M"] <= 128 or n not in r["ms"]:
                    continue
                tiles = -(-r["M"] // d[0]) * -(-r["N"] // d[1])
                rounds = -(-tiles // CUS)
                rows.append([rounds, rounds * r["K"] * d[0] * d[1] / 1e9])
                ys.append(r["ms"][n])
        if len(rows) < 2:
            out.append((0.0, 0.0))
            continue
        A = np.array(rows)
        y = np.array(ys)
        w = 1.0 / y
        c, dd = np.linalg.lstsq(A * w[:, None], y * w, rcond=None)[0]
        if c < 0:
            c = 0.0
            dd = float(np.sum(A[:, 1] * w * w * y) / np.sum((A[:, 1] * w) ** 2))
        out.append((float(c), float(dd)) if dd > 0 else (0.0, 0.0))
    return out


def write_table(results, path):
    names = [w8a8.tile_name(t) for t in range(w8a8.tile_count())]
    costs = tile_costs(results, names)
    lines = [HEADER, "// Fallback cost model per tile: {c, d}, one round = c + d * K * TM * TN / 1e9 ms.",
             "static const TileCost kTileCost[] = {"]
    for n, (c, dd) in zip(names, costs):
        lines.append(f"    {{{c:.6e}, {dd:.6e}}},  // {n}")
    lines.append("};")
    lines.append("")
    lines.append("static const TableEntry kTileTable[] = {")
    for r in results:
        lines.append(f"    {{{r['m_lo']}, {r['m_hi']}, {r['N']}, {r['K']}, "
                     f"{names.index(r['best'])}}},  // M={r['M']} {r['best']} "
                     f"{r['best_tops']:.0f} TOPS")
    lines.append("    {0, 0, 0, 0, -1},  // sentinel")
    lines.append("};")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", required=True)
    ap.add_argument("--json")
    ap.add_argument("--iters", type=int, default=20)
    ap.add_argument("--set", default="all", choices=["all", "workloads", "paper"])
    ap.add_argument("--from-json", help="rewrite the table from a saved sweep (no timing)")
    a = ap.parse_args()
    if a.from_json:
        with open(a.from_json) as f:
            res = json.load(f)
        for r in res:
            r.setdefault("m_lo", r["M"])
            r.setdefault("m_hi", r["M"])
    else:
        res = sweep(a.iters, a.set)
    write_table(res, a.out)
    if a.json and not a.from_json:
        with open(a.json, "w") as f:
            json.dump(res, f, indent=1)


if __name__ == "__main__":
    main()
