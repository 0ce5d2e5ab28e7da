"""Offline tile sweep: time every GEMM tile on each workload shape and write the
per-shape table (tile_table.inc) the library compiles in.

The paper tunes its kernel per (M, N, K) with an autotuner over 36 configurations at
first call (Section 3, "Why autotuning is load-bearing"); here the search runs once,
offline, on the target GPU, and its result is a constant table in the library.

Usage (on an MI355X): python -m paper_2606_14598_amd.tune --out tile_table.inc [--json r.json]
"""
from __future__ import annotations

import argparse
import json
import os
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
// shapes not listed use the fallback rule in gemm_i8.hip.
"""


def time_ms(fn, iters=20, warmup=3):
    """Mean ms per call of fn: `iters` calls captured once in a HIP graph and replayed,
    so microsecond kernels are timed without the host's per-launch overhead."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for _ in range(iters):
                fn()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    st.record()
    for _ in range(3):
        g.replay()
    en.record()
    torch.cuda.synchronize()
    return st.elapsed_time(en) / (3 * iters)


def shapes():
    seen = set()
    for c in sorted(si.WORKLOADS):
        for s in si.WORKLOADS[c]:
            key = (s.M, s.N, s.K)
            if key not in seen:
                seen.add(key)
                yield s


def _dev_bf16(bits, dev):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)


def sweep(iters: int):
    """Time every tile on every workload shape, on the workload's own synthetic inputs
    quantized by the library: the matrix cores' sustained rate depends on the operand
    bits (switching power), so uniform random or constant codes would mislead."""
    dev = torch.device("cuda:0")
    results = []
    for s in shapes():
        x, w, bb = si.make_inputs(s)
        xq, sx = w8a8.quantize_act(_dev_bf16(x, dev))
        wq, sw = w8a8.quantize_weight(_dev_bf16(w, dev))
        b = _dev_bf16(bb, dev)
        row = {"M": s.M, "N": s.N, "K": s.K, "ms": {}}
        y = torch.empty((s.M, s.N), dtype=torch.bfloat16, device=dev)
        for t in range(w8a8.tile_count()):
            ms = time_ms(lambda: w8a8.gemm(xq, sx, wq, sw, b, tile=t, out=y), iters)
            row["ms"][w8a8.tile_name(t)] = ms
        best = min(row["ms"], key=row["ms"].get)
        row["best"] = best
        row["best_tops"] = 2 * s.M * s.N * s.K / (row["ms"][best] * 1e-3) / 1e12
        print(json.dumps(row), flush=True)
        results.append(row)
    return results


def write_table(results, path):
    names = [w8a8.tile_name(t) for t in range(w8a8.tile_count())]
    lines = [HEADER, "static const TableEntry kTileTable[] = {"]
    for r in results:
        lines.append(f"    {{{r['M']}, {r['M']}, {r['N']}, {r['K']}, {names.index(r['best'])}}},"
                     f"  // {r['best']} {r['best_tops']:.0f} TOPS")
    lines.append("    {0, 0, 0, 0, -1},  // sentinel")
    lines.append("};")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", required=True)
    ap.add_argument("--json")
    ap.add_argument("--iters", type=int, default=20)
    a = ap.parse_args()
    res = sweep(a.iters)
    write_table(res, a.out)
    if a.json:
        with open(a.json, "w") as f:
            json.dump(res, f, indent=1)


if __name__ == "__main__":
    main()
