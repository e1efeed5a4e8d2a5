#!/usr/bin/env python3
"""Benchmark of the fused Tetra decode-GEMV on one MI355X.

A step is one token-equivalent pass over the weight matrices of a
Qwen3-shaped model at batch 1: every projection (q, k, v, o, gate, up, down)
of every layer runs once through tetra_gemv on one stream (captured in a HIP
graph so host launch cost is not timed).  The default workload is the
Qwen3-14B shape set x 40 layers (280 matrices, 3.34 GB of codes), larger
than the 256 MB last-level cache, so every step streams from HBM.

Inputs are synthetic and seeded: uniformly random code bytes (every 48-bit
word is legal), fp16 row scales U(0.5, 2) * 1e-2, fp16 tails N(0, 1) * sigma,
fp16 activations N(0, 1).  All buffers are resident in HBM before timing.

Prints one JSON line (rank 0, N = 1):
  value    = algorithmic bytes per step / wall time per step (GB/s)
  roofline = algorithmic bytes per gemv launch / average launch duration
             over the timed region (HIP events on the launch stream), against
             the 8 TB/s HBM peak; traffic = HBM bytes per launch from the
             committed rocprofv3 counter profile when it matches this kernel
             source and workload, else null
  cpu_baseline = the CPU oracle on a bounded sample of the same workload
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "Tetra GEMV achieved HBM GB/s (% of peak) and bits read/weight, batch 1"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--model", default="14B", choices=["4B", "8B", "14B"])
    ap.add_argument("--layers", type=int, default=0, help="0 = all layers of the model")
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--mode", default="deps", choices=["matrix", "deps", "layer"],
                    help="matrix: one launch per matrix; deps: per layer [q,k,v] [o] "
                         "[gate,up] [down] (the launches a decode step can fuse); "
                         "layer: one grouped launch per layer")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="instead of the benchmark: copy a buffer of this many MiB five "
                         "times with torch (a plain copy kernel of known size, the "
                         "calibration for HBM byte counters)")
    return ap.parse_args()


class Matrix:
    """One packed Tetra projection resident on the GPU."""

    def __init__(self, torch, tt, name, M, K, gen, seed):
        self.name, self.M, self.K = name, M, K
        self.nblk, self.T = K // 24, K % 24
        nbytes = tt.codes_bytes(M, K)
        toff = tt.tail_offset(M, K)
        self.blob = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        # any byte string is a legal code region (every 48-bit word is legal)
        self.blob[:toff].random_(0, 256, generator=gen)
        self.blob[toff:].zero_()
        g = torch.Generator(device="cuda").manual_seed(seed)
        self.sigma = (torch.rand(M, generator=g, device="cuda") * 1.5 + 0.5).mul_(1e-2).half()
        if self.T:
            tail = (torch.randn(M, self.T, generator=g, device="cuda") *
                    self.sigma.float()[:, None]).half()
            self.blob[toff:toff + 2 * M * self.T].copy_(tail.view(torch.uint8).reshape(-1))
        # bytes the kernel must read: code chunks, tail, row scales
        self.code_bytes = toff
        self.read_bytes = (M // 64) * self.nblk * 384 + (M % 64 > 0) * self.nblk * 384 \
            + 2 * M * self.T + 2 * M
        self.weights = M * K


def build_workload(torch, tt, model, layers, batch):
    from paper_2609_35465_amd import workloads
    shapes = workloads.layer_shapes(model)
    L = layers or workloads.QWEN3[model]["layers"]
    gen = torch.Generator(device="cuda").manual_seed(workloads.SEED_BASE + 3)
    mats, xs, ys = [], {}, []
    for layer in range(L):
        for i, (name, M, K) in enumerate(shapes):
            mats.append(Matrix(torch, tt, name, M, K, gen, workloads.seed_for(3, 16 * layer + i)))
            if (layer, K) not in xs:
                xs[(layer, K)] = torch.randn(batch, K, generator=gen, device="cuda").half()
            ys.append(torch.empty(batch, M, dtype=torch.float32, device="cuda"))
    plan = [(m, xs[(li // len(shapes), m.K)], ys[li]) for li, m in enumerate(mats)]
    return plan, L


GROUPS = {
    "matrix": [["q"], ["k"], ["v"], ["o"], ["gate"], ["up"], ["down"]],
    "deps": [["q", "k", "v"], ["o"], ["gate", "up"], ["down"]],
    "layer": [["q", "k", "v", "o", "gate", "up", "down"]],
}


def build_launches(tt, plan, mode, nproj=7):
    """One ctypes problem array per launch, in step order."""
    launches = []
    for l0 in range(0, len(plan), nproj):
        layer = plan[l0:l0 + nproj]
        by_name = {m.name: (m, x, y) for m, x, y in layer}
        for names in GROUPS[mode]:
            items = [(by_name[n][0].blob, by_name[n][0].sigma, by_name[n][1], by_name[n][2],
                      by_name[n][0].M, by_name[n][0].K) for n in names]
            launches.append((tt.make_problems(items), [by_name[n][0] for n in names]))
    return launches


def run_step(tt, launches, batch, stream):
    for probs, _ in launches:
        tt.gemv_grouped(probs, batch, stream)


def parity_spot_check(torch, tt, plan, batch):
    """Sampled rows of the first matrices of each shape against the oracle."""
    from oracle import gemv as ogemv
    worst = 0.0
    seen = set()
    for m, x, y in plan:
        if m.name in seen:
            continue
        seen.add(m.name)
        rows = np.unique(np.r_[0:8, m.M - 8:m.M, np.linspace(0, m.M - 1, 24).astype(int)])
        blob = m.blob.cpu().numpy()
        words, tail = tt.unpack_rows(blob, m.M, m.K)
        sig = m.sigma.cpu().numpy()
        xh = x.cpu().numpy()
        ref, norm = ogemv.gemv_f64(words, sig, tail, xh, rows=rows)
        got = y.cpu().numpy()[:, rows].astype(np.float64)
        worst = max(worst, float((np.abs(got - ref) / norm).max()))
    return worst


def cpu_baseline(torch, tt, plan, seconds):
    """The CPU oracle (float64 numpy, one thread) over the step's matrices in
    step order, 2048 rows at a time, until it has run for `seconds`; rate in
    GB/s of Tetra bytes (6 B per block, 2 B per tail weight and row scale).
    Copying a matrix to the host and unpacking it are not timed."""
    from oracle import gemv as ogemv
    t_used, bytes_done, rows_done, mats = 0.0, 0, 0, []
    for m, x, _ in plan:
        if t_used >= seconds:
            break
        blob = m.blob.cpu().numpy()
        words, tail = tt.unpack_rows(blob, m.M, m.K)
        sig = m.sigma.cpu().numpy()
        xh = x.cpu().numpy()
        done = 0
        for r0 in range(0, m.M, 2048):
            if t_used >= seconds:
                break
            rows = np.arange(r0, min(r0 + 2048, m.M))
            t0 = time.perf_counter()
            ogemv.gemv_f64(words, sig, tail, xh, rows=rows)
            t_used += time.perf_counter() - t0
            done += len(rows)
            bytes_done += len(rows) * (m.nblk * 6 + 2 * m.T + 2)
        rows_done += done
        mats.append(f"{m.name} {m.M}x{m.K}" + ("" if done == m.M else f" ({done} rows)"))
    return {
        "value": round(bytes_done / t_used / 1e9, 6), "unit": "GB/s", "cores": 1,
        "kind": "oracle",
        "sample": f"{len(mats)} matrices of the step in step order "
                  f"[{', '.join(mats)}], {rows_done} rows in {t_used:.1f} s, "
                  f"float64 numpy, batch {plan[0][1].shape[0]}",
    }


KERNEL_SOURCES = ("paper_2609_35465_amd/csrc/kernels.h", "paper_2609_35465_amd/csrc/device_tables.h",
                  "paper_2609_35465_amd/csrc/word_format.h", "paper_2609_35465_amd/csrc/tetra.hip")
TRAFFIC_PROFILE = "profiles/gemv_kernel_qwen3-14b-40-layers_traffic.md"


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()


def recorded_traffic(args, layers):
    """HBM bytes per gemv launch from the committed counter profile, or None
    when the profile is absent, was taken on another workload, or the kernel
    sources have changed since it was taken."""
    path = os.path.join(ROOT, TRAFFIC_PROFILE)
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].strip().split(": ", 1)
            rec[k] = v.strip().strip("`")
    want = {"source_sha256": kernel_source_hash(), "mode": args.mode,
            "batch": str(args.batch), "model": args.model, "layers": str(layers)}
    if any(rec.get(k) != v for k, v in want.items()):
        return None
    try:
        return int(rec["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: the fused GEMV has no multi-GPU path in "
              "this build (rows shard without communication; see the design notes). "
              "Run with --gpus 1.", file=sys.stderr)
        return 2
    import torch
    import paper_2609_35465_amd as tt

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_probe_mib:
        n = args.copy_probe_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").random_(0, 256)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        assert torch.equal(src, dst)
        print(json.dumps({"copy_probe_bytes": n, "copies": 5}), flush=True)
        return 0
    stream = torch.cuda.current_stream()
    plan, L = build_workload(torch, tt, args.model, args.layers, args.batch)
    torch.cuda.synchronize()

    bytes_read = sum(m.read_bytes for m, _, _ in plan)
    bytes_xy = sum(2 * m.K * args.batch + 4 * m.M * args.batch for m, _, _ in plan)
    weights = sum(m.weights for m, _, _ in plan)
    algo_bytes = bytes_read + bytes_xy

    launches = build_launches(tt, plan, args.mode)
    # warm-up (also uploads the decoder tables)
    for _ in range(max(1, args.warmup)):
        run_step(tt, launches, args.batch, stream.cuda_stream)
    torch.cuda.synchronize()
    parity = parity_spot_check(torch, tt, plan, args.batch)

    graph = None
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            run_step(tt, launches, args.batch, torch.cuda.current_stream().cuda_stream)
        # replays must reproduce the eager result
        ref = [y.clone() for _, _, y in plan[:7]]
        for _ in range(3):
            for _, _, y in plan[:7]:
                y.zero_()
            graph.replay()
            torch.cuda.synchronize()
            for r, (_, _, y) in zip(ref, plan[:7]):
                assert torch.equal(r, y), "graph replay differs from the eager run"

    def step():
        if graph is not None:
            graph.replay()
        else:
            run_step(tt, launches, args.batch, stream.cuda_stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps

    # average gemv_kernel launch over the timed region (HIP events on the
    # launch stream; the step is nothing but back-to-back gemv launches)
    avg_launch_ms = ms_step / len(launches)
    achieved = (algo_bytes / len(launches)) / (avg_launch_ms * 1e-3) / 1e9
    traffic = recorded_traffic(args, L)

    value = algo_bytes / (ms_step * 1e-3) / 1e9
    bits_w = bytes_read * 8 / weights
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16-in/f32-acc",
        "data": "synthetic",
        "config": {
            "workload": f"Qwen3-{args.model}-shaped linear set x {L} layers "
                        f"({len(plan)} Tetra matrices), batch {args.batch}, one token-equivalent pass",
            "batch": args.batch, "layers": L, "matrices": len(plan),
            "hip_graph": graph is not None, "launches_per_step": len(launches),
            "launch_grouping": args.mode,
        },
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "bits_read_per_weight": round(bits_w, 4),
        "weights_per_s": round(weights / (ms_step * 1e-3), 1),
        "token_equiv_latency_ms": round(ms_step, 4),
        "parity_worst_rel_err": parity,
        "roofline": {
            "bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
            "kernel": "gemv_kernel", "avg_launch_us": round(avg_launch_ms * 1e3, 3),
            "bytes_per_launch": round(algo_bytes / len(launches)),
        },
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(torch, tt, plan, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
