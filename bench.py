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
import re
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
    ap.add_argument("--chain-layers", type=int, default=4,
                    help="--mode chain: layers per launch (a launch holds at most 32 matrices and 16 phases: 4 layers)")
    ap.add_argument("--no-deps-figure", action="store_true",
                    help="--mode chain: skip timing the same step as 160 separate launches")
    ap.add_argument("--mode", default="chain", choices=["matrix", "deps", "layer", "chain"],
                    help="matrix: one launch per matrix; deps: per layer [q,k,v] [o] "
                         "[gate,up] [down] as four launches (the dependency groups of a "
                         "decode step); chain: the same groups as the phases of one "
                         "tetra_gemv_chain launch per --chain-layers layers, each phase "
                         "starting after the one before has finished on every workgroup; "
                         "layer: one grouped launch per layer (not a legal decode order)")
    ap.add_argument("--workload", default="tetra",
                    choices=["tetra", "c4", "head", "rotate", "prefill", "encode", "single", "stream"],
                    help="tetra: every projection a Tetra matrix (the GEMV metric); c4: the "
                         "full decode step -- 10%% of the projections (seeded) stored as int4 "
                         "w4g128 and one 4-bit embedding row gathered per step; head: the "
                         "4-bit output head GEMV (151936 x 5120, groups of 64) alone; rotate: "
                         "the online activation rotations of one layer; prefill: a 203-token "
                         "prompt through the Tetra projections on the matrix cores; single: "
                         "the one 1536 x 1536 matrix at batch 1, over distinct copies (cold "
                         "buffers); stream: the achievable HBM read rate of this GPU (a "
                         "plain reduction over distinct buffers, no Tetra code)")
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


class Int4Matrix:
    """One int4 (w4g128, fp16 scale/offset per group) projection on the GPU."""

    def __init__(self, torch, name, M, K, gen):
        self.name, self.M, self.K = name, M, K
        self.q = torch.empty((M, K // 2), dtype=torch.uint8, device="cuda").random_(0, 256, generator=gen)
        scale = (torch.rand((M, K // 128), generator=gen, device="cuda") * 1.5 + 0.5) * (1e-2 / 8)
        self.so = torch.stack([scale, -7.5 * scale], dim=-1).half().contiguous()
        self.read_bytes = M * K // 2 + M * (K // 128) * 4
        self.weights = M * K


class Emb4Table:
    """The 4-bit embedding table (groups of 64) and the token gathered per step."""

    def __init__(self, torch, rows, dim, gen, token):
        self.rows, self.dim = rows, dim
        self.q = torch.empty((rows, dim // 2), dtype=torch.uint8, device="cuda").random_(0, 256, generator=gen)
        scale = (torch.rand((rows, dim // 64), generator=gen, device="cuda") * 1.5 + 0.5) * (1e-2 / 8)
        self.so = torch.stack([scale, -7.5 * scale], dim=-1).half().contiguous()
        self.tokens = torch.tensor([token], dtype=torch.int32, device="cuda")
        self.out = torch.empty((1, dim), dtype=torch.float32, device="cuda")
        self.read_bytes = dim // 2 + (dim // 64) * 4


def build_workload(torch, tt, model, layers, batch, workload="tetra"):
    from paper_2609_35465_amd import workloads
    shapes = workloads.layer_shapes(model)
    L = layers or workloads.QWEN3[model]["layers"]
    gen = torch.Generator(device="cuda").manual_seed(workloads.SEED_BASE + 3)
    n_total = L * len(shapes)
    int4_set = set()
    if workload == "c4":
        int4_set = set(workloads.int4_pick(workloads.SEED_BASE + 4, n_total).tolist())
    mats, xs, ys = [], {}, []
    for layer in range(L):
        for i, (name, M, K) in enumerate(shapes):
            li = layer * len(shapes) + i
            if li in int4_set:
                mats.append(Int4Matrix(torch, name, M, K, gen))
            else:
                mats.append(Matrix(torch, tt, name, M, K, gen, workloads.seed_for(3, 16 * layer + i)))
            if (layer, K) not in xs:
                xs[(layer, K)] = torch.randn(batch, K, generator=gen, device="cuda").half()
            ys.append(torch.empty(batch, M, dtype=torch.float32, device="cuda"))
    plan = [(m, xs[(li // len(shapes), m.K)], ys[li]) for li, m in enumerate(mats)]
    emb = None
    if workload == "c4":
        q = workloads.QWEN3[model]
        emb = Emb4Table(torch, 151936, q["hidden"], gen, token=int(workloads.SEED_BASE % 151936))
    return plan, L, emb


GROUPS = {
    "matrix": [["q"], ["k"], ["v"], ["o"], ["gate"], ["up"], ["down"]],
    "deps": [["q", "k", "v"], ["o"], ["gate", "up"], ["down"]],
    "layer": [["q", "k", "v", "o", "gate", "up", "down"]],
}


def build_chains(tt, plan, chain_layers, nproj=7):
    """Launches of one step as chains: the dependency groups of chain_layers
    layers are the phases of one tetra_gemv_chain launch; a group with int4
    members ends its chain (its Tetra members are the chain's last phase) and
    its int4 members run next, so the order of the groups is kept."""
    launches = []
    cur, counts, mats = [], [], []

    def flush():
        if counts:
            launches.append(("chain", tt.make_problems(cur), list(counts), list(mats)))
        cur.clear(), counts.clear(), mats.clear()

    for l0 in range(0, len(plan), nproj):
        if (l0 // nproj) % chain_layers == 0:
            flush()
        layer = plan[l0:l0 + nproj]
        by_name = {m.name: (m, x, y) for m, x, y in layer}
        for names in GROUPS["deps"]:
            tet = [n for n in names if isinstance(by_name[n][0], Matrix)]
            i4 = [n for n in names if not isinstance(by_name[n][0], Matrix)]
            if tet and (len(cur) + len(tet) > tt.MAX_GROUP or len(counts) == tt.MAX_PHASES):
                flush()
            if tet:
                cur.extend((by_name[n][0].blob, by_name[n][0].sigma, by_name[n][1], by_name[n][2],
                            by_name[n][0].M, by_name[n][0].K) for n in tet)
                counts.append(len(tet))
                mats.extend(by_name[n][0] for n in tet)
            if i4:
                flush()
                for n in i4:
                    launches.append(("int4",) + by_name[n])
    flush()
    return launches


def build_launches(tt, plan, mode, nproj=7, emb=None, chain_layers=1):
    """Launches of one step, in order: ("tetra", problem array, matrices),
    ("chain", problem array, phase counts, matrices), ("int4", matrix, x, y)
    or ("emb4", table)."""
    launches = []
    if emb is not None:
        launches.append(("emb4", emb))
    if mode == "chain":
        return launches + build_chains(tt, plan, chain_layers, nproj)
    for l0 in range(0, len(plan), nproj):
        layer = plan[l0:l0 + nproj]
        by_name = {m.name: (m, x, y) for m, x, y in layer}
        for names in GROUPS[mode]:
            tet = [n for n in names if isinstance(by_name[n][0], Matrix)]
            if tet:
                items = [(by_name[n][0].blob, by_name[n][0].sigma, by_name[n][1], by_name[n][2],
                          by_name[n][0].M, by_name[n][0].K) for n in tet]
                launches.append(("tetra", tt.make_problems(items), [by_name[n][0] for n in tet]))
            for n in names:
                if not isinstance(by_name[n][0], Matrix):
                    launches.append(("int4",) + by_name[n])
    return launches


def run_step(tt, launches, batch, stream, only_tetra=False):
    for ln in launches:
        if ln[0] == "tetra":
            tt.gemv_grouped(ln[1], batch, stream)
        elif ln[0] == "chain":
            tt.gemv_chain(ln[1], ln[2], batch, None, stream)
        elif only_tetra:
            continue
        elif ln[0] == "int4":
            m, x, y = ln[1:]
            tt.int4_gemv(m.q, m.so, x, y, m.M, m.K, batch, stream)
        else:
            e = ln[1]
            tt.emb4_gather(e.q, e.so, e.rows, e.dim, e.tokens, e.out, stream)


def parity_spot_check(torch, tt, plan, batch):
    """Sampled rows of the first matrices of each shape against the oracle."""
    from oracle import gemv as ogemv
    worst = 0.0
    seen = set()
    for m, x, y in plan:
        if m.name in seen or not isinstance(m, Matrix):
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


def parity_spot_check_int4(torch, plan):
    """Sampled rows of each int4 shape against the oracle (worst relative error)."""
    from oracle import int4 as oint4
    worst, seen = 0.0, set()
    for m, x, y in plan:
        if isinstance(m, Matrix) or m.name in seen:
            continue
        seen.add(m.name)
        rows = np.unique(np.r_[0:8, m.M - 8:m.M, np.linspace(0, m.M - 1, 24).astype(int)])
        ref, norm = oint4.int4_gemv_f64(m.q.cpu().numpy(), m.so.cpu().numpy(), x.cpu().numpy(), rows=rows)
        got = y.cpu().numpy()[:, rows].astype(np.float64)
        worst = max(worst, float((np.abs(got - ref) / norm).max()))
    return worst


_CPU_DATA = []


def _cpu_init(paths):
    """Pool worker set-up: memory-map the host copies of the sampled matrices."""
    global _CPU_DATA
    _CPU_DATA = [tuple(np.load(os.path.join(d, f + ".npy"), mmap_mode="r") for f in ("w", "s", "t", "x"))
                 for d in paths]


def _cpu_task(task):
    """One chunk of rows of one sampled matrix through the oracle."""
    from oracle import gemv as ogemv
    mi, r0, r1 = task
    words, sig, tail, x = _CPU_DATA[mi]
    ogemv.gemv_f64(words, sig, tail if tail.size else None, x, rows=np.arange(r0, r1))
    return mi, r1 - r0


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(torch, tt, plan, seconds):
    """The CPU oracle as it stands (float64 numpy, oracle.gemv.gemv_f64) over
    the step's matrices in step order, 2048 rows per task, run by a pool of
    worker processes on the host's cores (at most 16, the host share of one
    GPU), until about `seconds` of wall time; rate in GB/s of Tetra bytes
    (6 B per block, 2 B per tail weight and row scale).  A single-process run
    on the first matrix first gives the one-core rate and sizes the sample.
    Copying matrices to the host and unpacking them are not timed."""
    import multiprocessing as mp
    import shutil
    import tempfile
    from oracle import gemv as ogemv
    cores = max(1, min(16, len(os.sched_getaffinity(0))))
    tmp = tempfile.mkdtemp(prefix="tetra_cpu_")
    try:
        paths, sizes, names = [], [], []

        def host_copy(m, x):
            d = os.path.join(tmp, str(len(paths)))
            os.makedirs(d)
            words, tail = tt.unpack_rows(m.blob.cpu().numpy(), m.M, m.K)
            np.save(os.path.join(d, "w.npy"), words)
            np.save(os.path.join(d, "s.npy"), m.sigma.cpu().numpy())
            np.save(os.path.join(d, "t.npy"), tail if tail is not None else np.zeros((0,), np.float16))
            np.save(os.path.join(d, "x.npy"), x.cpu().numpy())
            paths.append(d)
            sizes.append(m.nblk * 6 + 2 * m.T + 2)
            names.append(f"{m.name} {m.M}x{m.K}")

        tetra = [(m, x) for m, x, _ in plan if isinstance(m, Matrix)]
        host_copy(*tetra[0])
        # one core: rows of the first matrix for about a tenth of the budget
        _cpu_init(paths)
        M0 = tetra[0][0].M
        t0, rows1 = time.perf_counter(), 0
        while time.perf_counter() - t0 < seconds / 10:
            r0 = rows1 % M0
            _cpu_task((0, r0, min(r0 + 2048, M0)))
            rows1 += min(r0 + 2048, M0) - r0
        t1 = time.perf_counter() - t0
        rate1 = rows1 * sizes[0] / t1
        # the pool's sample: the step's matrices in order, about `seconds` of
        # work (at most 24 matrices), cycled through until the time is used
        want = rate1 * cores * seconds
        have = tetra[0][0].M * sizes[0]
        for m, x in tetra[1:24]:
            if have >= want:
                break
            host_copy(m, x)
            have += m.M * sizes[-1]
        chunks = [(i, r0, min(r0 + 2048, tetra[i][0].M)) for i in range(len(paths))
                  for r0 in range(0, tetra[i][0].M, 2048)]
        ctx = mp.get_context("spawn")
        with ctx.Pool(cores, initializer=_cpu_init, initargs=(paths,)) as pool:
            pool.map(_cpu_task, [(0, 0, 1)] * cores)          # workers up and warm
            done_rows = [0] * len(paths)
            pending, k = [], 0
            t0 = time.perf_counter()
            # two chunks in flight per worker, new ones only while time is left
            while True:
                while len(pending) < 2 * cores and time.perf_counter() - t0 < seconds:
                    pending.append(pool.apply_async(_cpu_task, (chunks[k % len(chunks)],)))
                    k += 1
                if not pending:
                    break
                mi, n = pending.pop(0).get()
                done_rows[mi] += n
            wall = time.perf_counter() - t0
        bytes_done = sum(r * sz for r, sz in zip(done_rows, sizes))
        return {
            "value": round(bytes_done / wall / 1e9, 6), "unit": "GB/s", "cores": cores,
            "kind": "oracle",
            "sample": f"the first {len(paths)} matrices of the step in step order "
                      f"[{', '.join(names[:7])}{', ...' if len(names) > 7 else ''}], cycled: "
                      f"{sum(done_rows)} rows in {wall:.1f} s on {cores} worker processes, float64 numpy "
                      f"(oracle.gemv.gemv_f64), batch {plan[0][1].shape[0]}; host CPU {cpu_model()}",
            "single_core_gbs": round(rate1 / 1e9, 6),
        }
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


KERNEL_SOURCES = ("paper_2609_35465_amd/csrc/kernels.h", "paper_2609_35465_amd/csrc/device_tables.h",
                  "paper_2609_35465_amd/csrc/word_format.h")
LAUNCH_SOURCE = "paper_2609_35465_amd/csrc/tetra.hip"
TRAFFIC_PROFILE = "profiles/gemv_kernel_qwen3-14b-40-layers_traffic.md"


def _code_only(text):
    """C++ source without its comments and blank lines, trailing spaces
    stripped: a change to a comment leaves the hash below as it was."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    out = []
    for line in text.split("\n"):
        i = line.find("//")
        while i >= 0 and line.count('"', 0, i) % 2 == 1:     # inside a string literal
            i = line.find("//", i + 2)
        if i >= 0:
            line = line[:i]
        line = line.rstrip()
        if line:
            out.append(line)
    return "\n".join(out)


def kernel_source_hash():
    """sha256 over what decides the measured kernel: the device sources of the
    GEMV, its launch planning (the `launch_gemv` function of the library) and
    the compiler flags, comments left out."""
    import hashlib
    from paper_2609_35465_amd import build as _build
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(_code_only(open(os.path.join(ROOT, f), encoding="utf-8").read()).encode())
    lines = open(os.path.join(ROOT, LAUNCH_SOURCE), encoding="utf-8").read().split("\n")
    start = next(i for i, l in enumerate(lines) if l.startswith("int launch_gemv("))
    end = next(i for i in range(start, len(lines)) if lines[i] == "}")
    h.update(_code_only("\n".join(lines[start:end + 1])).encode())
    h.update(" ".join(_build.HIP_FLAGS).encode())
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
            "batch": str(args.batch), "model": args.model, "layers": str(layers),
            "workload": args.workload}
    if any(rec.get(k) != v for k, v in want.items()):
        return None
    try:
        return int(rec["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


HEAD_ROWS, HEAD_DIM = 151936, 5120


def main_head(args, torch, tt):
    """The 4-bit output head (151,936 x 5,120, groups of 64): one
    tetra_head4_gemv launch per step, alternating between two copies of the
    table (876 MB together, more than the last-level cache) so that every
    launch streams from HBM."""
    from oracle import int4 as oint4
    rows, dim, B = HEAD_ROWS, HEAD_DIM, args.batch
    gen = torch.Generator(device="cuda").manual_seed(0x7E7A_0000 + 0x50)
    tables = []
    for _ in range(2):
        q = torch.empty((rows, dim // 2), dtype=torch.uint8, device="cuda").random_(0, 256, generator=gen)
        sc = (torch.rand((rows, dim // 64), generator=gen, device="cuda") * 1.5 + 0.5) * (1e-2 / 8)
        tables.append((q, torch.stack([sc, -7.5 * sc], dim=-1).half().contiguous()))
    from paper_2609_35465_amd import workloads
    x = torch.as_tensor(workloads.activations(0x7E7A_0050, B, dim)).cuda()
    ys = [torch.empty((B, rows), dtype=torch.float32, device="cuda") for _ in tables]
    stream = torch.cuda.current_stream()

    def step_pair(s=None):
        st = (s or stream).cuda_stream
        for (q, so), y in zip(tables, ys):
            tt.head4_gemv(q, so, x, y, rows, dim, B, stream=st)

    for _ in range(max(1, args.warmup)):
        step_pair()
    torch.cuda.synchronize()
    # parity: sampled rows of both tables against the oracle
    sample = np.unique(np.r_[0:8, rows - 8:rows, np.linspace(0, rows - 1, 48).astype(int)])
    idx = torch.as_tensor(sample, device="cuda")
    worst = 0.0
    for (q, so), y in zip(tables, ys):
        ref, norm = oint4.int4_gemv_f64(q[idx].cpu().numpy(), so[idx].cpu().numpy(), x.cpu().numpy(), group=64)
        got = y.cpu().numpy()[:, sample].astype(np.float64)
        worst = max(worst, float((np.abs(got - ref) / norm).max()))
    graph = None
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step_pair(torch.cuda.current_stream())
        ref = [y.clone() for y in ys]
        for _ in range(3):
            for y in ys:
                y.zero_()
            graph.replay()
            torch.cuda.synchronize()
            assert all(torch.equal(r, y) for r, y in zip(ref, ys)), "graph replay differs from the eager run"
    run = graph.replay if graph is not None else step_pair
    pairs = max(1, args.steps // 2)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(pairs):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / (2 * pairs)
    read_bytes = rows * dim // 2 + rows * (dim // 64) * 4
    algo = read_bytes + 2 * dim * B + 4 * rows * B
    value = algo / (ms_step * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": 2 * pairs,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f16-in/f32-acc", "data": "synthetic",
        "config": {"workload": f"4-bit output head {rows} x {dim}, groups of 64, batch {B}, "
                               "two tables alternating", "batch": B, "hip_graph": graph is not None},
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "bits_read_per_weight": round(read_bytes * 8 / (rows * dim), 4),
        "weights_per_s": round(rows * dim / (ms_step * 1e-3), 1),
        "parity_head4_worst_rel_err": worst,
        "roofline": {"bound": "hbm", "achieved": round(value, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(value / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "int4_gemv_kernel (groups of 64)", "avg_launch_us": round(ms_step * 1e3, 3),
                     "bytes_per_launch": algo},
    }
    if not args.no_cpu_baseline:
        # the oracle on 2048-row slices of the first table until the time is used
        q, so = tables[0]
        xh = x.cpu().numpy()
        t_used, done = 0.0, 0
        for r0 in range(0, rows, 2048):
            if t_used >= args.cpu_seconds:
                break
            qs, ss = q[r0:r0 + 2048].cpu().numpy(), so[r0:r0 + 2048].cpu().numpy()
            t0 = time.perf_counter()
            oint4.int4_gemv_f64(qs, ss, xh, group=64)
            t_used += time.perf_counter() - t0
            done += len(qs)
        out["cpu_baseline"] = {
            "value": round(done * (dim // 2 + (dim // 64) * 4) / t_used / 1e9, 6), "unit": "GB/s",
            "cores": 1, "kind": "oracle",
            "sample": f"{done} rows of the head in {t_used:.1f} s, float64 numpy, batch {B}"}
    print(json.dumps(out), flush=True)
    return 0


def main_rotate(args, torch, tt):
    """The online activation rotation at the 14B widths: per decode layer one
    rotation of the hidden vector (5,120, blocks of 1,024) for the q/k/v and
    gate/up groups each, one of the attention output (5,120) for o, and one of
    the intermediate vector (17,408, blocks of 1,024) for down.  A step is the
    four rotations of one layer, replayed from a HIP graph."""
    from oracle import rotation as orot
    from paper_2609_35465_amd import workloads
    B = args.batch
    widths = [(5120, 1024), (5120, 1024), (5120, 1024), (17408, 1024)]
    rng = np.random.default_rng(0x7E7A_0060)
    bufs = []
    for K, n in widths:
        x = torch.as_tensor(workloads.activations(0x7E7A_0060 + K, B, K)).cuda()
        bits = torch.as_tensor(rng.integers(0, 256, (K + 7) // 8, dtype=np.uint8)).cuda()
        bufs.append((x, bits, torch.empty_like(x), K, n))
    stream = torch.cuda.current_stream()

    def step(s=None):
        st = (s or stream).cuda_stream
        for x, bits, out, K, n in bufs:
            tt.rotate(x, bits, out, K, n, B, stream=st)

    step()
    torch.cuda.synchronize()
    worst = 0.0
    for x, bits, out, K, n in bufs:
        ref = orot.rotate_f64(x.cpu().numpy(), bits.cpu().numpy(), n)
        got = out.cpu().numpy().astype(np.float64)
        worst = max(worst, float((np.abs(got - ref) / np.maximum(np.abs(ref), 1e-3)).max()))
    graph = None
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step(torch.cuda.current_stream())
    run = graph.replay if graph is not None else step
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    algo = sum(4 * K * B + (K + 7) // 8 for _, _, _, K, _ in bufs)
    value = algo / (ms_step * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32 (fp16 in/out)", "data": "synthetic",
        "config": {"workload": f"online rotation of one 14B layer's activations: 3 x 5120 + 17408, "
                               f"Hadamard blocks of 1024, batch {B}", "batch": B, "hip_graph": graph is not None},
        "us_per_rotation": round(ms_step * 1e3 / len(bufs), 3),
        "rotate_worst_rel_err": worst,
        "roofline": {"bound": "hbm", "achieved": round(value, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(value / HBM_PEAK_GBS, 6), "traffic": None, "kernel": "rotate_kernel",
                     "avg_launch_us": round(ms_step * 1e3 / len(bufs), 3),
                     "bytes_per_launch": round(algo / len(bufs))},
    }
    if not args.no_cpu_baseline:
        xs = [(x.cpu().numpy(), bits.cpu().numpy(), K, n) for x, bits, _, K, n in bufs]
        t_used, done = 0.0, 0
        while t_used < min(args.cpu_seconds, 10.0):
            for xh, bh, K, n in xs:
                t0 = time.perf_counter()
                orot.rotate_f64(xh, bh, n)
                t_used += time.perf_counter() - t0
            done += 1
        out["cpu_baseline"] = {"value": round(done * algo / t_used / 1e9, 6), "unit": "GB/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"{done} layers' rotations (dense float64 Hadamard blocks) in {t_used:.1f} s"}
    print(json.dumps(out), flush=True)
    return 0


PREFILL_TOKENS = 203
MFMA_F16_PEAK_TFLOPS = 2500.0


def main_prefill(args, torch, tt):
    """A prompt through the Tetra projections: the 14B linear set of
    `--layers` layers (default 4) at 203 tokens, one tetra_gemm launch per
    matrix, replayed from a HIP graph."""
    from paper_2609_35465_amd import workloads
    from oracle import gemv as ogemv
    N = PREFILL_TOKENS
    L = args.layers or 4
    shapes = workloads.layer_shapes(args.model)
    gen = torch.Generator(device="cuda").manual_seed(0x7E7A_0070)
    mats, xs = [], {}
    for layer in range(L):
        for i, (name, M, K) in enumerate(shapes):
            m = Matrix(torch, tt, name, M, K, gen, workloads.seed_for(3, layer * len(shapes) + i))
            if K not in xs:
                xs[K] = torch.as_tensor(workloads.activations(0x7E7A_0070 + K, N, K)).cuda()
            mats.append((m, xs[K], torch.empty((N, M), dtype=torch.float32, device="cuda")))
    stream = torch.cuda.current_stream()
    ws = tt.gemm_workspace()

    def step(s=None):
        st = (s or stream).cuda_stream
        for m, x, y in mats:
            tt.gemm(m.blob, m.sigma, x, y, m.M, m.K, N, ws, stream=st)

    step()
    torch.cuda.synchronize()
    # parity: sampled rows of one matrix of each shape against the oracle
    worst = 0.0
    for m, x, y in mats[:len(shapes)]:
        blob = m.blob.cpu().numpy()
        words, tail = tt.unpack_rows(blob, m.M, m.K)
        rows = np.unique(np.r_[0:4, m.M - 4:m.M, np.linspace(0, m.M - 1, 8).astype(int)])
        ref, norm = ogemv.gemv_f64(words, m.sigma.cpu().numpy(), tail, x.cpu().numpy(), rows=rows)
        got = y.cpu().numpy()[:, rows].astype(np.float64)
        worst = max(worst, float((np.abs(got - ref) / norm).max()))
    graph = None
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step(torch.cuda.current_stream())
    run = graph.replay if graph is not None else step
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    steps = max(1, args.steps // 4)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / steps
    flops = sum(2.0 * m.M * m.K * N for m, _, _ in mats)
    tflops = flops / (ms_step * 1e-3) / 1e12
    bytes_read = sum(m.read_bytes for m, _, _ in mats)
    out = {
        "metric": METRIC, "value": round(bytes_read / (ms_step * 1e-3) / 1e9, 2), "unit": "GB/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f16 (MFMA), f32 acc",
        "data": "synthetic",
        "config": {"workload": f"prompt of {N} tokens through the Qwen3-{args.model}-shaped linear set x {L} "
                               f"layers ({len(mats)} Tetra matrices)", "tokens": N, "layers": L,
                   "hip_graph": graph is not None, "launches_per_step": len(mats)},
        "tflops": round(tflops, 2),
        "parity_worst_rel_err": worst,
        "roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": MFMA_F16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tflops / MFMA_F16_PEAK_TFLOPS, 4), "traffic": None,
                     "kernel": "gemm_kernel", "avg_launch_us": round(ms_step * 1e3 / len(mats), 3),
                     "flops_per_launch": round(flops / len(mats))},
    }
    if not args.no_cpu_baseline:
        # the oracle on 256-row slices of the first matrices, all tokens, until the time is used
        t_used, fl = 0.0, 0.0
        for m, x, _ in mats:
            if t_used >= args.cpu_seconds:
                break
            words, tail = tt.unpack_rows(m.blob.cpu().numpy(), m.M, m.K)
            sig, xh = m.sigma.cpu().numpy(), x.cpu().numpy()
            for r0 in range(0, m.M, 256):
                if t_used >= args.cpu_seconds:
                    break
                rows = np.arange(r0, min(r0 + 256, m.M))
                t0 = time.perf_counter()
                ogemv.gemv_f64(words, sig, tail, xh, rows=rows)
                t_used += time.perf_counter() - t0
                fl += 2.0 * len(rows) * m.K * N
        out["cpu_baseline"] = {"value": round(fl / t_used / 1e12, 6), "unit": "TFLOP/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"{fl / (2 * N) / 1e6:.1f} M weights x {N} tokens in {t_used:.1f} s, "
                                         "float64 numpy"}
    print(json.dumps(out), flush=True)
    return 0


ENCODE_BLOCKS = 20000
VALU32_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12      # 32-bit vector lane operations per second, in T


def main_encode(args, torch, tt):
    """The encoder on the paper's retention workload: 20,000 Gaussian blocks of
    24 weights (unit variance, row scale 1), two trial radii, one launch."""
    from oracle import encoder as oencoder
    n = ENCODE_BLOCKS
    rng = np.random.default_rng(0x7E7A_0080)
    w = rng.standard_normal((n, 24)).astype(np.float32)
    wd = torch.from_numpy(w).cuda()
    sd = torch.ones(n, dtype=torch.float32, device="cuda")
    out = torch.zeros(3 * n, dtype=torch.int16, device="cuda")
    stream = torch.cuda.current_stream()

    def run():
        tt.encode(wd, sd, n, out, stream=stream.cuda_stream)

    run()
    torch.cuda.synchronize()
    b = out.cpu().numpy().view(np.uint16).reshape(n, 3).astype(np.uint64)
    words = b[:, 0] | (b[:, 1] << np.uint64(16)) | (b[:, 2] << np.uint64(32))
    rec = oencoder.reconstruct(words, np.ones(n))
    mse = float(((w.astype(np.float64) - rec) ** 2).mean())
    # parity: sampled blocks against the oracle, word for word
    idx = rng.choice(n, 4, replace=False)
    mism = int((oencoder.encode_blocks(w[idx], 1.0, tt.ENCODE_RADII) != words[idx]).sum())
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    steps = max(1, args.steps // 4)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / steps
    # the definition's work: every (p, pattern byte) pair scores every row of
    # each section's lists (4096 + 2048 + 4096 rows) with 8 additions, per
    # trial radius; the kernel builds the eight scores of a thread's (p, byte)
    # pairs from shared partial sums, 22 additions per row instead of 64, and
    # the roofline counts those it executes
    adds = 2.0 * 256 * (4096 + 2048 + 4096) * 8 * n
    executed = adds * 22.0 / 64.0
    tops = executed / (ms_step * 1e-3) / 1e12
    tops_def = adds / (ms_step * 1e-3) / 1e12
    out_j = {
        "metric": "Tetra encoder throughput, 24-weight blocks per second", "value": round(n / (ms_step * 1e-3), 1),
        "unit": "blocks/s", "n_gpus": 1, "steps": steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "i32 scores, f64 choices",
        "data": "synthetic",
        "config": {"workload": f"{n} Gaussian blocks of 24 weights, radii {tt.ENCODE_RADII[0]:g} and "
                               f"{tt.ENCODE_RADII[1]:g}", "blocks": n},
        "retention": round(oencoder.retention(mse), 5), "mse_per_weight": round(mse, 6),
        "parity_sampled_mismatches": mism,
        "roofline": {"bound": "alu", "achieved": round(tops, 3), "peak": round(VALU32_PEAK_TOPS, 1),
                     "unit": "Tops/s", "frac": round(tops / VALU32_PEAK_TOPS, 4), "traffic": None,
                     "kernel": "encode_kernel", "avg_launch_us": round(ms_step * 1e3, 1),
                     "ops": "executed 32-bit score additions (22 per list row and eight (p, byte) pairs)",
                     "ops_per_launch": executed,
                     "effective": {"achieved": round(tops_def, 3), "frac": round(tops_def / VALU32_PEAK_TOPS, 4),
                                   "ops": "the definition's 8 additions per (p, byte) pair and list row",
                                   "ops_per_launch": adds}},
    }
    if not args.no_cpu_baseline:
        t_used, done = 0.0, 0
        while t_used < min(args.cpu_seconds, 15.0) and done < n:
            t0 = time.perf_counter()
            oencoder.encode_block(w[done], 1.0, tt.ENCODE_RADII)
            t_used += time.perf_counter() - t0
            done += 1
        out_j["cpu_baseline"] = {"value": round(done / t_used, 3), "unit": "blocks/s", "cores": 1, "kind": "oracle",
                                 "sample": f"the first {done} blocks in {t_used:.1f} s, numpy"}
    print(json.dumps(out_j), flush=True)
    return 0


def main_single(args, torch, tt):
    """The one 1536 x 1536 matrix at batch 1 (the smallest configuration):
    one tetra_gemv per launch, over enough distinct copies of the packed
    matrix (at least 1 GiB) that no launch finds its codes in a cache;
    the launches run back to back in a HIP graph."""
    from oracle import gemv as ogemv
    stream = torch.cuda.current_stream()
    gen = torch.Generator(device="cuda").manual_seed(3)
    from paper_2609_35465_amd import workloads
    name, M, K = workloads.single_shape()[0]
    m = Matrix(torch, tt, name, M, K, gen, workloads.seed_for(0, 0))
    x = torch.randn(args.batch, K, generator=gen, device="cuda").half()
    n_copies = -(-(1 << 30) // m.blob.numel())
    blobs = [m.blob.clone() for _ in range(n_copies)]
    y = torch.full((args.batch, M), float("nan"), dtype=torch.float32, device="cuda")
    tt.gemv(blobs[0], m.sigma, x, y, M, K, args.batch)
    torch.cuda.synchronize()
    words, tail = tt.unpack_rows(m.blob.cpu().numpy(), M, K)
    ref, norm = ogemv.gemv_f64(words, m.sigma.cpu().numpy(), tail, x.cpu().numpy())
    parity = float((np.abs(y.cpu().numpy().astype(np.float64) - ref) / norm).max())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for b in blobs:
            tt.gemv(b, m.sigma, x, y, M, K, args.batch, torch.cuda.current_stream().cuda_stream)
    for _ in range(max(1, args.warmup)):
        g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = max(1, args.steps // 4)
    e0.record(stream)
    for _ in range(reps):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_launch = e0.elapsed_time(e1) / (reps * n_copies)
    algo = m.read_bytes + 2 * K * args.batch + 4 * M * args.batch
    value = algo / (ms_launch * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": reps * n_copies,
        "warmup": args.warmup, "ms_per_step": round(ms_launch, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f16-in/f32-acc", "data": "synthetic",
        "config": {"workload": f"single Tetra GEMV {M} x {K}, batch {args.batch}, over {n_copies} distinct "
                               f"copies of the packed matrix ({n_copies * m.blob.numel() / 2**30:.2f} GiB), "
                               f"one launch per step", "batch": args.batch, "hip_graph": True},
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "bits_read_per_weight": round(m.read_bytes * 8 / m.weights, 4),
        "weights_per_s": round(m.weights / (ms_launch * 1e-3), 1),
        "parity_worst_rel_err": parity,
        "roofline": {"bound": "hbm", "achieved": round(value, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(value / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "gemv_kernel",
                     "avg_launch_us": round(ms_launch * 1e3, 3), "bytes_per_launch": algo},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(torch, tt, [(m, x, y)], args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


def main_stream(args, torch):
    """The achievable HBM read rate of this GPU: torch row sums (rows of 4096
    fp32) over 8 distinct 256 MiB buffers (2 GiB in all, far above the
    256 MB last-level cache), one kernel per buffer, back to back on one
    stream; outputs are 1/4096 of the bytes read.  A plain copy of the same
    buffers (read and write counted) is reported beside it."""
    stream = torch.cuda.current_stream()
    n, each, row = 8, 256 << 20, 4096
    bufs = [torch.empty(each // 4, dtype=torch.float32, device="cuda").uniform_().view(-1, row) for _ in range(n)]
    outs = [torch.empty(each // 4 // row, dtype=torch.float32, device="cuda") for _ in range(n)]
    dsts = [torch.empty_like(bufs[0]) for _ in range(2)]

    def reads():
        for b, o in zip(bufs, outs):
            torch.sum(b, 1, out=o)

    def copies():
        for i, b in enumerate(bufs):
            dsts[i % 2].copy_(b)

    def timed(fn):
        for _ in range(max(1, args.warmup)):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps

    ms = timed(reads)
    value = n * each / (ms * 1e-3) / 1e9
    ms_copy = timed(copies)
    print(json.dumps({"metric": "achievable HBM read GB/s (torch row sums over 2 GiB of distinct buffers)",
                      "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
                      "ms_per_step": round(ms, 4), "higher_is_better": True,
                      "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2), "data": "synthetic",
                      "copy_gbs_read_plus_write": round(2 * n * each / (ms_copy * 1e-3) / 1e9, 2),
                      "config": {"workload": "read-only streaming probe", "buffers": n, "buffer_bytes": each,
                                 "row_elements": row}}), flush=True)
    return 0


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (a "
              "matrix's row tiles would shard over GPUs without communication, each "
              "GPU producing its own rows of y). Run with --gpus 1.", file=sys.stderr)
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
    if args.workload == "head":
        return main_head(args, torch, tt)
    if args.workload == "rotate":
        return main_rotate(args, torch, tt)
    if args.workload == "prefill":
        return main_prefill(args, torch, tt)
    if args.workload == "encode":
        return main_encode(args, torch, tt)
    if args.workload == "single":
        return main_single(args, torch, tt)
    if args.workload == "stream":
        return main_stream(args, torch)
    stream = torch.cuda.current_stream()
    plan, L, emb = build_workload(torch, tt, args.model, args.layers, args.batch, args.workload)
    torch.cuda.synchronize()

    tetra = [(m, x, y) for m, x, y in plan if isinstance(m, Matrix)]
    bytes_read = sum(m.read_bytes for m, _, _ in plan) + (emb.read_bytes if emb else 0)
    bytes_xy = sum(2 * m.K * args.batch + 4 * m.M * args.batch for m, _, _ in plan)
    weights = sum(m.weights for m, _, _ in plan)
    algo_bytes = bytes_read + bytes_xy
    tetra_bytes = sum(m.read_bytes + 2 * m.K * args.batch + 4 * m.M * args.batch for m, _, _ in tetra)

    launches = build_launches(tt, plan, args.mode, emb=emb, chain_layers=args.chain_layers)
    n_tetra = sum(1 for ln in launches if ln[0] in ("tetra", "chain"))
    # warm-up (also uploads the decoder tables and sets up the workspace)
    for _ in range(max(1, args.warmup)):
        run_step(tt, launches, args.batch, stream.cuda_stream)
    torch.cuda.synchronize()
    parity = parity_spot_check(torch, tt, plan, args.batch)
    parity_int4 = parity_spot_check_int4(torch, plan) if args.workload == "c4" else None

    def capture(only_tetra):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            run_step(tt, launches, args.batch, torch.cuda.current_stream().cuda_stream, only_tetra)
        # replays must reproduce the eager result
        check = [(m, x, y) for m, x, y in plan[:7] if isinstance(m, Matrix) or not only_tetra]
        ref = [y.clone() for _, _, y in check]
        for _ in range(3):
            for _, _, y in check:
                y.zero_()
            g.replay()
            torch.cuda.synchronize()
            for r, (_, _, y) in zip(ref, check):
                assert torch.equal(r, y), "graph replay differs from the eager run"
        return g

    graph = None if args.no_graph else capture(False)

    def timed(step, steps):
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            step()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    if graph is not None:
        ms_step = timed(graph.replay, args.steps)
    else:
        ms_step = timed(lambda: run_step(tt, launches, args.batch, stream.cuda_stream), args.steps)

    # average gemv_kernel launch over a timed region of back-to-back gemv
    # launches (HIP events on the launch stream): the step itself for the
    # all-Tetra workload, a Tetra-only replay of the same step otherwise
    if args.workload == "tetra":
        tetra_ms = ms_step
    elif graph is not None:
        tetra_ms = timed(capture(True).replay, args.steps)
    else:
        tetra_ms = timed(lambda: run_step(tt, launches, args.batch, stream.cuda_stream, True), args.steps)
    avg_launch_ms = tetra_ms / n_tetra
    achieved = (tetra_bytes / n_tetra) / (avg_launch_ms * 1e-3) / 1e9
    traffic = recorded_traffic(args, L)

    # beside a chained step, the same step as separate launches (one per
    # dependency group: 160 for the 14B set), labelled as such
    deps_fig = None
    if args.mode == "chain" and not args.no_deps_figure:
        dl = build_launches(tt, plan, "deps", emb=emb)
        if graph is not None:
            gd = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gd):
                run_step(tt, dl, args.batch, torch.cuda.current_stream().cuda_stream)
            ms_deps = timed(gd.replay, args.steps)
        else:
            ms_deps = timed(lambda: run_step(tt, dl, args.batch, stream.cuda_stream), args.steps)
        deps_fig = {"launch_grouping": "deps", "launches_per_step": len(dl),
                    "ms_per_step": round(ms_deps, 4),
                    "value": round(algo_bytes / (ms_deps * 1e-3) / 1e9, 2), "unit": "GB/s"}

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
            "workload": (f"Qwen3-{args.model}-shaped linear set x {L} layers "
                         f"({len(tetra)} Tetra matrices), batch {args.batch}, one token-equivalent pass"
                         if args.workload == "tetra" else
                         f"Qwen3-{args.model}-shaped decode step: {L} layers, {len(tetra)} Tetra + "
                         f"{len(plan) - len(tetra)} int4 w4g128 matrices, one 4-bit embedding row of "
                         f"151936 x {emb.dim}, batch {args.batch}"),
            "batch": args.batch, "layers": L, "matrices": len(plan), "tetra_matrices": len(tetra),
            "hip_graph": graph is not None, "launches_per_step": len(launches),
            "launch_grouping": args.mode,
        } | ({"chain_layers": args.chain_layers,
              "phases_per_step": sum(len(ln[2]) for ln in launches if ln[0] == "chain")}
             if args.mode == "chain" else {}),
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "bits_read_per_weight": round(bits_w, 4),
        "weights_per_s": round(weights / (ms_step * 1e-3), 1),
        "token_equiv_latency_ms": round(ms_step, 4),
        "parity_worst_rel_err": parity,
        "parity_int4_worst_rel_err": parity_int4,
        "separate_launches": deps_fig,
        "roofline": {
            "bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
            "kernel": "gemv_kernel", "avg_launch_us": round(avg_launch_ms * 1e3, 3),
            "bytes_per_launch": round(tetra_bytes / n_tetra),
        },
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(torch, tt, plan, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
