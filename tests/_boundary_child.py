"""Child process of the boundary tests in test_gpu_parity.py (run as a
fresh process, so that the library call it makes first is the process's
first).  Usage: python tests/_boundary_child.py MODE; prints one line per
check and exits non-zero on a failure."""

import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import torch  # noqa: E402

import paper_2609_35465_amd as tt  # noqa: E402
from paper_2609_35465_amd import workloads  # noqa: E402
from oracle import gemv as ogemv  # noqa: E402


def packed(seed, M, K):
    words, sigma, tail = workloads.tetra_matrix(seed, M, K)
    blob = torch.from_numpy(tt.pack_rows(words, tail, M, K)).cuda()
    return words, sigma, tail, blob, torch.from_numpy(sigma).cuda()


def worst(words, sigma, tail, x, y):
    ref, norm = ogemv.gemv_f64(words, sigma, tail, x)
    return float((np.abs(y.astype(np.float64) - ref) / norm).max())


def first_call_in_capture():
    """The process's first library call is made while torch captures a graph;
    every replay must match the oracle."""
    M, K = 640, 24 * 70 + 8
    words, sigma, tail, blob, sg = packed(41, M, K)
    x = workloads.activations(41, 1, K)
    xd = torch.from_numpy(x).cuda()
    y = torch.full((1, M), float("nan"), device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        tt.gemv(blob, sg, xd, y, M, K, 1, stream=torch.cuda.current_stream().cuda_stream)
    print("captured", flush=True)
    for r in range(3):
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        e = worst(words, sigma, tail, x, y.cpu().numpy())
        print(f"replay {r}: worst {e:.3e}", flush=True)
        assert e <= 1e-5, e


def two_streams():
    """Two streams run GEMVs on different matrices at the same time, each
    with its own workspace slot: both match the oracle and the bits of a
    one-stream run, every time."""
    shapes = [(4096, 5120), (5120, 17408)]
    mats = [packed(50 + i, M, K) for i, (M, K) in enumerate(shapes)]
    xs = [workloads.activations(60 + i, 1, K) for i, (_, K) in enumerate(shapes)]
    xds = [torch.from_numpy(x).cuda() for x in xs]
    ref_bits, refs = [], []
    for (words, sigma, tail, blob, sg), x, xd, (M, K) in zip(mats, xs, xds, shapes):
        y = torch.empty((1, M), device="cuda")
        tt.gemv(blob, sg, xd, y, M, K, 1)
        torch.cuda.synchronize()
        refs.append(worst(words, sigma, tail, x, y.cpu().numpy()))
        ref_bits.append(y.clone())
    print(f"one stream: worst {max(refs):.3e}", flush=True)
    assert max(refs) <= 1e-5
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    ys = [[torch.full((1, M), float("nan"), device="cuda") for _ in range(8)] for M, _ in shapes]
    for rep in range(8):
        for i, ((words, sigma, tail, blob, sg), (M, K)) in enumerate(zip(mats, shapes)):
            with torch.cuda.stream(streams[i]):
                tt.gemv(blob, sg, xds[i], ys[i][rep], M, K, 1, stream=streams[i].cuda_stream)
    torch.cuda.synchronize()
    for i in range(2):
        for rep in range(8):
            assert torch.equal(ys[i][rep], ref_bits[i]), (i, rep)
    print("two streams: 16 launches equal to the one-stream bits", flush=True)


def busy_slots():
    """A 17th stream is refused with TETRA_EBUSY until a stream gives its
    slot back."""
    M, K = 64, 48
    words, sigma, tail, blob, sg = packed(70, M, K)
    x = torch.from_numpy(workloads.activations(70, 1, K)).cuda()
    y = torch.empty((1, M), device="cuda")
    streams = [torch.cuda.Stream() for _ in range(17)]
    for s in streams[:16]:
        tt.gemv(blob, sg, x, y, M, K, 1, stream=s.cuda_stream)
    try:
        tt.gemv(blob, sg, x, y, M, K, 1, stream=streams[16].cuda_stream)
        raise AssertionError("17th stream was not refused")
    except tt.TetraError as e:
        assert e.status == tt.EBUSY, e.status
    print("17th stream refused with TETRA_EBUSY", flush=True)
    torch.cuda.synchronize()
    tt.release_stream(streams[3].cuda_stream)
    tt.gemv(blob, sg, x, y, M, K, 1, stream=streams[16].cuda_stream)
    torch.cuda.synchronize()
    e = worst(words, sigma, tail, workloads.activations(70, 1, K), y.cpu().numpy())
    assert e <= 1e-5, e
    print(f"after a release the 17th stream runs: worst {e:.3e}", flush=True)


if __name__ == "__main__":
    {"capture": first_call_in_capture, "streams": two_streams, "busy": busy_slots}[sys.argv[1]]()
    print("ok", flush=True)
