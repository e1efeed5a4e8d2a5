"""Seeded synthetic workloads: Qwen3-shaped Tetra projections at batch 1/4.

This module draws inputs only; it holds none of the decode arithmetic, so the
CPU oracle and the HIP path can be fed the same bytes.

Every 48-bit value is a legal Tetra word (each field has a power-of-two
range), so uniformly random words stand in for encoded weights.  Row scales
are fp16 U(0.5, 2) * 1e-2, the unquantised tail is fp16 N(0, 1) * sigma_row,
activations are fp16 N(0, 1) of shape [batch, K].

Shapes (out x in) follow the dense Qwen3 models: seven projections per layer
(q, k, v, o, gate, up, down); 36 layers at 4B and 8B, 40 at 14B.
"""

import numpy as np

SEED_BASE = 0x7E7A0000

QWEN3 = {
    "4B": {"hidden": 2560, "q": 4096, "kv": 1024, "inter": 9728, "layers": 36},
    "8B": {"hidden": 4096, "q": 4096, "kv": 1024, "inter": 12288, "layers": 36},
    "14B": {"hidden": 5120, "q": 5120, "kv": 1024, "inter": 17408, "layers": 40},
}

PROJ_NAMES = ("q", "k", "v", "o", "gate", "up", "down")


def layer_shapes(model: str):
    """[(name, M_out, K_in)] for one layer of the named Qwen3 size."""
    c = QWEN3[model]
    h, q, kv, f = c["hidden"], c["q"], c["kv"], c["inter"]
    return [("q", q, h), ("k", kv, h), ("v", kv, h), ("o", h, q),
            ("gate", f, h), ("up", f, h), ("down", h, f)]


def single_shape():
    return [("single", 1536, 1536)]


def config_shapes(config: int):
    """Matrices of a config: 0 single, 1 4B set, 2 8B set, 3 14B set."""
    if config == 0:
        return single_shape()
    return layer_shapes({1: "4B", 2: "8B", 3: "14B"}[config])


def seed_for(config: int, index: int) -> int:
    return SEED_BASE + 16 * config + index


def tetra_matrix(seed: int, M: int, K: int):
    """(words uint64 [M, K//24], sigma fp16 [M], tail fp16 [M, K%24])."""
    rng = np.random.Generator(np.random.PCG64(seed))
    nblk, T = K // 24, K % 24
    raw = rng.integers(0, 256, size=(M, nblk, 6), dtype=np.uint8)
    words = np.zeros((M, nblk), dtype=np.uint64)
    for i in range(6):
        words |= raw[..., i].astype(np.uint64) << np.uint64(8 * i)
    sigma = (rng.uniform(0.5, 2.0, size=M) * 1e-2).astype(np.float16)
    tail = (rng.standard_normal((M, T)) * sigma.astype(np.float64)[:, None]).astype(np.float16)
    return words, sigma, tail


def activations(seed: int, batch: int, K: int):
    rng = np.random.Generator(np.random.PCG64(seed ^ 0x5A5A))
    return rng.standard_normal((batch, K)).astype(np.float16)


def int4_matrix(seed: int, M: int, K: int, group: int = 128):
    """(q uint8 [M, K/2], scale/offset fp16 [M, K/group, 2])."""
    rng = np.random.Generator(np.random.PCG64(seed ^ 0x1234))
    q = rng.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
    scale = rng.uniform(0.5, 2.0, size=(M, K // group)) * 1e-2 / 8
    so = np.stack([scale, -7.5 * scale], axis=-1).astype(np.float16)
    return q, so


def int4_pick(seed: int, n_total: int, frac: float = 0.1):
    """Seeded choice of which matrices of a step are stored as int4."""
    rng = np.random.Generator(np.random.PCG64(seed ^ 0x77))
    k = int(round(frac * n_total))
    return np.sort(rng.permutation(n_total)[:k])


def emb4_table(seed: int, rows: int, dim: int, group: int = 64):
    rng = np.random.Generator(np.random.PCG64(seed ^ 0xE4))
    q = rng.integers(0, 256, size=(rows, dim // 2), dtype=np.uint8)
    scale = rng.uniform(0.5, 2.0, size=(rows, dim // group)) * 1e-2 / 8
    so = np.stack([scale, -7.5 * scale], axis=-1).astype(np.float16)
    token = int(rng.integers(0, rows))
    return q, so, token
