"""Secondary int4 paths of a served file (oracle, test-only).

Paper passages followed:
* Sec. 4.1 and Sec. 4.3: an int4 projection record holds 4-bit weights in
  groups of 128 with an f16 scale and offset per group; a separate kernel
  dequantises each weight with its group's scale and offset and accumulates
  in f32.
* Sec. 4.4: the embedding table is stored in 4 bits in groups of 64 with an
  f16 scale and offset per group; the GPU dequantises the rows of the input
  tokens on the fly.

Readings (the paper gives no bit layout): w = scale * q + offset with q the
unsigned nibble in [0, 15]; groups run along K (along the embedding dimension
for the table); byte k//2 of a row holds element k in its low nibble when k
is even and in its high nibble when k is odd; scale and offset are stored as
fp16 pairs [rows][groups][2].  The dequantised value is formed in f32 as
fma-free fl32(fl32(scale * q) + offset).  Parity unpinned for the layout.

Pins (tests): q = 0 everywhere gives the offsets; a single nonzero nibble
moves exactly one weight by scale * q.
"""

import numpy as np


def unpack_nibbles(q: np.ndarray) -> np.ndarray:
    q = np.asarray(q, dtype=np.uint8)
    out = np.empty(q.shape[:-1] + (q.shape[-1] * 2,), dtype=np.int64)
    out[..., 0::2] = q & 0xF
    out[..., 1::2] = q >> 4
    return out


def dequant_affine(q: np.ndarray, so_f16: np.ndarray, group: int) -> np.ndarray:
    """float32 [rows, K] from nibbles q [rows, K/2] and so [rows, K/group, 2]."""
    n = unpack_nibbles(q).astype(np.float32)
    so = np.asarray(so_f16, dtype=np.float16).astype(np.float32)
    scale = np.repeat(so[..., 0], group, axis=-1)
    off = np.repeat(so[..., 1], group, axis=-1)
    return ((scale * n).astype(np.float32) + off).astype(np.float32)


def int4_gemv_f64(q, so_f16, x_f16, group: int = 128, rows=None):
    """(y_ref, norm) float64 [batch, M] of the int4 projection."""
    q = np.asarray(q)
    so_f16 = np.asarray(so_f16)
    if rows is not None:
        q, so_f16 = q[rows], so_f16[rows]
    w = dequant_affine(q, so_f16, group).astype(np.float64)
    x = np.atleast_2d(np.asarray(x_f16, np.float16)).astype(np.float64)
    return x @ w.T, np.abs(x) @ np.abs(w).T


def emb4_row(q, so_f16, token: int, group: int = 64) -> np.ndarray:
    """float32 [dim] dequantised embedding row of ``token``."""
    return dequant_affine(np.asarray(q)[token:token + 1],
                          np.asarray(so_f16)[token:token + 1], group)[0]
