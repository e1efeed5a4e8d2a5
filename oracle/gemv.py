"""Dequantised weights and the float64 matrix-vector product (oracle, test-only).

Paper passages followed:
* Eq. 2: w_j = y_j / ||y|| * gain[g] * sigma_row.
* Sec. 4.1: a Tetra projection stores one scale per output row and keeps the
  K mod 24 trailing weights of each row unquantised (f16 on the GPU).
* Sec. 5.1: one output per row, sigma_row applied after the block sums, the
  unquantised tail added last.  The kernel check recomputes every row in f64
  and compares within a multiple of sum_j |w_j x_j|.

Readings: the row scale and the tail are fp16 (the paper's kernel reads the
scale in f32 and the tail in f16); x is fp16 [batch, K]; the block scale is
the f32 s_blk of ``codec.decode``.

Definitions used as the parity target:
    y_ref[b, row] = sigma_row * sum_blk s_blk * sum_j y_j x[b, 24*blk + j]
                    + sum_t tail_t x[b, 24*nblk + t]          (float64)
    norm[b, row]  = sum_k |w_k x[b, k]|                       (float64)

Pins (tests): the dequantised block has Euclidean norm gain[g]*sigma_row for
every nonzero block; x = e_k returns column k of the dequantised matrix;
all-zero words leave only the tail term.
"""

import numpy as np

from . import codec


def split_k(K: int):
    return K // 24, K % 24


def dequant(words, sigma_f16, tail_f16=None) -> np.ndarray:
    """float32 [M, K] weights, w = fl32(fl32(y * s_blk) * sigma)."""
    words = np.asarray(words, dtype=np.uint64)
    M, nblk = words.shape
    y, _, s = codec.decode(words)
    sig = np.asarray(sigma_f16, dtype=np.float16).astype(np.float32)
    w = (y.astype(np.float32) * s[..., None]).astype(np.float32)
    w = (w * sig[:, None, None]).astype(np.float32).reshape(M, nblk * 24)
    if tail_f16 is not None and np.size(tail_f16):
        w = np.concatenate([w, np.asarray(tail_f16, np.float16).astype(np.float32)], axis=1)
    return w


def gemv_f64(words, sigma_f16, tail_f16, x_f16, rows=None):
    """(y_ref, norm), both float64 [batch, len(rows)]."""
    words = np.asarray(words, dtype=np.uint64)
    if rows is not None:
        rows = np.asarray(rows, dtype=np.int64)
        words = words[rows]
        sigma_f16 = np.asarray(sigma_f16)[rows]
        if tail_f16 is not None and np.size(tail_f16):
            tail_f16 = np.asarray(tail_f16)[rows]
    M, nblk = words.shape
    x = np.atleast_2d(np.asarray(x_f16, dtype=np.float16)).astype(np.float64)
    y, _, s = codec.decode(words)
    sig = np.asarray(sigma_f16, dtype=np.float16).astype(np.float64)
    xb = x[:, :nblk * 24].reshape(x.shape[0], nblk, 24)
    # exact integer-times-fp16 dots per block, then the block scale, then sigma
    d = np.einsum("mbj,nbj->nmb", y.astype(np.float64), xb)
    out = sig[None, :] * (d * s.astype(np.float64)[None]).sum(axis=2)
    wabs = np.abs(y.astype(np.float64) * s.astype(np.float64)[..., None]
                  * sig[:, None, None])
    norm = np.einsum("mbj,nbj->nm", wabs, np.abs(xb))
    if tail_f16 is not None and np.size(tail_f16):
        tl = np.asarray(tail_f16, dtype=np.float16).astype(np.float64)
        xt = x[:, nblk * 24:]
        out = out + xt @ tl.T
        norm = norm + np.abs(xt) @ np.abs(tl).T
    return out, norm
